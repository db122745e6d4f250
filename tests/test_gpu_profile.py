"""The library's launch timing (am_profile_*): with sampling, one launch in n
of a recorded class is bracketed, and the class totals cover exactly the
sampled launches (their count, their summed algorithmic bytes)."""

import pytest
import torch

from paper_1904_10584_amd import binding as am
from tests.gpu_util import say

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("every", [1, 3, 7])
def test_sampled_brackets_count_every_nth_launch(every):
    n, launches = 1 << 20, 10
    say(f"profile sampling: every={every}, {launches} SGD launches of n={n}")
    master = torch.zeros(n, dtype=torch.float32, device="cuda")
    upd = torch.ones(n, dtype=torch.float32, device="cuda")
    # one unsampled run for the per-launch figures
    am.profile_begin([am.K_SGD])
    am.sgd_apply(master, upd, 0.5)
    am.profile_end()
    one = am.profile_get(am.K_SGD)
    assert one["launches"] == 1 and one["ms"] > 0.0 and one["bytes"] > 0.0
    am.profile_begin([am.K_SGD], every=every)
    for _ in range(launches):
        am.sgd_apply(master, upd, 0.5)
    am.profile_end()
    got = am.profile_get(am.K_SGD)
    want = (launches + every - 1) // every  # launches 0, every, 2 every, ...
    assert got["launches"] == want
    assert got["bytes"] == pytest.approx(want * one["bytes"])
    assert got["ms"] > 0.0
    # unrecorded classes stay empty
    assert am.profile_get(am.K_ENCODE)["launches"] == 0
    am.profile_begin([], every=1)  # (restores the default interval)
    am.profile_end()
    torch.cuda.synchronize()
    assert float(master[0]) == pytest.approx(-0.5 * (launches + 1))
