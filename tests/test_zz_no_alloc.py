"""The encode entry point that allocates nothing (library-owned scratch),
called through the C ABI, against grad_threshold_encode with a workspace:
residual, words and count bit for bit, on two calls in a row (the second
with a smaller input, so that it runs on scratch left by the first), and
its size limit checked on the host before anything is enqueued."""

import numpy as np
import pytest
import torch

from paper_1904_10584_amd import binding as am

pytestmark = pytest.mark.gpu


def _inputs(n, seed):
    rng = np.random.default_rng(seed)
    g = (rng.standard_normal(n) * 1e-4).astype(np.float32)
    r = (rng.standard_normal(n) * 5e-5).astype(np.float32)
    return torch.from_numpy(g).cuda(), torch.from_numpy(r).cuda()


def _encode(n, seed, tau, noalloc):
    g, r = _inputs(n, seed)
    words = torch.full((n,), -1, dtype=torch.int32, device="cuda")
    count = torch.full((1,), -1, dtype=torch.int64, device="cuda")
    if noalloc:
        am.grad_threshold_encode_noalloc(g, r, tau, words, count)
    else:
        ws = torch.zeros(am.encode_workspace_bytes(n), dtype=torch.uint8, device="cuda")
        am.grad_threshold_encode(g, r, tau, words, count, ws)
    torch.cuda.synchronize()
    c = int(count.cpu()[0])
    return r.cpu().numpy().view(np.uint32), words[:c].cpu().numpy().view(np.uint32), c


def test_noalloc_encode_matches_workspace_encode_twice():
    tau = 1e-4
    for n, seed in ((24_145_848, 1), (1_000_003, 2)):
        r_a, w_a, c_a = _encode(n, seed, tau, noalloc=True)
        r_b, w_b, c_b = _encode(n, seed, tau, noalloc=False)
        assert c_a == c_b and c_a > 0
        np.testing.assert_array_equal(r_a, r_b)
        np.testing.assert_array_equal(w_a, w_b)


def test_noalloc_encode_size_limit():
    n = am.ENCODE_NOALLOC_MAX_N + 1
    g = torch.zeros(16, dtype=torch.float32, device="cuda")
    count = torch.full((1,), 5, dtype=torch.int64, device="cuda")
    # the host check rejects n before any pointer is used: pass n explicitly
    st = am.lib().grad_threshold_encode_noalloc(n, am._dev(g, "g"), am._dev(g, "r"), 1e-4,
                                               am._dev(g, "w"), n, am._dev(count, "c"), None)
    assert st == am.EUNSUPPORTED
    assert "n <=" in am.lib().am_last_error().decode()
    torch.cuda.synchronize()
    assert int(count.cpu()[0]) == 5
