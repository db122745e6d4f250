"""The bf16 per-step forward with the LSTM cell in the recurrent product's
epilogue (one launch per step) against the same step as two launches (the
product into fp32 scratch, then the cell kernel): same arithmetic in the
same order, so logits, final state and every gradient must agree bit for
bit.  Shapes cover 128- and 64-wide tiles, a partial last column tile
(4H = 320), ragged row tiles and variable lengths.  Parity of the fused path
with the oracle is covered by the model tests' per-step runs."""

import numpy as np
import pytest

import oracle
from paper_1904_10584_amd import binding as am
from paper_1904_10584_amd import synth
from tests.gpu_util import gpu_forward_backward, say

pytestmark = pytest.mark.gpu

CASES = [
    # (layers, input, hidden, classes, T, B, lengths)
    (2, 64, 1536, 96, 3, 512, None),          # 128 x 128 tiles (B = 512, 4H = 6144)
    (2, 24, 80, 40, 9, 37, "varlen"),         # 64 x 64 tiles, 4H = 320, ragged rows
    (1, 16, 256, 56, 5, 130, None),           # rows past a tile boundary
]


@pytest.mark.parametrize("case", CASES, ids=["wide-512x1536", "h80-varlen", "h256-b130"])
def test_fused_step_matches_two_launch_step_bitwise(case, monkeypatch):
    L, D, H, C, T, B, lk = case
    say(f"step fusion: L={L} D={D} H={H} C={C} T={T} B={B} lengths={lk}")
    lengths = None
    if lk == "varlen":
        lengths = np.sort(np.random.default_rng(5).integers(1, T + 1, B))[::-1].astype(np.int32)
        lengths[0] = T
    dims = oracle.ModelDims(L, D, H, C)
    counts, offs = oracle.batch_schedule(T, B, lengths)
    N = int(offs[-1])
    master = synth.init_params(oracle.param_count(dims), H, seed=11)
    x = synth.features(N, D, seed=12)
    idx, prob = synth.teacher_targets(N, C, 4, 0.95, seed=13)
    rng = np.random.default_rng(14)
    h0 = rng.uniform(-0.5, 0.5, (L, B, H)).astype(np.float32)
    c0 = rng.uniform(-0.5, 0.5, (L, B, H)).astype(np.float32)
    m = am.Model(L, D, H, C, am.BF16)
    monkeypatch.setenv("AM_RECURRENCE", "step")
    out = {}
    for fusion in ("1", "0"):
        monkeypatch.setenv("AM_STEP_FUSION", fusion)
        out[fusion] = gpu_forward_backward(m, master, x, T, B, idx, prob, lengths=lengths,
                                           h0=h0, c0=c0, want_state=True)
    for key in ("logits", "dlogits", "grads", "hT", "cT"):
        a, b = out["1"][key], out["0"][key]
        assert np.isfinite(a).all(), key
        assert np.array_equal(a.view(np.uint32), b.view(np.uint32)), \
            f"{key}: {int(np.sum(a.view(np.uint32) != b.view(np.uint32)))} elements differ"
    assert out["1"]["loss"] == out["0"]["loss"]
