"""GPU parity of the LSTM acoustic model forward/backward against the fp64
oracle at sizes the oracle finishes in seconds: several tiles of every kernel
plus ragged tails, variable lengths, initial states, fp32 (1e-4) and bf16
(2e-2) paths, and run-to-run determinism."""

import numpy as np
import pytest
import torch

import oracle
from paper_1904_10584_amd import binding as am
from paper_1904_10584_amd import synth
from tests.gpu_util import (assert_close, bf16_dev, check_grads, gpu_forward_backward,
                            oracle_forward_backward, say)

pytestmark = pytest.mark.gpu

F32_TOL = 1e-4
BF16_TOL = 2e-2


@pytest.fixture(params=["auto", "fenced", "device", "step"], autouse=True)
def recurrence_path(request, monkeypatch):
    """Every test runs with the default recurrence kernels (XCD-local where
    the shape is covered), with the XCD-local kernels forced onto their
    fenced exchange (the path a block that spans XCDs takes), with the
    device-scope persistent kernels, and with one launch per time step."""
    monkeypatch.delenv("AM_STEP_KERNELS", raising=False)
    monkeypatch.delenv("AM_XCD_FENCED", raising=False)
    if request.param in ("auto", "fenced"):
        monkeypatch.delenv("AM_RECURRENCE", raising=False)
        if request.param == "fenced":
            monkeypatch.setenv("AM_XCD_FENCED", "1")
    else:
        monkeypatch.setenv("AM_RECURRENCE", request.param)
    return request.param


def _problem(dims, T, B, K, mass, lengths=None, seed=0, state=False, one_hot_frac=0.0):
    counts, offs = oracle.batch_schedule(T, B, lengths)
    N = int(offs[-1])
    n = oracle.param_count(dims)
    master = synth.init_params(n, dims.hidden, seed=seed)
    x = synth.features(N, dims.input_dim, seed=seed + 1)
    idx, prob = synth.teacher_targets(N, dims.classes, K, mass, seed=seed + 2,
                                      one_hot_frac=one_hot_frac)
    h0 = c0 = None
    if state:
        rng = np.random.default_rng(seed + 9)
        h0 = rng.uniform(-0.5, 0.5, (dims.layers, B, dims.hidden)).astype(np.float32)
        c0 = rng.uniform(-0.5, 0.5, (dims.layers, B, dims.hidden)).astype(np.float32)
    return master, x, idx, prob, h0, c0


def _check(got, ref, dims, tol, state=False):
    """Loss, then the per-tensor rel L2 and element-wise bounds on logits,
    dlogits, every gradient tensor and (state) the final h and c."""
    assert abs(got["loss"] - ref["loss"]) <= tol * abs(ref["loss"])
    assert_close("logits", got["logits"], ref["logits"], tol)
    assert_close("dlogits", got["dlogits"], ref["dlogits"], tol)
    worst = check_grads(got["grads"], ref["grads"], dims, tol)
    if state:
        assert_close("hT", got["hT"], ref["hT"], tol)
        assert_close("cT", got["cT"], ref["cT"], tol)
    return worst


def test_tiny_fp32_step_matches_oracle():
    # 2 layers x 64 cells, 64-dim input, 500 classes, 16 chunks x 50 frames, k = 5
    w = synth.WORKLOADS["tiny-2x64"]
    dims = oracle.ModelDims(w["layers"], w["input_dim"], w["hidden"], w["classes"])
    say("tiny fp32 step")
    master, x, idx, prob, _, _ = _problem(dims, w["T"], w["B"], w["K"], w["mass"])
    m = am.Model(dims.layers, dims.input_dim, dims.hidden, dims.classes, am.F32)
    got = gpu_forward_backward(m, master, x, w["T"], w["B"], idx, prob)
    ref = oracle_forward_backward(dims, master, x, w["T"], w["B"], idx, prob)
    l2, mr = _check(got, ref, dims, F32_TOL)
    say(f"  gradients: max rel L2 {l2:.2e}, max element ratio {mr:.2e}")


@pytest.mark.parametrize("case", ["ragged", "varlen_state"])
def test_fp32_ragged_shapes(case):
    # hidden 48: a partial 32-wide k-step; 70 sequences: a partial 64-row tile;
    # 36-dim input and 500 classes: partial GEMM k- and n-tiles.
    dims = oracle.ModelDims(3, 36, 48, 500)
    T, B = 7, 70
    lengths = None
    state = case == "varlen_state"
    if state:
        lengths = np.sort(np.random.default_rng(4).integers(0, T + 1, B))[::-1].astype(np.int32)
        lengths[0] = T
    say(f"fp32 {case}")
    master, x, idx, prob, h0, c0 = _problem(dims, T, B, 4, 0.9, lengths, seed=3, state=state)
    m = am.Model(dims.layers, dims.input_dim, dims.hidden, dims.classes, am.F32)
    got = gpu_forward_backward(m, master, x, T, B, idx, prob, lengths, h0, c0, want_state=True)
    ref = oracle_forward_backward(dims, master, x, T, B, idx, prob, lengths, h0, c0)
    _check(got, ref, dims, F32_TOL, state=True)


@pytest.mark.parametrize("lengths_kind", [None, "varlen"])
def test_bf16_small_matches_oracle(lengths_kind):
    dims = oracle.ModelDims(2, 64, 128, 520)
    T, B = 12, 80
    lengths = None
    if lengths_kind:
        lengths = np.sort(np.random.default_rng(1).integers(1, T + 1, B))[::-1].astype(np.int32)
    say(f"bf16 small {lengths_kind}")
    master, x, idx, prob, _, _ = _problem(dims, T, B, 8, 0.98, lengths, seed=11, one_hot_frac=0.1)
    m = am.Model(dims.layers, dims.input_dim, dims.hidden, dims.classes, am.BF16)
    got = gpu_forward_backward(m, master, x, T, B, idx, prob, lengths, want_state=True)
    ref = oracle_forward_backward(dims, master, x, T, B, idx, prob, lengths, bf16=True)
    l2, mr = _check(got, ref, dims, BF16_TOL, state=True)
    say(f"  gradients: max rel L2 {l2:.2e}, max element ratio {mr:.2e}")


@pytest.mark.parametrize("blocks", ["pairs", "single"])
def test_bf16_wide_batch_block_layouts(blocks, monkeypatch):
    # 200 sequences (> 128): by default blocks of 16 sequences, two per XCD
    # (13 blocks, the last one half full); AM_XCD_BLOCKS=1 selects blocks of
    # 32, one per XCD.  Varying lengths end blocks at different steps.
    if blocks == "single":
        monkeypatch.setenv("AM_XCD_BLOCKS", "1")
    else:
        monkeypatch.delenv("AM_XCD_BLOCKS", raising=False)
    dims = oracle.ModelDims(2, 64, 128, 520)
    T, B = 6, 200
    lengths = np.sort(np.random.default_rng(8).integers(1, T + 1, B))[::-1].astype(np.int32)
    lengths[0] = T
    say(f"bf16 wide batch, {blocks}")
    master, x, idx, prob, h0, c0 = _problem(dims, T, B, 8, 0.98, lengths, seed=17, state=True)
    m = am.Model(dims.layers, dims.input_dim, dims.hidden, dims.classes, am.BF16)
    got = gpu_forward_backward(m, master, x, T, B, idx, prob, lengths, h0, c0, want_state=True)
    ref = oracle_forward_backward(dims, master, x, T, B, idx, prob, lengths, h0, c0, bf16=True)
    l2, mr = _check(got, ref, dims, BF16_TOL, state=True)
    say(f"  gradients: max rel L2 {l2:.2e}, max element ratio {mr:.2e}")


def test_runs_are_bitwise_deterministic():
    dims = oracle.ModelDims(2, 64, 128, 520)
    T, B = 9, 130
    master, x, idx, prob, _, _ = _problem(dims, T, B, 8, 0.98, seed=21)
    m = am.Model(dims.layers, dims.input_dim, dims.hidden, dims.classes, am.BF16)
    a = gpu_forward_backward(m, master, x, T, B, idx, prob)
    b = gpu_forward_backward(m, master, x, T, B, idx, prob)
    for k in ("logits", "dlogits", "grads"):
        np.testing.assert_array_equal(a[k].view(np.uint32), b[k].view(np.uint32))
    assert a["loss"] == b["loss"]


def test_chunk_with_no_frames_and_single_frame():
    dims = oracle.ModelDims(2, 8, 16, 8)
    T, B = 3, 3
    lengths = np.array([3, 1, 0], np.int32)
    master, x, idx, prob, h0, c0 = _problem(dims, T, B, 2, 0.9, lengths, seed=5, state=True)
    m = am.Model(dims.layers, dims.input_dim, dims.hidden, dims.classes, am.F32)
    got = gpu_forward_backward(m, master, x, T, B, idx, prob, lengths, h0, c0, want_state=True)
    ref = oracle_forward_backward(dims, master, x, T, B, idx, prob, lengths, h0, c0)
    _check(got, ref, dims, F32_TOL, state=True)


def test_timed_out_pass_yields_zero_gradient():
    # The time-out flag (last word of the workspace's first 8 KiB sync slot)
    # is set from the host between forward and backward, as a barrier wait
    # that ran out would set it; no kernel waits on it.  The backward must
    # then leave a zero gradient and the check must report the time-out.
    dims = oracle.ModelDims(2, 64, 128, 520)
    T, B = 5, 40
    master, x, idx, prob, _, _ = _problem(dims, T, B, 8, 0.98, seed=31)
    m = am.Model(dims.layers, dims.input_dim, dims.hidden, dims.classes, am.BF16)
    params = bf16_dev(master)
    xd = bf16_dev(x)
    N = T * B
    logits = torch.empty((N, m.classes), dtype=torch.float32, device="cuda")
    ws = torch.empty(am.workspace_bytes(m, T, B, N), dtype=torch.uint8, device="cuda")
    am.lstm_am_forward(m, params, xd, T, B, logits, ws)
    dz = torch.full((N, m.classes), 1e-3, dtype=torch.bfloat16, device="cuda")
    grads = torch.full((am.param_count(m),), 7.0, dtype=torch.float32, device="cuda")
    ws[8188:8192].view(torch.int32).fill_(1)
    am.lstm_am_backward(m, params, xd, T, B, dz, ws, grads)
    with pytest.raises(am.AmError) as ei:
        am.workspace_check(ws)
    assert ei.value.status == am.ETIMEOUT
    assert bool(torch.all(grads == 0.0))
    # the next forward clears the flag; a normal pass leaves a nonzero gradient
    am.lstm_am_forward(m, params, xd, T, B, logits, ws)
    am.lstm_am_backward(m, params, xd, T, B, dz, ws, grads)
    am.workspace_check(ws)
    assert float(grads.abs().max()) > 0.0
