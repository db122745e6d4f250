"""GPU parity of the LSTM acoustic model forward/backward against the fp64
oracle at sizes the oracle finishes in seconds: several tiles of every kernel
plus ragged tails, variable lengths, initial states, fp32 (1e-4) and bf16
(2e-2) paths, and run-to-run determinism."""

import numpy as np
import pytest

import oracle
from paper_1904_10584_amd import binding as am
from paper_1904_10584_amd import synth
from tests.gpu_util import (gpu_forward_backward, oracle_forward_backward, per_tensor_errors,
                            rel_l2, say)

pytestmark = pytest.mark.gpu

F32_TOL = 1e-4
BF16_TOL = 2e-2


@pytest.fixture(params=["auto", "device", "step"], autouse=True)
def recurrence_path(request, monkeypatch):
    """Every test runs with the default recurrence kernels (XCD-local where
    the shape is covered), with the device-scope persistent kernels, and
    with one launch per time step."""
    monkeypatch.delenv("AM_STEP_KERNELS", raising=False)
    if request.param == "auto":
        monkeypatch.delenv("AM_RECURRENCE", raising=False)
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
    assert abs(got["loss"] - ref["loss"]) <= tol * abs(ref["loss"])
    assert rel_l2(got["logits"], ref["logits"]) <= tol
    assert rel_l2(got["dlogits"], ref["dlogits"]) <= tol
    errs = per_tensor_errors(got["grads"], ref["grads"], dims)
    bad = {k: v for k, v in errs.items() if not v <= tol}
    assert not bad, bad
    if state:
        assert rel_l2(got["hT"], ref["hT"]) <= tol
        assert rel_l2(got["cT"], ref["cT"]) <= tol
    return errs


def test_tiny_fp32_step_matches_oracle():
    # 2 layers x 64 cells, 64-dim input, 500 classes, 16 chunks x 50 frames, k = 5
    w = synth.WORKLOADS["tiny-2x64"]
    dims = oracle.ModelDims(w["layers"], w["input_dim"], w["hidden"], w["classes"])
    say("tiny fp32 step")
    master, x, idx, prob, _, _ = _problem(dims, w["T"], w["B"], w["K"], w["mass"])
    m = am.Model(dims.layers, dims.input_dim, dims.hidden, dims.classes, am.F32)
    got = gpu_forward_backward(m, master, x, w["T"], w["B"], idx, prob)
    ref = oracle_forward_backward(dims, master, x, w["T"], w["B"], idx, prob)
    errs = _check(got, ref, dims, F32_TOL)
    say(f"  max rel err {max(errs.values()):.2e}")


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
    errs = _check(got, ref, dims, BF16_TOL, state=True)
    say(f"  max rel err {max(errs.values()):.2e}")


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
    errs = _check(got, ref, dims, BF16_TOL, state=True)
    say(f"  max rel err {max(errs.values()):.2e}")


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
