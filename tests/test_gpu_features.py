"""GPU parity of the student-input pieces (§II-B) against the oracle, through
the C ABI: stacked low-frame-rate features with causal mean subtraction and
global normalisation (bit for bit, fp32 and bf16), targets delayed by the
look-ahead (bit for bit), a chunked forward with carried state against the
unchunked forward, and the whole path from raw frames to gradients."""

import numpy as np
import pytest
import torch

import oracle
from paper_1904_10584_amd import binding as am
from paper_1904_10584_amd import synth
from tests.gpu_util import assert_close, bf16_dev, check_grads, say, to_dev

pytestmark = pytest.mark.gpu


def _sorted_raw_lengths(rng, B, lo, hi, offset):
    """Raw lengths whose stacked lengths are non-increasing (plus empty ones)."""
    U = np.sort(rng.integers(lo, hi + 1, B))[::-1].astype(np.int32)
    U[-2:] = [2, 0]  # too short for a stack, and empty
    T = np.array([oracle.lfr_frames(int(u), 3, 3, offset) for u in U])
    assert np.all(np.diff(T) <= 0)
    return U, T


def _oracle_packed(raw, U, T, mean, std, offset):
    """Oracle features of each utterance, placed in the packed layout."""
    B = len(U)
    Tmax = int(T[0]) if B else 0
    counts, offs = oracle.batch_schedule(Tmax, B, T)
    out = np.zeros((int(offs[-1]), 192))
    r0 = 0
    for b in range(B):
        f = oracle.lfr_features(raw[r0:r0 + U[b]], mean, std, 3, 3, offset)
        for t in range(f.shape[0]):
            out[int(offs[t]) + b] = f[t]
        r0 += int(U[b])
    return out


@pytest.mark.parametrize("offset", [0, 1, 2])
@pytest.mark.parametrize("bf16", [False, True])
def test_lfr_features_bit_exact(offset, bf16):
    rng = np.random.default_rng(10 + offset)
    U, T = _sorted_raw_lengths(rng, 23, 30, 700, offset)
    raw = synth.raw_logmel(U, seed=7 + offset)
    mean = rng.normal(0, 0.5, 192).astype(np.float32)
    std = rng.uniform(0.5, 2.0, 192).astype(np.float32)
    N = int(T.sum())
    say(f"lfr features offset={offset} bf16={bf16} utterances={len(U)} frames={N}")
    x = torch.zeros((N, 192), dtype=torch.bfloat16 if bf16 else torch.float32, device="cuda")
    am.lfr_features(U, to_dev(raw), to_dev(mean), to_dev(std), x, offset=offset)
    torch.cuda.synchronize()
    ref = _oracle_packed(raw, U, T, mean, std, offset).astype(np.float32)
    if bf16:
        got = x.cpu().view(torch.int16).numpy().view(np.uint16)
        np.testing.assert_array_equal(got, oracle.bf16_bits(ref))
    else:
        np.testing.assert_array_equal(x.cpu().numpy().view(np.uint32), ref.view(np.uint32))


@pytest.mark.parametrize("lengths_kind", [None, "varlen"])
@pytest.mark.parametrize("delay", [0, 1, 3])
def test_delay_targets_bit_exact(lengths_kind, delay):
    T, B, K = 40, 37, 20
    lengths = None
    if lengths_kind:
        lengths = np.sort(np.random.default_rng(3).integers(0, T + 1, B))[::-1].astype(np.int32)
    counts, offs = oracle.batch_schedule(T, B, lengths)
    N = int(offs[-1])
    idx, prob = synth.teacher_targets(N, 3000, K, 0.98, one_hot_frac=0.1)
    ref_i, ref_p, ref_m = oracle.delay_targets(idx, prob, T, B, lengths, delay)
    io = torch.full((N, K), 7, dtype=torch.int32, device="cuda")
    po = torch.full((N, K), 7.0, dtype=torch.float32, device="cuda")
    mo = torch.full((N,), 7, dtype=torch.uint8, device="cuda")
    am.delay_targets(T, B, to_dev(idx), to_dev(prob), io, po, mo, delay, lengths=lengths)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(io.cpu().numpy(), ref_i)
    np.testing.assert_array_equal(po.cpu().numpy().view(np.uint32), ref_p.astype(np.float32).view(np.uint32))
    np.testing.assert_array_equal(mo.cpu().numpy(), ref_m)


def _forward(m, params, x, T, B, h0=None, c0=None):
    N = x.shape[0]
    logits = torch.empty((N, m.classes), dtype=torch.float32, device="cuda")
    ws = torch.empty(am.workspace_bytes(m, T, B, N), dtype=torch.uint8, device="cuda")
    hT = torch.empty((m.layers, B, m.hidden), dtype=torch.float32, device="cuda")
    cT = torch.empty_like(hT)
    am.lstm_am_forward(m, params, x, T, B, logits, ws, h0=h0, c0=c0, hT=hT, cT=cT)
    am.workspace_check(ws)
    return logits, hT, cT


@pytest.mark.parametrize("bf16", [False, True])
def test_chunked_forward_with_carried_state_equals_unchunked(bf16):
    # the 5x768 student on 64 chunks: 48 frames at once, or 20 then 28 frames
    # with the state carried; the same kernels take the same steps
    L, D0, H, C = 5, 192, 768, 3000
    T, B, T1 = 48, 64, 20
    m = am.Model(L, D0, H, C, am.BF16 if bf16 else am.F32)
    n = am.param_count(m)
    master = synth.init_params(n, H)
    x = synth.features(T * B, D0)
    if bf16:
        params, xd = bf16_dev(master), bf16_dev(x)
    else:
        params, xd = to_dev(master), to_dev(x)
    say(f"carried state bf16={bf16}")
    full, hT, cT = _forward(m, params, xd, T, B)
    a, ha, ca = _forward(m, params, xd[:T1 * B], T1, B)
    b, hb, cb = _forward(m, params, xd[T1 * B:], T - T1, B, h0=ha, c0=ca)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(torch.cat([a, b]).cpu().numpy().view(np.uint32), full.cpu().numpy().view(np.uint32))
    np.testing.assert_array_equal(hb.cpu().numpy().view(np.uint32), hT.cpu().numpy().view(np.uint32))
    np.testing.assert_array_equal(cb.cpu().numpy().view(np.uint32), cT.cpu().numpy().view(np.uint32))


def test_raw_frames_to_gradients_with_carried_state_and_delay():
    # raw 10 ms frames -> stacked features (offset 1) -> second chunk of a
    # forward whose state is carried from a first chunk -> targets delayed by
    # three frames -> soft CE on the masked rows -> BPTT; against the oracle
    dims = oracle.ModelDims(2, 192, 128, 520)
    B, offset, d, K = 12, 1, 3, 8
    rng = np.random.default_rng(40)
    U = np.full(B, 3 * 30 + offset + 2, np.int32)  # 30 stacked frames each
    T = oracle.lfr_frames(int(U[0]), 3, 3, offset)
    raw = synth.raw_logmel(U, seed=41)
    mean = rng.normal(2.0, 0.5, 192).astype(np.float32)
    std = rng.uniform(2.0, 4.0, 192).astype(np.float32)
    n = oracle.param_count(dims)
    master = synth.init_params(n, dims.hidden, seed=42)
    h0 = rng.uniform(-0.5, 0.5, (dims.layers, B, dims.hidden)).astype(np.float32)
    c0 = rng.uniform(-0.5, 0.5, (dims.layers, B, dims.hidden)).astype(np.float32)
    idx, prob = synth.teacher_targets(T * B, dims.classes, K, 0.98, seed=43)
    say(f"raw frames to gradients: T={T} B={B}")

    m = am.Model(dims.layers, dims.input_dim, dims.hidden, dims.classes, am.F32)
    x = torch.empty((T * B, 192), dtype=torch.float32, device="cuda")
    am.lfr_features(U, to_dev(raw), to_dev(mean), to_dev(std), x, offset=offset)
    io = torch.empty((T * B, K), dtype=torch.int32, device="cuda")
    po = torch.empty((T * B, K), dtype=torch.float32, device="cuda")
    mo = torch.empty((T * B,), dtype=torch.uint8, device="cuda")
    am.delay_targets(T, B, to_dev(idx), to_dev(prob), io, po, mo, d)
    params = to_dev(master)
    logits = torch.empty((T * B, dims.classes), dtype=torch.float32, device="cuda")
    ws = torch.empty(am.workspace_bytes(m, T, B, T * B), dtype=torch.uint8, device="cuda")
    am.lstm_am_forward(m, params, x, T, B, logits, ws, h0=to_dev(h0), c0=to_dev(c0))
    loss = torch.zeros(1, dtype=torch.float32, device="cuda")
    dz = torch.empty_like(logits)
    cws = torch.empty(am.ce_workspace_bytes(T * B), dtype=torch.uint8, device="cuda")
    am.sparse_soft_ce(logits, io, po, loss, dz, cws, mask=mo)
    grads = torch.empty(n, dtype=torch.float32, device="cuda")
    am.lstm_am_backward(m, params, x, T, B, dz, ws, grads)
    am.workspace_check(ws)
    torch.cuda.synchronize()

    xr = np.zeros((T * B, 192))
    for b in range(B):
        f = oracle.lfr_features(raw[b * U[0]:(b + 1) * U[0]], mean, std, 3, 3, offset)
        xr[b::B] = f
    np.testing.assert_array_equal(x.cpu().numpy().view(np.uint32), xr.astype(np.float32).view(np.uint32))
    ref_logits, cache = oracle.lstm_am_forward(master, dims, xr.astype(np.float32), T, B, None, h0, c0)
    i_d, p_d, msk = oracle.delay_targets(idx, prob, T, B, None, d)
    ref_loss, ref_dz = oracle.sparse_soft_ce(ref_logits, i_d, p_d, msk)
    ref_grads = oracle.lstm_am_backward(master, dims, cache, ref_dz)
    assert abs(float(loss.cpu()[0]) - ref_loss) <= 1e-4 * abs(ref_loss)
    assert_close("logits", logits.cpu().numpy(), ref_logits, 1e-4)
    assert_close("dlogits", dz.cpu().numpy(), ref_dz, 1e-4)
    check_grads(grads.cpu().numpy(), ref_grads, dims, 1e-4)
