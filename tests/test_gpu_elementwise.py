"""GPU parity of the HBM-bound entry points against the oracle: SGD and the
bf16 cast (bit-exact), threshold encode/decode (bit-exact) and the sparse
soft-target cross-entropy (fp32 tolerance).  Calls go through the C ABI."""

import numpy as np
import pytest
import torch

import oracle
from paper_1904_10584_amd import binding as am
from tests.gpu_util import assert_close, say, to_dev

pytestmark = pytest.mark.gpu


def _bits32(a):
    return np.asarray(a, np.float32).view(np.uint32)


@pytest.mark.parametrize("n,offset", [(1, 0), (1003, 0), (1 << 20, 0), (77777, 1)])
def test_sgd_bit_exact(n, offset):
    say(f"sgd n={n} offset={offset}")
    rng = np.random.default_rng(n)
    w = rng.standard_normal(n + offset).astype(np.float32)
    u = (rng.standard_normal(n + offset) * 3).astype(np.float32)
    w[:5] = [0.0, -0.0, 1e-40, 3e38, -1e-45][: min(5, n + offset)]
    lr = np.float32(0.01)
    wd = to_dev(w)
    ud = to_dev(u)
    bd = torch.zeros(n + offset, dtype=torch.bfloat16, device="cuda")
    am.sgd_apply(wd[offset:], ud[offset:], lr, bd[offset:])
    ref_w, ref_b = oracle.sgd_apply(w[offset:], u[offset:], lr)
    got_w = wd.cpu().numpy()[offset:]
    got_b = bd.cpu().view(torch.int16).numpy().view(np.uint16)[offset:]
    np.testing.assert_array_equal(_bits32(got_w), _bits32(ref_w))
    np.testing.assert_array_equal(got_b, ref_b)


def test_cast_bit_exact_special_values():
    hi = np.arange(1 << 16, dtype=np.uint32) << np.uint32(16)
    lows = np.array([0, 1, 0x7FFF, 0x8000, 0x8001, 0xFFFF], dtype=np.uint32)
    x = (hi[:, None] | lows[None, :]).ravel().view(np.float32)
    d = torch.empty(x.shape[0], dtype=torch.bfloat16, device="cuda")
    am.cast_f32_to_bf16(to_dev(x), d)
    got = d.cpu().view(torch.int16).numpy().view(np.uint16)
    np.testing.assert_array_equal(got, oracle.bf16_bits(x))


def _encode_gpu(g, r, tau, capacity=None):
    n = g.shape[0]
    gd, rd = to_dev(g), to_dev(r)
    words = torch.zeros(max(capacity or n, 1), dtype=torch.int32, device="cuda")
    count = torch.full((1,), -7, dtype=torch.int64, device="cuda")
    ws = torch.zeros(max(am.encode_workspace_bytes(n), 256), dtype=torch.uint8, device="cuda")
    am.grad_threshold_encode(gd, rd, tau, words, count, ws)
    c = int(count.cpu()[0])
    return rd.cpu().numpy(), words.cpu().numpy().view(np.uint32)[:c], c, words, count


# (beyond 8192 tiles of 4096 elements the compaction takes a scan of the
# tile counts: 40,000,003)
@pytest.mark.parametrize("n", [0, 1, 4095, 4096, 4097, 1_000_003, 40_000_003])
def test_encode_bit_exact(n):
    say(f"encode n={n}")
    rng = np.random.default_rng(n + 1)
    tau = np.float32(1e-3)
    g = (rng.standard_normal(n) * 1e-3).astype(np.float32)
    r = (rng.standard_normal(n) * 5e-4).astype(np.float32)
    ref_r, ref_w, ref_c = oracle.grad_threshold_encode(g, r, tau)
    got_r, got_w, got_c, _, _ = _encode_gpu(g, r, tau)
    assert got_c == ref_c
    np.testing.assert_array_equal(_bits32(got_r), _bits32(ref_r))
    np.testing.assert_array_equal(got_w, ref_w)


def test_encode_adversarial_and_extremes():
    tau = np.float32(0.5)
    sub = np.array([1], np.uint32).view(np.float32)[0]
    base_g = np.array([0.5, -0.5, np.nextafter(np.float32(0.5), np.float32(1)), 1.0, -1.75, -0.0,
                       sub, np.inf, -np.inf, np.nan, 3e38, 0.0], np.float32)
    base_r = np.array([0, 0, 0, 0, 0, -0.0, sub, 0, 0, 0, 3e38, 1e-30], np.float32)
    g = np.tile(base_g, 700)
    r = np.tile(base_r, 700)
    ref_r, ref_w, ref_c = oracle.grad_threshold_encode(g, r, tau)
    got_r, got_w, got_c, _, _ = _encode_gpu(g, r, tau)
    assert got_c == ref_c
    np.testing.assert_array_equal(_bits32(got_r), _bits32(ref_r))
    np.testing.assert_array_equal(got_w, ref_w)
    # every element sent / none sent
    for tau2, gg in ((np.float32(1e-3), np.full(9000, 1.0, np.float32)),
                     (np.float32(np.inf), np.full(9000, 1.0, np.float32))):
        rr = np.zeros_like(gg)
        ref_r, ref_w, ref_c = oracle.grad_threshold_encode(gg, rr, tau2)
        got_r, got_w, got_c, _, _ = _encode_gpu(gg, rr, tau2)
        assert got_c == ref_c
        np.testing.assert_array_equal(got_w, ref_w)
        np.testing.assert_array_equal(_bits32(got_r), _bits32(ref_r))


def test_encode_multi_step_residual_feedback():
    rng = np.random.default_rng(5)
    n, tau = 300_001, np.float32(2e-3)
    r = np.zeros(n, np.float32)
    rd = to_dev(r)
    words = torch.zeros(n, dtype=torch.int32, device="cuda")
    count = torch.zeros(1, dtype=torch.int64, device="cuda")
    ws = torch.zeros(am.encode_workspace_bytes(n), dtype=torch.uint8, device="cuda")
    for step in range(5):
        g = (rng.standard_normal(n) * 1e-3).astype(np.float32)
        r, ref_w, ref_c = oracle.grad_threshold_encode(g, r, tau)
        am.grad_threshold_encode(to_dev(g), rd, tau, words, count, ws)
        c = int(count.cpu()[0])
        assert c == ref_c, step
        np.testing.assert_array_equal(_bits32(rd.cpu().numpy()), _bits32(r))
        np.testing.assert_array_equal(words.cpu().numpy().view(np.uint32)[:c], ref_w)


def test_encode_workspace_reused_across_sizes():
    # one workspace serves calls of different sizes in any order: what a
    # larger call leaves in the scratch never reaches a smaller one
    rng = np.random.default_rng(17)
    tau = np.float32(1e-4)
    nmax = 24_145_848
    ws = torch.zeros(am.encode_workspace_bytes(nmax), dtype=torch.uint8, device="cuda")
    words = torch.zeros(nmax, dtype=torch.int32, device="cuda")
    count = torch.zeros(1, dtype=torch.int64, device="cuda")
    for n in (1_000_003, 5_000, nmax, 40_000, 1_000_003):
        g = (rng.standard_normal(n) * 1e-4).astype(np.float32)
        r = (rng.standard_normal(n) * 5e-5).astype(np.float32)
        ref_r, ref_w, ref_c = oracle.grad_threshold_encode(g, r, tau)
        rd = to_dev(r)
        am.grad_threshold_encode(to_dev(g), rd, tau, words[:n], count, ws)
        c = int(count.cpu()[0])
        assert c == ref_c, n
        np.testing.assert_array_equal(_bits32(rd.cpu().numpy()), _bits32(ref_r))
        np.testing.assert_array_equal(words[:c].cpu().numpy().view(np.uint32), ref_w)


@pytest.mark.parametrize("accumulate", [False, True])
@pytest.mark.parametrize("n", [1, 4097, 1_000_003])
def test_decode_bit_exact(n, accumulate):
    rng = np.random.default_rng(n)
    tau = np.float32(1e-3)
    g = (rng.standard_normal(n) * 1.5e-3).astype(np.float32)
    r = np.zeros(n, np.float32)
    _, ref_w, ref_c = oracle.grad_threshold_encode(g, r, tau)
    _, _, c, words, count = _encode_gpu(g, r, tau)
    base = rng.standard_normal(n).astype(np.float32)
    dense = to_dev(base) if accumulate else to_dev(np.full(n, 7.0, np.float32))
    am.grad_threshold_decode(words, count, tau, dense, accumulate=accumulate)
    ref = oracle.grad_threshold_decode(ref_w, ref_c, tau, n, dense=base, accumulate=accumulate)
    np.testing.assert_array_equal(_bits32(dense.cpu().numpy()), _bits32(ref))


def _bf16_rounding(m):
    """The library's bf16 rounding of the masters m (sgd_apply with lr 0 and
    a zero update), i.e. the copy an SGD call leaves; torch's own conversion
    differs at NaN."""
    scratch = to_dev(m.copy())
    b = torch.empty(m.shape[0], dtype=torch.bfloat16, device="cuda")
    am.sgd_apply(scratch, torch.zeros_like(scratch), 0.0, b)
    return b


@pytest.mark.parametrize("n,offset", [(1, 0), (4097, 1), (1_000_003, 0)])
@pytest.mark.parametrize("lr", [0.01, 0.0, -0.0, -0.5, float("nan"), float("inf")])
@pytest.mark.parametrize("with_bf16", [True, False])
def test_decode_sgd_matches_decode_then_sgd(n, offset, lr, with_bf16):
    """The fused pass against the two calls on the GPU (bit for bit, master
    values with NaNs and signed zeros; the learning rates that are not +0.0
    or positive and finite make it rewrite every element) and, for finite
    values, against the oracle's decode followed by its SGD.  The bf16 copies
    start as the masters' rounding, the state every SGD call leaves them in."""
    say(f"decode+sgd n={n} offset={offset} lr={lr} bf16={with_bf16}")
    rng = np.random.default_rng(n + offset)
    tau = np.float32(1e-3)
    g = (rng.standard_normal(n) * 1.5e-3).astype(np.float32)
    _, ref_w, ref_c = oracle.grad_threshold_encode(g, np.zeros(n, np.float32), tau)
    _, _, c, words, count = _encode_gpu(g, np.zeros(n, np.float32), tau)
    m0 = rng.standard_normal(n + offset).astype(np.float32)
    special = np.array([0.0, -0.0, 1e-40, -3e38, np.nan], np.float32)
    m0[offset:offset + min(5, n)] = special[:min(5, n)]
    lr32 = np.float32(lr)
    fused = to_dev(m0)
    two = to_dev(m0)
    fb = _bf16_rounding(m0) if with_bf16 else None
    tb = _bf16_rounding(m0) if with_bf16 else None
    am.grad_threshold_decode_sgd(words, count, tau, fused[offset:], lr32,
                                 fb[offset:] if with_bf16 else None)
    dense = torch.full((n,), 7.0, dtype=torch.float32, device="cuda")
    am.grad_threshold_decode(words, count, tau, dense)
    am.sgd_apply(two[offset:], dense, lr32, tb[offset:] if with_bf16 else None)
    np.testing.assert_array_equal(_bits32(fused.cpu().numpy()), _bits32(two.cpu().numpy()))
    if with_bf16:
        np.testing.assert_array_equal(fb.cpu().view(torch.int16).numpy(), tb.cpu().view(torch.int16).numpy())
    if np.isfinite(lr32):
        finite = np.isfinite(m0[offset:])
        u = oracle.grad_threshold_decode(ref_w, ref_c, tau, n)
        ref_m, ref_b = oracle.sgd_apply(m0[offset:], u, lr32)
        got = fused.cpu().numpy()[offset:]
        np.testing.assert_array_equal(_bits32(got[finite]), _bits32(ref_m[finite]))
        if with_bf16:
            got_b = fb.cpu().view(torch.int16).numpy().view(np.uint16)[offset:]
            np.testing.assert_array_equal(got_b[finite], ref_b[finite])


@pytest.mark.parametrize("lr", [0.01, -0.5])
def test_decode_sgd_touches_only_named_elements(lr):
    """With lr +0.0 or positive and finite only the elements a word names are
    written (master and bf16 copy); every other element keeps both, here a
    bf16 sentinel that is not the master's rounding.  With any other lr
    every element is rewritten, as decode then SGD would."""
    n = 300_001
    rng = np.random.default_rng(11)
    tau = np.float32(1e-3)
    g = (rng.standard_normal(n) * 1.2e-3).astype(np.float32)
    _, ref_w, ref_c = oracle.grad_threshold_encode(g, np.zeros(n, np.float32), tau)
    _, _, c, words, count = _encode_gpu(g, np.zeros(n, np.float32), tau)
    assert c == ref_c and 0 < c < n
    m0 = rng.standard_normal(n).astype(np.float32)
    master = to_dev(m0)
    wb = torch.full((n,), 0x1234, dtype=torch.int16, device="cuda").view(torch.bfloat16)
    am.grad_threshold_decode_sgd(words, count, tau, master, np.float32(lr), wb)
    u = oracle.grad_threshold_decode(ref_w, ref_c, tau, n)
    ref_m, ref_b = oracle.sgd_apply(m0, u, np.float32(lr))
    named = np.zeros(n, bool)
    named[(ref_w[:ref_c] >> 1).astype(np.int64)] = True
    got_m = master.cpu().numpy()
    got_b = wb.cpu().view(torch.int16).numpy().view(np.uint16)
    np.testing.assert_array_equal(_bits32(got_m), _bits32(ref_m))
    np.testing.assert_array_equal(got_b[named], ref_b[named])
    if lr > 0:
        assert np.all(got_b[~named] == 0x1234)
        np.testing.assert_array_equal(_bits32(got_m[~named]), _bits32(m0[~named]))
    else:
        np.testing.assert_array_equal(got_b, ref_b)


def test_decode_sgd_count_clamped_to_capacity():
    """A device count above the words' capacity is clamped, as in decode."""
    n = 50_000
    rng = np.random.default_rng(3)
    tau = np.float32(1e-3)
    g = (rng.standard_normal(n) * 1.5e-3).astype(np.float32)
    _, _, c, words, count = _encode_gpu(g, np.zeros(n, np.float32), tau)
    cap = max(1, c // 2)
    part = words[:cap].clone()
    big = torch.tensor([c + 1000], dtype=torch.int64, device="cuda")
    m0 = rng.standard_normal(n).astype(np.float32)
    fused, two = to_dev(m0), to_dev(m0)
    am.grad_threshold_decode_sgd(part, big, tau, fused, 0.01)
    dense = torch.zeros(n, dtype=torch.float32, device="cuda")
    am.grad_threshold_decode(part, big, tau, dense)
    am.sgd_apply(two, dense, 0.01)
    np.testing.assert_array_equal(_bits32(fused.cpu().numpy()), _bits32(two.cpu().numpy()))


def _ce_case(N, C, K, seed, empty_slots=False, dup=False, mask=False):
    rng = np.random.default_rng(seed)
    z = (rng.standard_normal((N, C)) * 3).astype(np.float32)
    idx = np.stack([rng.choice(C, K, replace=False) for _ in range(N)]).astype(np.int32)
    prob = (rng.dirichlet(np.full(K, 0.3), size=N) * 0.95).astype(np.float32)
    if empty_slots and K > 1:
        idx[::3, -1] = -1
    if dup and K > 1:
        idx[::5, 1] = idx[::5, 0]
    m = (rng.random(N) > 0.3).astype(np.uint8) if mask else None
    return z, idx, prob, m


@pytest.mark.parametrize("N,C,K,opts", [
    (1, 4, 1, {}), (37, 500, 5, {"empty_slots": True}), (1000, 3000, 20, {"dup": True}),
    (130, 8192, 20, {"mask": True}), (257, 6000, 1, {}), (64, 260, 3, {"mask": True, "empty_slots": True}),
    (50, 512, 100, {"empty_slots": True, "dup": True}),
])
@pytest.mark.parametrize("dz_bf16", [False, True])
@pytest.mark.parametrize("reduction", [am.MEAN_VALID, am.SUM])
def test_soft_ce_matches_oracle(N, C, K, opts, dz_bf16, reduction):
    say(f"soft_ce N={N} C={C} K={K} {opts} bf16={dz_bf16} red={reduction}")
    z, idx, prob, m = _ce_case(N, C, K, seed=N + C, **opts)
    ref_loss, ref_dz = oracle.sparse_soft_ce(z, idx, prob, m, reduction)
    dz = torch.empty((N, C), dtype=torch.bfloat16 if dz_bf16 else torch.float32, device="cuda")
    loss = torch.zeros(1, dtype=torch.float32, device="cuda")
    ws = torch.empty(am.ce_workspace_bytes(N), dtype=torch.uint8, device="cuda")
    am.sparse_soft_ce(to_dev(z), to_dev(idx), to_dev(prob), loss, dz, ws,
                      mask=to_dev(m) if m is not None else None, reduction=reduction)
    got_loss = float(loss.cpu()[0])
    got_dz = dz.float().cpu().numpy()
    assert abs(got_loss - ref_loss) <= 1e-5 * abs(ref_loss) + 1e-7
    tol = 4e-3 if dz_bf16 else 1e-5
    assert_close("dlogits", got_dz, ref_dz, tol)
    if m is not None:
        assert np.all(got_dz[m == 0] == 0.0)


def test_soft_ce_masked_rows_ignore_their_logits():
    # (the kernel reads a row's mask before its logits and loads no logit of
    # a masked row; here the masked rows hold NaN, which must not reach the
    # loss or any gradient row)
    N, C, K = 40, 512, 4
    z, idx, prob, _ = _ce_case(N, C, K, seed=3)
    m = np.ones(N, np.uint8)
    m[5:9] = 0
    z_poison = z.copy()
    z_poison[5:9] = np.nan
    ref_loss, ref_dz = oracle.sparse_soft_ce(z, idx, prob, m)
    dz = torch.empty((N, C), dtype=torch.float32, device="cuda")
    loss = torch.zeros(1, dtype=torch.float32, device="cuda")
    ws = torch.empty(am.ce_workspace_bytes(N), dtype=torch.uint8, device="cuda")
    am.sparse_soft_ce(to_dev(z_poison), to_dev(idx), to_dev(prob), loss, dz, ws, mask=to_dev(m))
    assert np.isfinite(float(loss.cpu()[0]))
    assert abs(float(loss.cpu()[0]) - ref_loss) <= 1e-5 * abs(ref_loss)
    assert np.all(np.isfinite(dz.cpu().numpy()))


@pytest.mark.parametrize("bad", [3000, -2])
def test_soft_ce_debug_mode_rejects_out_of_range_indices(bad, monkeypatch):
    # AM_DEBUG=1: the call synchronises, finds the index outside [-1, C) and
    # returns AM_EINVAL with nothing enqueued; without it the index is an
    # empty slot
    N, C, K = 64, 3000, 20
    z, idx, prob, _ = _ce_case(N, C, K, seed=12)
    idx[37, 11] = bad
    dz = torch.full((N, C), 5.0, dtype=torch.float32, device="cuda")
    loss = torch.full((1,), 5.0, dtype=torch.float32, device="cuda")
    ws = torch.empty(am.ce_workspace_bytes(N), dtype=torch.uint8, device="cuda")
    args = (to_dev(z), to_dev(idx), to_dev(prob), loss, dz, ws)
    monkeypatch.setenv("AM_DEBUG", "1")
    with pytest.raises(am.AmError) as ei:
        am.sparse_soft_ce(*args)
    assert ei.value.status == am.EINVAL
    assert "row 37, slot 11" in str(ei.value)
    torch.cuda.synchronize()
    assert float(loss.cpu()[0]) == 5.0 and bool(torch.all(dz == 5.0))
    monkeypatch.delenv("AM_DEBUG")
    am.sparse_soft_ce(*args)
    ref_loss, ref_dz = oracle.sparse_soft_ce(z, np.where((idx >= 0) & (idx < C), idx, -1), prob)
    assert abs(float(loss.cpu()[0]) - ref_loss) <= 1e-5 * abs(ref_loss)
    assert_close("dlogits", dz.cpu().numpy(), ref_dz, 1e-5)
