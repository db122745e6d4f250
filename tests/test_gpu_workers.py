"""GPU parity of the per-GPU pieces of the multi-worker trainers against the
oracle, bit for bit, through the C ABI: the aggregate of several workers'
threshold-compressed updates (§VI-A) and the BMUF-NBM global step (§VI-B).
Sizes span several tiles with ragged tails, plus the full 24,145,848-element
model of the 5x768 student."""

import numpy as np
import pytest
import torch

import oracle
from paper_1904_10584_amd import binding as am
from paper_1904_10584_amd import synth
from tests.gpu_util import say, to_dev

pytestmark = pytest.mark.gpu

N_PAPER = 24_145_848


def _bits32(a):
    return np.asarray(a, np.float32).view(np.uint32)


# ---- multi-worker aggregate ---------------------------------------------------

def _worker_streams(n, S, tau, capacity, scale=1e-4, seed=6):
    """Each worker's encode (oracle, on its own gradient and residual)."""
    g = synth.worker_gradients(n, S, scale, seed=seed)
    r = synth.worker_gradients(n, S, scale * 0.5, seed=seed + 100)
    words = np.full((S, capacity), 0xFFFFFFFF, np.uint32)  # garbage past the counts
    counts = np.zeros(S, np.int64)
    for s in range(S):
        _, w, c = oracle.grad_threshold_encode(g[s], r[s], tau)
        c = min(c, capacity)
        words[s, :c] = w[:c]
        counts[s] = c
    return words, counts


def _decode_multi_gpu(words, counts, tau, n, base=None, accumulate=False):
    S = words.shape[0]
    wd = to_dev(words.view(np.int32)) if S > 0 else torch.zeros((0, 1), dtype=torch.int32, device="cuda")
    cd = to_dev(counts) if S > 0 else torch.zeros(0, dtype=torch.int64, device="cuda")
    if base is None:
        dense = torch.full((n,), 7.0, dtype=torch.float32, device="cuda")  # must be overwritten
    else:
        dense = to_dev(base.copy())
    ws = torch.zeros(max(am.decode_multi_workspace_bytes(S, n), 256), dtype=torch.uint8, device="cuda")
    am.grad_threshold_decode_multi(wd, cd, tau, dense, ws, accumulate=accumulate)
    torch.cuda.synchronize()
    return dense.cpu().numpy()


@pytest.mark.parametrize("n,S", [(1, 1), (4096, 3), (4097, 3), (250_001, 8), (1_000_003, 5)])
@pytest.mark.parametrize("accumulate", [False, True])
def test_decode_multi_bit_exact(n, S, accumulate):
    say(f"decode_multi n={n} S={S} acc={accumulate}")
    tau = np.float32(1e-4)
    words, counts = _worker_streams(n, S, tau, n)
    base = (np.random.default_rng(n).standard_normal(n) * 1e-3).astype(np.float32)
    base[::13] = -0.0
    got = _decode_multi_gpu(words, counts, tau, n, base if accumulate else None, accumulate)
    ref = oracle.grad_threshold_decode_multi(words, counts, tau, n, base, accumulate)
    np.testing.assert_array_equal(_bits32(got), _bits32(ref))


def test_decode_multi_capacity_and_counts():
    # counts beyond the capacity are clamped; a negative count is empty
    n, S, tau = 70_000, 4, np.float32(1e-4)
    words, counts = _worker_streams(n, S, tau, 9000)
    counts_dev = counts.copy()
    counts_dev[1] = 10 ** 9
    counts_dev[2] = -5
    ref_counts = counts.copy()
    ref_counts[1] = 9000
    ref_counts[2] = 0
    got = _decode_multi_gpu(words, counts_dev, tau, n)
    ref = oracle.grad_threshold_decode_multi(words, ref_counts, tau, n)
    np.testing.assert_array_equal(_bits32(got), _bits32(ref))


def test_decode_multi_no_streams():
    got = _decode_multi_gpu(np.zeros((0, 1), np.uint32), np.zeros(0, np.int64), 1e-3, 5000)
    np.testing.assert_array_equal(_bits32(got), np.zeros(5000, np.uint32))


def test_decode_multi_single_stream_matches_decode_entry():
    n, tau = 300_000, np.float32(1e-4)
    words, counts = _worker_streams(n, 1, tau, n)
    wd = to_dev(words[0].view(np.int32))
    cd = to_dev(counts[:1])
    dense = torch.full((n,), 3.0, dtype=torch.float32, device="cuda")
    am.grad_threshold_decode(wd, cd, tau, dense)
    got = _decode_multi_gpu(words, counts, tau, n)
    np.testing.assert_array_equal(_bits32(got), _bits32(dense.cpu().numpy()))


@pytest.mark.timeout(300)
def test_decode_multi_full_model_eight_workers():
    n, S, tau = N_PAPER, 8, np.float32(1e-4)
    say(f"decode_multi full size n={n} S={S}")
    words, counts = _worker_streams(n, S, tau, n, scale=2.5e-5)
    say(f"  words per worker {counts.tolist()}")
    got = _decode_multi_gpu(words, counts, tau, n)
    ref = oracle.grad_threshold_decode_multi(words, counts, tau, n)
    np.testing.assert_array_equal(_bits32(got), _bits32(ref))


# ---- BMUF-NBM -----------------------------------------------------------------

def _bmuf_case(n, N, seed=0):
    base = synth.init_params(n, 768, seed=seed)
    models = synth.worker_models(base, N, 1e-3, seed=5 + seed)
    delta = (np.random.default_rng(100 + seed).standard_normal(n) * 1e-4).astype(np.float32)
    return base, models, delta


@pytest.mark.parametrize("n,N,count", [(1, 1, 1), (4099, 3, 3), (1_000_003, 8, 8), (65_536, 8, 1)])
@pytest.mark.parametrize("outputs", [False, True])
def test_bmuf_bit_exact(n, N, count, outputs):
    say(f"bmuf n={n} N={N} count={count} outputs={outputs}")
    base, models, delta = _bmuf_case(n, N)
    if count == 1 and N > 1:  # an all-reduced sum as the single addend
        models = models.astype(np.float64).sum(axis=0).astype(np.float32)[None, :]
    eta = np.float32(0.875)
    zeta = np.float32(oracle.bmuf_zeta(1.0, N, 0.875))
    eta_next = np.float32(0.9)
    wg, dd, md = to_dev(base), to_dev(delta), to_dev(models)
    lm = torch.zeros(n, dtype=torch.float32, device="cuda") if outputs else None
    lb = torch.zeros(n, dtype=torch.bfloat16, device="cuda") if outputs else None
    am.bmuf_block_update(md, N, wg, dd, eta, eta_next, zeta, lm, lb)
    torch.cuda.synchronize()
    ref_w, ref_d, ref_b = oracle.bmuf_block_update(models, N, base, delta, eta, eta_next, zeta)
    np.testing.assert_array_equal(_bits32(wg.cpu().numpy()), _bits32(ref_w))
    np.testing.assert_array_equal(_bits32(dd.cpu().numpy()), _bits32(ref_d))
    if outputs:
        np.testing.assert_array_equal(_bits32(lm.cpu().numpy()), _bits32(ref_w))
        np.testing.assert_array_equal(lb.cpu().view(torch.int16).numpy().view(np.uint16), ref_b)


def test_bmuf_unaligned_and_aliased_restart_copy():
    # offset views (not 16-byte aligned) and the restart copy written over
    # the first addend
    n, N = 10_001, 4
    base, models, delta = _bmuf_case(n, N, seed=3)
    flat = np.concatenate([np.zeros(1, np.float32), models.ravel()])
    md_all = to_dev(flat)
    md = md_all[1:].view(N, n)
    wg_all, dd_all = to_dev(np.concatenate([[0], base]).astype(np.float32)), to_dev(np.concatenate([[0], delta]).astype(np.float32))
    wg, dd = wg_all[1:], dd_all[1:]
    am.bmuf_block_update(md, N, wg, dd, 0.5, 0.5, 1.5, local_master=md[0])
    torch.cuda.synchronize()
    ref_w, ref_d, _ = oracle.bmuf_block_update(models, N, base, delta, 0.5, 0.5, 1.5)
    np.testing.assert_array_equal(_bits32(wg.cpu().numpy()), _bits32(ref_w))
    np.testing.assert_array_equal(_bits32(dd.cpu().numpy()), _bits32(ref_d))
    np.testing.assert_array_equal(_bits32(md[0].cpu().numpy()), _bits32(ref_w))


@pytest.mark.timeout(300)
def test_bmuf_full_model_eight_workers_two_blocks():
    n, N = N_PAPER, 8
    say(f"bmuf full size n={n} N={N}")
    base, models, delta = _bmuf_case(n, N, seed=1)
    delta[:] = 0.0
    eta, zeta = 0.875, oracle.bmuf_zeta(1.0, N, 0.875)
    wg, dd, md = to_dev(base), to_dev(delta), to_dev(models)
    ref_w, ref_d = base, delta
    for blk in range(2):
        am.bmuf_block_update(md, N, wg, dd, eta, eta, zeta)
        ref_w, ref_d, _ = oracle.bmuf_block_update(models, N, ref_w, ref_d, eta, eta, zeta)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(_bits32(wg.cpu().numpy()), _bits32(ref_w))
    np.testing.assert_array_equal(_bits32(dd.cpu().numpy()), _bits32(ref_d))
