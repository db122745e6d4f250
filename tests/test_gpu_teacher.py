"""GPU parity of teacher target generation (§V-A, §V-C) against the oracle,
through the C ABI: the bidirectional LSTM teacher's logits (fp32 within
1e-4, bf16 within 2e-2; fixed and variable length, and sampled sequences of
the 5x768 teacher at full batch size), the k best logits (bit for bit on the
same logits, with ties, NaN and signed zeros) and the rebuilt posteriors."""

import numpy as np
import pytest
import torch

import oracle
from paper_1904_10584_amd import binding as am
from paper_1904_10584_amd import synth
from tests.gpu_util import assert_close, bf16_dev, say, to_dev

pytestmark = pytest.mark.gpu


def _teacher_gpu(m, master, x, T, B, lengths=None):
    bf = m.dtype == am.BF16
    params = bf16_dev(master) if bf else to_dev(master)
    xd = bf16_dev(x) if bf else to_dev(x)
    N = x.shape[0]
    logits = torch.empty((N, m.classes), dtype=torch.float32, device="cuda")
    ws = torch.empty(am.teacher_workspace_bytes(m, T, B, N), dtype=torch.uint8, device="cuda")
    am.blstm_teacher_forward(m, params, xd, T, B, logits, ws, lengths=lengths)
    am.workspace_check(ws)
    torch.cuda.synchronize()
    return logits.cpu().numpy()


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("lengths_kind", [None, "varlen"])
def test_teacher_small_matches_oracle(dtype, lengths_kind):
    d = oracle.TeacherDims(2, 64, 128, 520)
    T, B = 12, 80
    lengths = None
    if lengths_kind:
        lengths = np.sort(np.random.default_rng(1).integers(1, T + 1, B))[::-1].astype(np.int32)
    counts, offs = oracle.batch_schedule(T, B, lengths)
    N = int(offs[-1])
    n = oracle.teacher_param_count(d)
    master = synth.init_params(n, d.hidden, seed=50)
    x = synth.features(N, d.input_dim, seed=51)
    m = am.Model(d.layers, d.input_dim, d.hidden, d.classes, am.BF16 if dtype == "bf16" else am.F32)
    say(f"teacher small {dtype} {lengths_kind}")
    got = _teacher_gpu(m, master, x, T, B, lengths)
    bf = dtype == "bf16"
    p = oracle.bf16_round(master) if bf else master.astype(np.float32)
    xe = oracle.bf16_round(x) if bf else x
    ref = oracle.teacher_forward(p, d, xe, T, B, lengths)
    l2, mr = assert_close("teacher logits", got, ref, 2e-2 if bf else 1e-4)
    say(f"  rel L2 {l2:.2e}, max element ratio {mr:.2e}")


@pytest.mark.timeout(300)
def test_teacher_paper_scale_sampled_sequences():
    # 5 x 768 bidirectional teacher, 3000 senones, 256 chunks x 64 frames
    d = oracle.TeacherDims(5, 192, 768, 3000)
    T, B = 64, 256
    n = oracle.teacher_param_count(d)
    master = synth.init_params(n, d.hidden, seed=52)
    x = synth.features(T * B, d.input_dim, seed=53)
    m = am.Model(d.layers, d.input_dim, d.hidden, d.classes, am.BF16)
    say(f"teacher 5x768 n={n}")
    got = _teacher_gpu(m, master, x, T, B)
    p = oracle.bf16_round(master)
    # one sequence of every 16-sequence block (the recurrence serves the
    # batch in such blocks, two per XCD), as one oracle batch
    sample = [16 * k + k for k in range(B // 16)]
    rows = (np.arange(T)[:, None] * B + np.array(sample)[None, :]).reshape(-1)
    ref = oracle.teacher_forward(p, d, oracle.bf16_round(x[rows]), T, len(sample))
    for i, b in enumerate(sample):
        mine = np.arange(T) * len(sample) + i
        l2, mr = assert_close(f"teacher logits(seq {b})", got[rows[mine]], ref[mine], 2e-2)
        say(f"  sequence {b}: rel L2 {l2:.2e}, max element ratio {mr:.2e}")


# (C % 4 != 0 takes the kernel's 4-byte-load path, the others its 16-byte one)
@pytest.mark.parametrize("C,K", [(520, 1), (520, 20), (3000, 20), (6000, 64), (64, 64),
                                 (517, 20), (3001, 33)])
def test_kbest_logits_bit_exact(C, K):
    rng = np.random.default_rng(C + K)
    N = 1037
    z = (rng.standard_normal((N, C)) * 3).astype(np.float32)
    z[::7] = np.round(z[::7])             # many ties
    z[3, :10] = np.nan
    z[5, 1::2] = -0.0
    z[5, ::2] = 0.0
    z[9] = -np.inf
    zd = to_dev(z)
    idx = torch.empty((N, K), dtype=torch.int32, device="cuda")
    val = torch.empty((N, K), dtype=torch.float32, device="cuda")
    am.kbest_logits(zd, idx, val)
    torch.cuda.synchronize()
    ri, rv = oracle.topk_logits(z, K)
    np.testing.assert_array_equal(idx.cpu().numpy(), ri)
    np.testing.assert_array_equal(val.cpu().numpy().view(np.uint32), rv.astype(np.float32).view(np.uint32))


def test_kbest_posteriors_match_oracle():
    rng = np.random.default_rng(7)
    v = np.sort(rng.standard_normal((5000, 20)) * 4, axis=1)[:, ::-1].astype(np.float32)
    prob = torch.empty((5000, 20), dtype=torch.float32, device="cuda")
    am.kbest_posteriors(to_dev(v.copy()), prob)
    torch.cuda.synchronize()
    ref = oracle.kbest_posteriors(v)
    np.testing.assert_allclose(prob.cpu().numpy(), ref, rtol=2e-6, atol=1e-30)
