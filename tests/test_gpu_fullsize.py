"""GPU parity at the full workload sizes, in the launch configuration the
benchmark times.  The oracle cannot run a whole 16k-frame batch in seconds,
so these tests use properties that hold at any size:

* chunks (sequences) are independent, so the logits of a few sampled chunks
  must equal the oracle's forward on those chunks alone;
* the gradient is linear in dlogits, so a backward whose dlogits are zero
  outside the sampled chunks must equal the oracle's backward on those chunks;
* the soft-target CE is row-wise, so it is checked on every row;
* the quantiser is checked bit for bit on the whole 24,145,848-element
  gradient at every one of 100 consecutive steps.
"""

import numpy as np
import pytest
import torch

import oracle
from paper_1904_10584_amd import binding as am
from paper_1904_10584_amd import synth, trainer
from tests.gpu_util import assert_close, check_grads, say

pytestmark = pytest.mark.gpu

BF16_TOL = 2e-2


def _setup(name, seed_offset=0):
    w = synth.WORKLOADS[name]
    dims = oracle.ModelDims(w["layers"], w["input_dim"], w["hidden"], w["classes"])
    lengths = None
    T = w["T"]
    if "len_lo" in w:
        lengths = synth.utterance_lengths(w["B"], w["len_lo"], w["len_hi"])
        T = int(lengths[0])
    m = am.Model(dims.layers, dims.input_dim, dims.hidden, dims.classes, am.BF16)
    st = trainer.StudentStep(m, T, w["B"], w["K"], lengths=lengths, lr=w["lr"], tau=w["tau"])
    master = synth.init_params(st.n, dims.hidden)
    x = synth.features(st.N, dims.input_dim)
    idx, prob = synth.teacher_targets(st.N, dims.classes, w["K"], w["mass"],
                                      one_hot_frac=w.get("one_hot_frac", 0.0))
    st.load_params(torch.from_numpy(master).cuda())
    st.load_batch(torch.from_numpy(x).cuda(), torch.from_numpy(idx).cuda(),
                  torch.from_numpy(prob).cuda())
    return w, dims, st, master, x, idx, prob, T, lengths


def _rows_of(b, T, B, lengths):
    counts, offs = oracle.batch_schedule(T, B, lengths)
    L = T if lengths is None else int(lengths[b])
    return np.array([int(offs[t]) + b for t in range(L)], dtype=np.int64)


def one_per_block(B, block=16):
    """One sequence from every block of `block` consecutive sequences (the
    recurrence kernels serve the batch in such blocks, spread over the XCDs),
    at a position that rotates with the block: sequence block * k + k % block."""
    return [block * k + k % block for k in range((B + block - 1) // block)]


def _sampled_check(name, sample):
    """Logits of every sampled sequence against the oracle's forward of the
    sampled sequences alone (one oracle batch), the CE on every row, and the
    gradient of a backward whose dlogits vanish outside the sampled
    sequences against the oracle's backward of those sequences."""
    w, dims, st, master, x, idx, prob, T, lengths = _setup(name)
    say(f"{name}: N={st.N} frames, sampled sequences {sample}")
    st.forward()
    st.loss_and_grad()
    torch.cuda.synchronize()
    logits = st.logits.cpu().numpy()
    dz_gpu = st.dlogits.float().cpu().numpy()
    loss_gpu = float(st.loss.cpu()[0])

    # every row of the CE, against the oracle on the GPU's own logits (the
    # bf16 dlogits carry a rounding of at most 2^-9 relative)
    ref_loss, ref_dz = oracle.sparse_soft_ce(logits, idx, prob)
    assert abs(loss_gpu - ref_loss) <= 1e-5 * abs(ref_loss)
    assert_close("dlogits(all rows)", dz_gpu, ref_dz, 4e-3)

    # the sampled sequences as one oracle batch: packed time-major rows of
    # the sample (sorted lengths stay non-increasing in sample order)
    sample = sorted(sample)
    seq_rows = [_rows_of(b, T, w["B"], lengths) for b in sample]
    S = len(sample)
    s_len = np.array([r.shape[0] for r in seq_rows], np.int32)
    Ts = int(s_len.max())
    s_lengths = None if lengths is None else s_len
    counts, offs = oracle.batch_schedule(Ts, S, s_lengths)
    src = np.empty(int(offs[-1]), np.int64)  # packed sample row -> batch row
    for t in range(Ts):
        for i in range(int(counts[t])):
            src[int(offs[t]) + i] = seq_rows[i][t]

    # backward restricted to the sampled sequences
    dz_sub = np.zeros_like(dz_gpu)
    dz_sub[src] = dz_gpu[src]
    st.dlogits.copy_(torch.from_numpy(dz_sub).to(torch.bfloat16).cuda())
    st.backward()
    st.check()
    torch.cuda.synchronize()
    grads = st.grads.cpu().numpy()

    p = oracle.bf16_round(master)
    lg, cache = oracle.lstm_am_forward(p, dims, oracle.bf16_round(x[src]), Ts, S, s_lengths)
    worst = 0.0
    for i, b in enumerate(sample):
        mine = np.array([int(offs[t]) + i for t in range(int(s_len[i]))], np.int64)
        _, mr = assert_close(f"logits(seq {b})", logits[seq_rows[i]], lg[mine], BF16_TOL)
        worst = max(worst, mr)
    ref_grads = oracle.lstm_am_backward(p, dims, cache, dz_gpu[src].astype(np.float64))
    l2, mr = check_grads(grads, ref_grads, dims, BF16_TOL)
    say(f"  logits: max element ratio {worst:.2e}; gradients: max rel L2 {l2:.2e}, "
        f"max element ratio {mr:.2e}")


@pytest.mark.timeout(300)
@pytest.mark.parametrize("exchange", ["auto", "fenced"])
def test_paper_scale_sampled_chunks(exchange, monkeypatch):
    # 256 chunks: 16 blocks of 16 sequences, two per XCD; one chunk of each.
    # "fenced" forces the XCD-local recurrences onto the exchange with
    # release/acquire fences that a block spanning XCDs would take.
    if exchange == "fenced":
        monkeypatch.setenv("AM_XCD_FENCED", "1")
    else:
        monkeypatch.delenv("AM_XCD_FENCED", raising=False)
    _sampled_check("paper-5x768", one_per_block(256))


@pytest.mark.timeout(300)
def test_wide_sampled_chunks():
    # 512 chunks: one of each 16-sequence block
    _sampled_check("wide-5x1536", one_per_block(512))


@pytest.mark.timeout(300)
def test_variable_length_sampled_sequences():
    # 128 utterances: 8 blocks of 16, one per XCD; one utterance of each
    _sampled_check("varlen-5x768", one_per_block(128))


@pytest.mark.timeout(600)
def test_threshold_compression_100_steps_bit_exact():
    # 100 consecutive training steps of the paper-scale model with GTC; the
    # GPU's fp32 gradient of each step is fed to the oracle quantiser, whose
    # residual, words and count must match the GPU's bit for bit every step.
    w, dims, st, master, x, idx, prob, T, lengths = _setup("paper-5x768")
    tau = np.float32(w["tau"])
    r_ref = np.zeros(st.n, np.float32)
    say(f"gtc 100 steps, n={st.n}")
    for step in range(100):
        check_sgd = step in (0, 57, 99)
        if check_sgd:
            master_before = st.master.cpu().numpy()
        st.forward()
        st.loss_and_grad()
        st.backward()
        st.check()
        torch.cuda.synchronize()
        g = st.grads.cpu().numpy()
        st.apply()
        torch.cuda.synchronize()
        r_ref, w_ref, c_ref = oracle.grad_threshold_encode(g, r_ref, tau)
        c = int(st.count.cpu()[0])
        assert c == c_ref, step
        np.testing.assert_array_equal(st.residual.cpu().numpy().view(np.uint32), r_ref.view(np.uint32))
        np.testing.assert_array_equal(st.words[:c].cpu().numpy().view(np.uint32), w_ref)
        if check_sgd:
            # the step applies decode and SGD as one pass; its master and
            # bf16 copy against the oracle's decode followed by its SGD
            u = oracle.grad_threshold_decode(w_ref, c_ref, tau, st.n)
            new_master, new_bits = oracle.sgd_apply(master_before, u, w["lr"])
            np.testing.assert_array_equal(st.master.cpu().numpy().view(np.uint32),
                                          new_master.view(np.uint32))
            np.testing.assert_array_equal(st.weights.cpu().view(torch.int16).numpy().view(np.uint16),
                                          new_bits)
        if step % 10 == 0:
            say(f"  step {step}: {c} words, loss {float(st.loss.cpu()[0]):.5f}")
