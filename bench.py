"""Benchmark of one GPU's student training step.

A step is the whole hot path on one batch: LSTM forward, sparse soft-target
cross-entropy, BPTT, threshold encode of the full gradient with residual
error feedback, decode, and SGD on the fp32 master weights with a fresh bf16
copy.  Default workload: 5 LSTM layers x 768 cells, 192-dim input, 3000
senones, 256 chunks x 64 frames, k = 20 teacher targets, bf16 weights and
activations with fp32 masters (synthetic, seeded inputs).

Prints one JSON line: frames/s over the timed steps, the roofline of the
kernel class that takes the most time (its average launch duration measured
with HIP events over the timed steps), and the CPU oracle timed on a bounded
sample of the same workload.
"""

import argparse
import hashlib
import json
import os
import sys
import time

# The CPU oracle's BLAS threads: the cores this process may run on, unless
# the environment already fixes the count (it is read when numpy loads).
AFFINITY_CORES = len(os.sched_getaffinity(0))
os.environ.setdefault("OMP_NUM_THREADS", str(AFFINITY_CORES))

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 MFMA
SAMPLE_EVERY = 7            # bracket one launch in 7 of the timed class (coprime to 5, 6, 635)
PEAK_FP32_TFLOPS = 157.3    # MI355X dense fp32 MFMA
PEAK_HBM_GBS = 8000.0       # MI355X HBM3E
METRIC = "training frames/sec on 1 MI355X (5x768 LSTM, 3000 senones); MFMA util %"


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default="paper-5x768")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-worker-kernels", action="store_true",
                    help="skip timing the side kernels (the step's HBM-bound kernels in and out of "
                         "cache, BMUF step, 8-stream aggregate, input features, target delay, teacher "
                         "target generation)")
    ap.add_argument("--cpu-chunks", type=int, default=0,
                    help="chunks the CPU oracle runs forward/backward on (0 = the whole batch)")
    ap.add_argument("--no-other-workloads", action="store_true",
                    help="skip the shorter measurement of the other workloads")
    return ap.parse_args()


def kernel_sources_digest(names):
    h = hashlib.sha256()
    for n in names:
        with open(os.path.join(ROOT, "paper_1904_10584_amd", "csrc", n), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def traffic_for(kclass, per_launch_units, workload="paper-5x768"):
    """HBM bytes per launch from a committed counter summary of this
    workload, if it still matches the kernel sources (else None)."""
    path = os.path.join(ROOT, "profiles", "counters.json")
    if not os.path.exists(path):
        return None
    with open(path) as fh:
        table = json.load(fh)
    if table.get("workload", "paper-5x768") != workload:
        return None
    ent = table.get(kclass)
    if not ent:
        return None
    if ent.get("sources_sha") != kernel_sources_digest(ent["sources"]):
        return None
    return ent["hbm_bytes_per_launch"]


def make_step(wl, am, synth, trainer):
    import torch
    w = synth.WORKLOADS[wl]
    dtype = am.BF16 if w["dtype"] == "bf16" else am.F32
    m = am.Model(w["layers"], w["input_dim"], w["hidden"], w["classes"], dtype)
    lengths = None
    if "len_lo" in w:
        lengths = synth.utterance_lengths(w["B"], w["len_lo"], w["len_hi"])
        T = int(lengths[0])
    else:
        T = w["T"]
    st = trainer.StudentStep(m, T, w["B"], w["K"], lengths=lengths, lr=w["lr"], tau=w["tau"], gtc=True)
    n = st.n
    st.load_params(torch.from_numpy(synth.init_params(n, w["hidden"])).cuda())
    x = synth.features(st.N, w["input_dim"])
    idx, prob = synth.teacher_targets(st.N, w["classes"], w["K"], w["mass"],
                                      one_hot_frac=w.get("one_hot_frac", 0.0))
    st.load_batch(torch.from_numpy(x).cuda(), torch.from_numpy(idx).cuda(),
                  torch.from_numpy(prob).cuda())
    torch.cuda.synchronize()
    return st, w, T, lengths


def step_flops(w, T, lengths):
    """Algorithmic flops of forward + backward: 6 flops per weight per frame
    (2 forward, 4 backward) except that the input gradient of layer 0 is not
    formed.  Recurrent products are skipped at each sequence's first frame
    only in the backward (no dA_{t+1}); counted as dense here."""
    L, D, H, C = w["layers"], w["input_dim"], w["hidden"], w["classes"]
    N = T * w["B"] if lengths is None else int(sum(lengths))
    G = 4 * H
    per_frame = 0
    for l in range(L):
        Dl = D if l == 0 else H
        per_frame += 2 * G * (Dl + H)              # forward products
        per_frame += 2 * G * (Dl + H)              # weight gradients
        per_frame += 2 * G * H                     # recurrent data gradient
        if l > 0:
            per_frame += 2 * G * Dl                # input data gradient
    per_frame += 3 * 2 * C * H                     # output layer fwd, dW, dH
    return per_frame * N, N


_CYCLES_PER_MS = None


def _hold_gpu(ms):
    """Keep the GPU busy for about `ms` (torch's spin kernel), so that the
    launches enqueued next wait in the queue and then run back to back: the
    events around each launch then time the GPU, not the host's launch path
    (which is longer than a small kernel)."""
    import torch
    global _CYCLES_PER_MS
    if _CYCLES_PER_MS is None:
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda._sleep(1000)
        a.record()
        torch.cuda._sleep(1_000_000)
        b.record()
        b.synchronize()
        _CYCLES_PER_MS = 1_000_000 / max(a.elapsed_time(b), 1e-3)
    torch.cuda._sleep(int(ms * _CYCLES_PER_MS))


def _hbm_entry(kt, reps):
    us = kt["ms"] * 1e3 / max(kt["launches"], 1)
    per_launch = kt["bytes"] / max(kt["launches"], 1)
    gbs = per_launch / (us * 1e-6) / 1e9
    return {"us_per_launch": round(us, 2), "algorithmic_bytes_per_launch": per_launch,
            "achieved_GBs": round(gbs, 1), "peak_GBs": PEAK_HBM_GBS,
            "frac": round(gbs / PEAK_HBM_GBS, 4), "launches": kt["launches"]}


def worker_kernels(am, n, reps):
    """Per-GPU pieces of the multi-worker trainers on the step's flat model
    (outside the timed step): the BMUF-NBM global step over 8 local models
    with the restart copies, and the aggregate of 8 workers' compressed
    updates at about a 1 % send rate.  Each launch is timed with HIP events;
    inputs stay resident in HBM (8 models = 773 MB, more than the 256 MB
    Infinity Cache)."""
    import torch
    dev = torch.device("cuda")
    gen = torch.Generator(device=dev)
    gen.manual_seed(5)
    S = 8
    out = {}
    # BMUF: N = 8 local models, eta = 0.875, zeta = C N (1 - eta) with C = 1
    base = torch.rand(n, generator=gen, device=dev) * 0.07 - 0.035
    models = base[None, :] + torch.randn((S, n), generator=gen, device=dev) * 1e-3
    wg = base.clone()
    delta = torch.zeros(n, device=dev)
    local = torch.empty(n, device=dev)
    local_bf = torch.empty(n, dtype=torch.bfloat16, device=dev)
    torch.cuda.synchronize()
    _hold_gpu(5.0)
    am.profile_begin([am.K_BMUF])
    for _ in range(reps):
        am.bmuf_block_update(models, S, wg, delta, 0.875, 0.875, 1.0, local, local_bf)
    am.profile_end()
    out["bmuf_update"] = dict(_hbm_entry(am.profile_get(am.K_BMUF), reps), workers=S,
                              bytes_per_element=4 * S + 16 + 6)
    del models, base, wg, delta, local, local_bf
    # aggregate of 8 streams: each worker's encode of N(0, sigma^2) gradients
    # with tau / sigma = 2.576 (a 1 % send rate), words [8][n]
    tau = 1e-4
    words = torch.zeros((S, n), dtype=torch.int32, device=dev)
    counts = torch.zeros(S, dtype=torch.int64, device=dev)
    ews = torch.zeros(am.encode_workspace_bytes(n), dtype=torch.uint8, device=dev)
    for s in range(S):
        g = torch.randn(n, generator=gen, device=dev) * (tau / 2.576)
        r = torch.zeros(n, device=dev)
        am.grad_threshold_encode(g, r, tau, words[s], counts[s:s + 1], ews)
    dense = torch.empty(n, device=dev)
    dws = torch.zeros(am.decode_multi_workspace_bytes(S, n), dtype=torch.uint8, device=dev)
    torch.cuda.synchronize()
    total_words = int(counts.sum())
    _hold_gpu(5.0)
    am.profile_begin([am.K_DECODE])
    for _ in range(reps):
        am.grad_threshold_decode_multi(words, counts, tau, dense, dws)
    am.profile_end()
    kt = am.profile_get(am.K_DECODE)
    # algorithmic bytes: every word read once, the dense update written once
    kt = dict(kt, bytes=(4.0 * n + 4.0 * total_words) * kt["launches"])
    out["decode_multi"] = dict(_hbm_entry(kt, reps), streams=S, words=total_words)
    return out


def hbm_kernels(am, synth, w, n, reps):
    """The step's HBM-bound kernels at the step's sizes, each timed two ways
    (HIP events around the library's launches): in a loop over the same
    buffers, and with a 1 GiB read of another buffer between launches so that
    their inputs come from HBM, not from the 256 MB Infinity Cache or the
    L2s (a read leaves those caches clean; a write would leave dirty lines
    whose write-back the timed kernel would pay).
    Algorithmic bytes: soft-target CE reads the fp32 logits and the k
    (index, probability) pairs and writes bf16 dlogits; the encoder reads g
    and r, writes r and the 2-bit codes' words (12 B per element + 4 B per
    emitted word); the decoder writes the dense update and reads the words
    (4 B per element + 4 B per word); SGD reads the master and the update
    and writes the master and its bf16 copy (14 B per element); the step's
    fused decode + SGD reads the master and the words and writes the bf16
    copy and the masters the words name (6 B per element + 8 B per word)."""
    import torch
    dev = torch.device("cuda")
    gen = torch.Generator(device=dev)
    gen.manual_seed(8)
    flush = torch.zeros(1 << 28, device=dev)  # 1 GiB

    def timed(cls, launch, count=None, word_bytes=4.0):
        # count: device word count of each launch (word_bytes per word are
        # added to the library's per-element bytes), summed on the device
        res = {}
        for mode in ("in_loop", "flushed"):
            launch()
            torch.cuda.synchronize()
            words = torch.zeros(1, dtype=torch.int64, device=dev)
            _hold_gpu(5.0)
            am.profile_begin([cls])
            for i in range(reps):
                if mode == "flushed":
                    flush.sum()
                launch()
                if count is not None:
                    words += count
            am.profile_end()
            kt = am.profile_get(cls)
            res[mode] = _hbm_entry(dict(kt, bytes=kt["bytes"] + word_bytes * float(words.item())), reps)
        return res

    out = {}
    N, C, K = w["T"] * w["B"], w["classes"], w["K"]
    idx_np, prob_np = synth.teacher_targets(N, C, K, w["mass"])
    idx = torch.from_numpy(idx_np).to(dev)
    prob = torch.from_numpy(prob_np).to(dev)
    z = torch.randn((N, C), generator=gen, device=dev) * 3.0
    dz = torch.empty((N, C), dtype=torch.bfloat16, device=dev)
    loss = torch.zeros(1, device=dev)
    cws = torch.empty(am.ce_workspace_bytes(N), dtype=torch.uint8, device=dev)
    out["soft_ce"] = dict(timed(am.K_CE, lambda: am.sparse_soft_ce(z, idx, prob, loss, dz, cws)),
                          frames=N, classes=C, k=K)
    del z, dz, idx, prob
    tau = w["tau"]
    g = torch.randn(n, generator=gen, device=dev) * 1e-3
    r = torch.zeros(n, device=dev)
    words = torch.zeros(n, dtype=torch.int32, device=dev)
    count = torch.zeros(1, dtype=torch.int64, device=dev)
    ews = torch.zeros(am.encode_workspace_bytes(n), dtype=torch.uint8, device=dev)
    out["encode"] = dict(timed(am.K_ENCODE, lambda: am.grad_threshold_encode(g, r, tau, words, count, ews),
                               count), elements=n, words_last=int(count.item()))
    dense = torch.empty(n, device=dev)
    out["decode"] = dict(timed(am.K_DECODE, lambda: am.grad_threshold_decode(words, count, tau, dense),
                               count), elements=n, words=int(count.item()))
    master = torch.randn(n, generator=gen, device=dev) * 0.03
    wbf = torch.empty(n, dtype=torch.bfloat16, device=dev)
    out["sgd"] = dict(timed(am.K_SGD, lambda: am.sgd_apply(master, g, 1e-6, wbf)), elements=n)
    # the step's decode + SGD pass over the same words: with a positive
    # learning rate only the named elements are touched, 14 bytes per word
    # (the word, the master read and stored, its bf16 copy)
    out["decode_sgd"] = dict(timed(am.K_SGD, lambda: am.grad_threshold_decode_sgd(words, count, tau, master, 1e-6, wbf),
                                   count, 14.0), elements=n, words=int(count.item()))
    del flush
    return out


def input_kernels(am, synth, w, N, reps):
    """The student's input pieces for one batch of the workload (outside the
    timed step): stacked 30 ms features from raw 10 ms log mel frames of
    every chunk (stack 3, skip 3, causal mean, global normalisation) and the
    targets delayed by a three-frame look-ahead."""
    import numpy as np
    import torch
    B, T, K = w["B"], w["T"], w["K"]
    U = np.full(B, 3 * T + 2, np.int32)
    raw = torch.from_numpy(synth.raw_logmel(U)).cuda()
    mean = torch.zeros(3 * 64, device="cuda")
    std = torch.ones(3 * 64, device="cuda")
    x = torch.empty((T * B, 3 * 64), dtype=torch.bfloat16, device="cuda")
    idx = torch.zeros((T * B, K), dtype=torch.int32, device="cuda")
    prob = torch.zeros((T * B, K), dtype=torch.float32, device="cuda")
    io, po = torch.empty_like(idx), torch.empty_like(prob)
    mo = torch.empty((T * B,), dtype=torch.uint8, device="cuda")
    torch.cuda.synchronize()
    out = {}
    _hold_gpu(5.0)
    am.profile_begin([am.K_MISC])
    for _ in range(reps):
        am.lfr_features(U, raw, mean, std, x)
    am.profile_end()
    out["lfr_features"] = dict(_hbm_entry(am.profile_get(am.K_MISC), reps), frames=T * B,
                               raw_frames=int(U.sum()))
    _hold_gpu(5.0)
    am.profile_begin([am.K_MISC])
    for _ in range(reps):
        am.delay_targets(T, B, idx, prob, io, po, mo, 3)
    am.profile_end()
    out["delay_targets"] = dict(_hbm_entry(am.profile_get(am.K_MISC), reps), rows=T * B, k=K)
    return out


def teacher_kernels(am, synth, w, reps):
    """Target generation for one batch of the workload (outside the timed
    step): the bidirectional LSTM teacher of the same depth and width as the
    student (each direction of each layer `hidden` cells), its logits' k best
    entries and the posteriors rebuilt from them."""
    import torch
    T, B, K, C = w["T"], w["B"], w["K"], w["classes"]
    m = am.Model(w["layers"], w["input_dim"], w["hidden"], C, am.BF16)
    n = am.teacher_param_count(m)
    gen = torch.Generator(device="cuda")
    gen.manual_seed(8)
    bound = 1.0 / w["hidden"] ** 0.5
    params = ((torch.rand(n, generator=gen, device="cuda") * 2 - 1) * bound).to(torch.bfloat16)
    x = torch.randn((T * B, w["input_dim"]), generator=gen, device="cuda").to(torch.bfloat16)
    logits = torch.empty((T * B, C), dtype=torch.float32, device="cuda")
    ws = torch.empty(am.teacher_workspace_bytes(m, T, B, T * B), dtype=torch.uint8, device="cuda")
    idx = torch.empty((T * B, K), dtype=torch.int32, device="cuda")
    val = torch.empty((T * B, K), dtype=torch.float32, device="cuda")
    prob = torch.empty_like(val)
    am.blstm_teacher_forward(m, params, x, T, B, logits, ws)  # warm-up
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    _hold_gpu(5.0)
    e0.record()
    for _ in range(reps):
        am.blstm_teacher_forward(m, params, x, T, B, logits, ws)
    e1.record()
    e1.synchronize()
    dt = e0.elapsed_time(e1) * 1e-3 / reps
    am.workspace_check(ws)
    out = {"teacher_forward": {"ms_per_batch": round(dt * 1e3, 3),
                               "frames_per_s": round(T * B / dt, 1),
                               "params": n, "frames": T * B}}
    _hold_gpu(5.0)
    am.profile_begin([am.K_MISC])
    for _ in range(reps):
        am.kbest_logits(logits, idx, val)
    am.profile_end()
    out["kbest_logits"] = dict(_hbm_entry(am.profile_get(am.K_MISC), reps), k=K)
    _hold_gpu(5.0)
    am.profile_begin([am.K_MISC])
    for _ in range(reps):
        am.kbest_posteriors(val, prob)
    am.profile_end()
    out["kbest_posteriors"] = dict(_hbm_entry(am.profile_get(am.K_MISC), reps), k=K)
    return out


def blas_threads():
    """Threads the oracle's BLAS actually runs with."""
    try:
        from threadpoolctl import threadpool_info
        return int(max((i.get("num_threads", 1) for i in threadpool_info()), default=1))
    except Exception:
        return 1


def cpu_oracle_step(wl, synth, S, seq_lengths=None):
    """The oracle's forward + CE + BPTT on S sequences of workload `wl` (all
    of T frames, or the given lengths); returns (seconds, frames)."""
    import numpy as np
    import oracle
    w = synth.WORKLOADS[wl]
    d = oracle.ModelDims(w["layers"], w["input_dim"], w["hidden"], w["classes"])
    n = oracle.param_count(d)
    master = synth.init_params(n, d.hidden)
    T = w["T"] if seq_lengths is None else int(seq_lengths[0])
    counts, offs = oracle.batch_schedule(T, S, seq_lengths)
    N = int(offs[-1])
    x = synth.features(N, d.input_dim)
    idx, prob = synth.teacher_targets(N, d.classes, w["K"], w["mass"],
                                      one_hot_frac=w.get("one_hot_frac", 0.0))
    bf = w["dtype"] == "bf16"
    p = oracle.bf16_round(master) if bf else master
    xe = oracle.bf16_round(x) if bf else x
    t0 = time.perf_counter()
    logits, cache = oracle.lstm_am_forward(p, d, xe, T, S, seq_lengths)
    loss, dz = oracle.sparse_soft_ce(logits, idx, prob)
    oracle.lstm_am_backward(p, d, cache, dz)
    return time.perf_counter() - t0, N


def cpu_baseline_other(synth):
    """The oracle on bounded samples of the other workloads: frames/s of the
    forward + CE + BPTT (the per-frame cost of these loops does not depend on
    the batch), and the quantiser of the 24,145,848-parameter model over 10
    consecutive steps with residual feedback (5 of them timed)."""
    import numpy as np
    import oracle
    out = {}
    for wl, S, lens in (("tiny-2x64", 16, None), ("wide-5x1536", 32, None),
                        ("varlen-5x768", 4, None)):
        if wl == "varlen-5x768":  # utterances spread over the sorted lengths
            w = synth.WORKLOADS[wl]
            all_lens = synth.utterance_lengths(w["B"], w["len_lo"], w["len_hi"])
            lens = all_lens[[0, 43, 86, 127]].astype(np.int32)
        sec, frames = cpu_oracle_step(wl, synth, S, lens)
        out[wl] = {"value": round(frames / sec, 2), "unit": "frames/s", "cores": blas_threads(),
                   "kind": "oracle",
                   "sample": f"forward+CE+BPTT of {S} sequences ({frames} frames, {sec:.1f} s)"}
    w = synth.WORKLOADS["paper-5x768"]
    n = oracle.param_count(oracle.ModelDims(w["layers"], w["input_dim"], w["hidden"], w["classes"]))
    rng = np.random.default_rng(9)
    tau = np.float32(w["tau"])
    r = np.zeros(n, np.float32)
    master = synth.init_params(n, w["hidden"])
    g = (rng.standard_normal(n) * 3e-5).astype(np.float32)
    steps, t0 = 5, time.perf_counter()
    for _ in range(steps):
        r, words, count = oracle.grad_threshold_encode(g, r, tau)
        u = oracle.grad_threshold_decode(words, count, tau, n)
        master, _ = oracle.sgd_apply(master, u, w["lr"])
    sec = (time.perf_counter() - t0) / steps
    out["gtc-100-steps"] = {"value": round(1e3 * sec, 1), "unit": "ms per quantiser step",
                            "cores": 1, "kind": "oracle",
                            "sample": (f"encode + decode + SGD of all {n} parameters, 5 of the "
                                       f"100 consecutive steps (N(0, 3e-5^2) gradients, "
                                       f"tau = 1e-4), {sec:.2f} s per step")}
    return out


def cpu_baseline(wl, synth, chunks):
    """The oracle, as it stands, on a bounded sample: forward, CE and BPTT on
    `chunks` chunks of the batch, plus encode, decode and SGD of the whole
    flat gradient; scaled to frames/s of a full step."""
    import numpy as np
    import oracle
    threads = blas_threads()
    w = synth.WORKLOADS[wl]
    d = oracle.ModelDims(w["layers"], w["input_dim"], w["hidden"], w["classes"])
    n = oracle.param_count(d)
    master = synth.init_params(n, d.hidden)
    T, B = w["T"], w["B"]
    S = B if chunks <= 0 else min(chunks, B)
    x = synth.features(T * S, d.input_dim)
    idx, prob = synth.teacher_targets(T * S, d.classes, w["K"], w["mass"])
    p = oracle.bf16_round(master) if w["dtype"] == "bf16" else master
    xe = oracle.bf16_round(x) if w["dtype"] == "bf16" else x
    t0 = time.perf_counter()
    logits, cache = oracle.lstm_am_forward(p, d, xe, T, S)
    loss, dz = oracle.sparse_soft_ce(logits, idx, prob)
    g = oracle.lstm_am_backward(p, d, cache, dz)
    t1 = time.perf_counter()
    r, words, count = oracle.grad_threshold_encode(g.astype(np.float32), np.zeros(n, np.float32), w["tau"])
    u = oracle.grad_threshold_decode(words, count, w["tau"], n)
    oracle.sgd_apply(master, u, w["lr"])
    t2 = time.perf_counter()
    step_s = (t1 - t0) * (B / S) + (t2 - t1)
    return {"value": round(T * B / step_s, 2), "unit": "frames/s", "cores": int(threads),
            "affinity_cores": AFFINITY_CORES, "kind": "oracle",
            "sample": (f"fp64 numpy oracle: forward+CE+BPTT on {S} of {B} chunks x {T} frames "
                       f"({t1 - t0:.1f} s, scaled x{B / S:g}) plus encode/decode/SGD of all "
                       f"{n} parameters ({t2 - t1:.1f} s)")}


def measure(wl, steps, warmup, am, synth, trainer):
    """One workload: warm-up steps, one recorded step with every kernel class
    (to find the class that takes the most time), then `steps` timed steps
    with that class bracketed by HIP events on its stream.  Returns the step
    time, frames/s, MFMA utilisation over the step, the roofline of the
    dominant class and the per-class milliseconds of the recorded step."""
    import torch
    st, w, T, lengths = make_step(wl, am, synth, trainer)
    for _ in range(warmup):
        st.step()
    torch.cuda.synchronize()
    classes = range(len(am.KERNEL_CLASSES))
    am.profile_begin(classes)
    st.step()
    am.profile_end()
    totals = {k: am.profile_get(k) for k in classes}
    dom = max(classes, key=lambda k: totals[k]["ms"])
    torch.cuda.synchronize()

    # one bracketed launch in SAMPLE_EVERY: each bracket costs a few µs of
    # queue time, and an interval coprime to the class's launches per step
    # visits each of its launch positions in turn
    am.profile_begin([dom], every=SAMPLE_EVERY)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        st.step()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    am.profile_end()
    st.check()  # a timed-out step barrier invalidates the measurement
    kt = am.profile_get(dom)
    ms_per_step = (t1 - t0) * 1e3 / steps
    flops, N = step_flops(w, T, lengths)
    frames_per_s = N / (ms_per_step * 1e-3)

    avg_ms = kt["ms"] / max(kt["launches"], 1)
    name = am.KERNEL_CLASSES[dom]
    hbm_classes = {am.K_CE, am.K_ENCODE, am.K_DECODE, am.K_SGD, am.K_MISC}
    bf16 = w["dtype"] == "bf16"
    peak_mfma = PEAK_BF16_TFLOPS if bf16 else PEAK_FP32_TFLOPS
    if dom in hbm_classes:
        per_launch = kt["bytes"] / max(kt["launches"], 1)
        achieved = per_launch / (avg_ms * 1e-3) / 1e9
        roof = {"bound": "hbm", "achieved": round(achieved, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s"}
    else:
        per_launch = kt["flops"] / max(kt["launches"], 1)
        achieved = per_launch / (avg_ms * 1e-3) / 1e12
        roof = {"bound": "mfma", "achieved": round(achieved, 2), "peak": peak_mfma, "unit": "TFLOP/s"}
    roof["frac"] = round(roof["achieved"] / roof["peak"], 4)
    roof["traffic"] = traffic_for(name, per_launch, wl)
    roof["kernel"] = name
    roof["launches_per_step"] = totals[dom]["launches"]
    roof["sampled_launches"] = kt["launches"]
    roof["avg_launch_us"] = round(avg_ms * 1e3, 2)
    roof["algorithmic_per_launch"] = per_launch
    # the quantiser at the step's own send rate (the recorded step's encode:
    # 12 B per element + 4 B per emitted word)
    count = int(st.count.item())
    ke = totals[am.K_ENCODE]
    enc = None
    if ke["launches"] > 0 and ke["ms"] > 0:
        ebytes = 12.0 * st.n + 4.0 * count
        egbs = ebytes / (ke["ms"] * 1e-3) / 1e9
        enc = {"send_rate": round(count / st.n, 5), "us": round(ke["ms"] * 1e3, 2),
               "algorithmic_bytes": ebytes, "achieved_GBs": round(egbs, 1),
               "frac": round(egbs / PEAK_HBM_GBS, 4)}
    res = {
        "encode_at_step_rate": enc,
        "st": st, "w": w, "T": T, "lengths": lengths, "N": N, "flops": flops, "bf16": bf16,
        "ms_per_step": ms_per_step, "frames_per_s": frames_per_s,
        "mfma_util_pct": round(100.0 * flops / (ms_per_step * 1e-3) / (peak_mfma * 1e12), 2),
        "roofline": roof,
        "kernel_ms_per_step": {am.KERNEL_CLASSES[k]: round(totals[k]["ms"], 3) for k in classes
                               if totals[k]["launches"] > 0},
    }
    return res


def main():
    args = parse()
    if args.gpus != 1:
        print(json.dumps({"error": "the training step runs on one GPU only; --gpus must be 1",
                          "n_gpus": args.gpus}))
        sys.exit(2)
    import torch
    from paper_1904_10584_amd import binding as am
    from paper_1904_10584_amd import synth, trainer

    torch.cuda.set_device(0)
    r = measure(args.workload, args.steps, args.warmup, am, synth, trainer)
    w, T, lengths, N = r["w"], r["T"], r["lengths"], r["N"]
    n = r["st"].n
    del r["st"]
    out = {
        "metric": METRIC,
        "value": round(r["frames_per_s"], 1),
        "unit": "frames/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(r["ms_per_step"], 3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if r["bf16"] else "f32",
        "data": "synthetic",
        "config": {"workload": args.workload, "layers": w["layers"], "hidden": w["hidden"],
                   "input_dim": w["input_dim"], "classes": w["classes"], "chunks": w["B"],
                   "frames_per_chunk": T if lengths is None else None,
                   "frames_per_step": N, "k": w["K"], "tau": w["tau"], "lr": w["lr"],
                   "step": "forward+soft_ce+bptt+threshold_encode+decode+sgd",
                   "parallelism": "single-gpu"},
        "mfma_util_pct": r["mfma_util_pct"],
        "step_tflop": round(r["flops"] / 1e12, 4),
        "roofline": r["roofline"],
        "kernel_ms_per_step": r["kernel_ms_per_step"],
        "encode_at_step_rate": r["encode_at_step_rate"],
    }
    torch.cuda.empty_cache()
    if not args.no_other_workloads and args.workload == "paper-5x768":
        # the other training workloads, fewer steps each (their own roofline
        # and per-class times)
        other = {}
        for wl, steps in (("wide-5x1536", 10), ("varlen-5x768", 10)):
            o = measure(wl, steps, 2, am, synth, trainer)
            del o["st"]
            other[wl] = {"value": round(o["frames_per_s"], 1), "unit": "frames/s",
                         "ms_per_step": round(o["ms_per_step"], 3), "steps": steps, "warmup": 2,
                         "frames_per_step": o["N"], "step_tflop": round(o["flops"] / 1e12, 4),
                         "mfma_util_pct": o["mfma_util_pct"], "roofline": o["roofline"],
                         "kernel_ms_per_step": o["kernel_ms_per_step"]}
            torch.cuda.empty_cache()
        out["other_workloads"] = other
    if not args.no_worker_kernels:
        out["hbm_kernels"] = hbm_kernels(am, synth, w, n, reps=10)
        out["worker_kernels"] = worker_kernels(am, n, reps=10)
        if lengths is None:
            out["input_kernels"] = input_kernels(am, synth, w, N, reps=10)
            if r["bf16"]:
                out["teacher_kernels"] = teacher_kernels(am, synth, w, reps=5)
    if not args.no_cpu_baseline and args.workload in ("paper-5x768", "tiny-2x64", "wide-5x1536"):
        out["cpu_baseline"] = cpu_baseline(args.workload, synth, args.cpu_chunks)
        if args.workload == "paper-5x768":
            out["cpu_baseline_other"] = cpu_baseline_other(synth)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
