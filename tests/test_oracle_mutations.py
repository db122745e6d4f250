"""Planted mistakes: each test loads a copy of one oracle module with one
plausible error written into it (a dropped term, a wrong sign, a wrong index,
a transposed operand) and checks that an independent pin rejects it.  The
mistakes live only in these in-memory copies, on the CPU."""

import os
import types

import numpy as np
import pytest
import torch

import oracle
from oracle import ModelDims, param_count, unpack_params

ORACLE_DIR = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "oracle")


def _mutant(module_file, old, new):
    src = open(os.path.join(ORACLE_DIR, module_file)).read()
    assert src.count(old) == 1, (module_file, old)
    mod = types.ModuleType("oracle._mutant")
    mod.__package__ = "oracle"
    exec(compile(src.replace(old, new), module_file, "exec"), mod.__dict__)
    return mod


D = ModelDims(layers=2, input_dim=3, hidden=4, classes=5)


def _torch_logits_and_grad(params, x, T, B, W):
    layers, out = unpack_params(params, D)
    lstm = torch.nn.LSTM(D.input_dim, D.hidden, num_layers=D.layers, dtype=torch.float64)
    with torch.no_grad():
        for l, p in enumerate(layers):
            getattr(lstm, f"weight_ih_l{l}").copy_(torch.from_numpy(p["Wx"]))
            getattr(lstm, f"weight_hh_l{l}").copy_(torch.from_numpy(p["Wh"]))
            getattr(lstm, f"bias_ih_l{l}").copy_(torch.from_numpy(p["b"]))
            getattr(lstm, f"bias_hh_l{l}").zero_()
    Wo = torch.tensor(out["Wo"], requires_grad=True)
    bo = torch.tensor(out["bo"], requires_grad=True)
    h, _ = lstm(torch.from_numpy(x.reshape(T, B, D.input_dim)))
    z = h.reshape(T * B, D.hidden) @ Wo.T + bo
    (torch.from_numpy(W) * z).sum().backward()
    g = np.zeros_like(params)
    gl, go = unpack_params(g, D)
    for l in range(D.layers):
        gl[l]["Wx"][...] = getattr(lstm, f"weight_ih_l{l}").grad.numpy()
        gl[l]["Wh"][...] = getattr(lstm, f"weight_hh_l{l}").grad.numpy()
        gl[l]["b"][...] = getattr(lstm, f"bias_ih_l{l}").grad.numpy()
    go["Wo"][...] = Wo.grad.numpy()
    go["bo"][...] = bo.grad.numpy()
    return z.detach().numpy(), g


def _lstm_pins_pass(mod):
    """True when the module's forward/backward agree with torch.nn.LSTM."""
    T, B = 5, 3
    rng = np.random.default_rng(0)
    params = rng.uniform(-0.6, 0.6, size=param_count(D))
    x = rng.standard_normal((T * B, D.input_dim))
    W = rng.standard_normal((T * B, D.classes))
    logits, cache = mod.lstm_am_forward(params, D, x, T, B)
    grad = mod.lstm_am_backward(params, D, cache, W)
    tz, tg = _torch_logits_and_grad(params, x, T, B, W)
    return np.allclose(logits, tz, rtol=0, atol=1e-12) and np.allclose(grad, tg, rtol=1e-10, atol=1e-12)


def test_unmutated_oracle_passes_lstm_pins():
    assert _lstm_pins_pass(oracle.lstm_am)


@pytest.mark.parametrize("old,new", [
    ("c_new = gf * c[:nb] + gi * gg", "c_new = gi * c[:nb] + gf * gg"),     # gates swapped
    ("go = _sigm(a[:, 3 * H:4 * H])", "go = _sigm(a[:, 2 * H:3 * H])"),     # wrong gate slice
    ("h[:nb] @ p[\"Wh\"].T", "h[:nb] @ p[\"Wh\"][:, ::-1].T"),              # wrong index
    ("dc = dh * go * (1.0 - tc * tc) + dc_next[:nb]", "dc = dh * go * (1.0 - tc * tc)"),  # dropped term
    ("d_f = dc * c_prev", "d_f = dc * c"),                                    # wrong time index
    ("d_g * (1.0 - gg * gg)", "d_g * (1.0 + gg * gg)"),                       # wrong sign
    ("glayers[l][\"Wh\"][...] = dA.T @ cl[\"Hs\"]", "glayers[l][\"Wh\"][...] = dA.T @ cl[\"H\"]"),
    ("dh_next[:nb] = da @ p[\"Wh\"]", "dh_next[:nb] = da @ p[\"Wh\"] * 0.0"),
    ("dH = dZ @ out[\"Wo\"]", "dH = dZ @ out[\"Wo\"] * 2.0"),
])
def test_lstm_mistakes_are_caught(old, new):
    assert not _lstm_pins_pass(_mutant("lstm_am.py", old, new))


def _ce_pins_pass(mod):
    rng = np.random.default_rng(1)
    N, C = 12, 9
    z = rng.standard_normal((N, C)) * 2
    P = rng.dirichlet(np.full(C, 0.5), size=N) * 0.9
    idx = np.stack([rng.permutation(C) for _ in range(N)])
    prob = np.take_along_axis(P, idx, axis=1)
    loss, dz = mod.sparse_soft_ce(z, idx, prob)
    zt = torch.tensor(z, requires_grad=True)
    tl = torch.nn.functional.cross_entropy(zt, torch.tensor(P))
    tl.backward()
    return abs(loss - tl.item()) <= 1e-12 * abs(tl.item()) and np.allclose(dz, zt.grad.numpy(), rtol=1e-10, atol=1e-15)


def test_unmutated_oracle_passes_ce_pins():
    assert _ce_pins_pass(oracle.soft_ce)


@pytest.mark.parametrize("old,new", [
    ("dz[f] = scale[f] * (mass * q - target)", "dz[f] = scale[f] * (q - target)"),   # mass dropped
    ("lf -= p[f, j] * (z[f, c] - lse)", "lf -= p[f, j] * (z[f, c] + lse)"),          # sign
    ("lse = zmax + np.log", "lse = np.log"),                                          # max not restored
])
def test_ce_mistakes_are_caught(old, new):
    assert not _ce_pins_pass(_mutant("soft_ce.py", old, new))


def _gtc_pins_pass(mod):
    tau = np.float32(2.0 ** -10)
    rng = np.random.default_rng(2)
    n = 20000
    g = (rng.integers(-5000, 5000, n) * 2.0 ** -20).astype(np.float32)
    r = (rng.integers(-1500, 1500, n) * 2.0 ** -20).astype(np.float32)
    g[:4] = [tau, -tau, 0, 0]
    r[:4] = 0
    new_r, words, count = mod.grad_threshold_encode(g, r, tau)
    sent = mod.grad_threshold_decode(words, count, tau, n)
    conserved = np.array_equal(new_r.astype(np.float64) + sent, r.astype(np.float64) + g)
    strict = not np.any(np.isin(words >> 1, [0, 1]))
    ascending = bool(np.all(np.diff(words >> 1) > 0))
    return conserved and strict and ascending


def test_unmutated_oracle_passes_gtc_pins():
    assert _gtc_pins_pass(oracle.gtc)


@pytest.mark.parametrize("old,new", [
    ("pos = a > tau", "pos = a >= tau"),                                  # non-strict test
    ("new_r[pos] = a[pos] - tau", "new_r[pos] = a[pos] + tau"),           # wrong sign
    ("    a = r + g\n", "    a = g\n"),                                       # residual dropped
    ("value = np.where((w & np.uint32(1)) != 0, -tau, tau)", "value = np.where((w & np.uint32(1)) != 0, tau, -tau)"),
])
def test_gtc_mistakes_are_caught(old, new):
    assert not _gtc_pins_pass(_mutant("gtc.py", old, new))


# ---- BMUF and the multi-worker aggregate ------------------------------------

@pytest.mark.parametrize("old,new", [
    ("new_w = (wg + d) + eta_next * d", "new_w = (wg + d)"),               # look-ahead dropped
    ("new_w = (wg + d) + eta_next * d", "new_w = (wg + d) + eta * d"),     # wrong momentum index
    ("g = wbar - wg", "g = wg - wbar"),                                    # wrong sign of G
    ("wbar = s / np.float64(workers)", "wbar = s / np.float64(m.shape[0])"),  # averages the addends
    ("d = eta * d0 + zeta * g", "d = eta * g + zeta * g"),                 # momentum forgets Delta
])
def test_bmuf_pins_reject(old, new):
    import tests.test_oracle_bmuf as pins
    mod = _mutant("bmuf.py", old, new)
    saved = oracle.bmuf_block_update
    oracle.bmuf_block_update = mod.bmuf_block_update
    try:
        failures = 0
        for name in ("test_single_worker_without_momentum_takes_the_local_model",
                     "test_block_momentum_closed_form_over_blocks",
                     "test_look_ahead_uses_the_next_momentum",
                     "test_all_reduced_sum_gives_the_same_step"):
            try:
                getattr(pins, name)()
            except AssertionError:
                failures += 1
        for w in (2, 4, 8):
            try:
                pins.test_without_momentum_is_model_averaging(w)
            except AssertionError:
                failures += 1
        assert failures > 0, (old, new)
    finally:
        oracle.bmuf_block_update = saved


@pytest.mark.parametrize("old,new", [
    ("sign = np.where((ws & np.uint32(1)) != 0, -1, 1)", "sign = np.where((ws & np.uint32(1)) != 0, 1, -1)"),
    ("ws = w[s, :int(counts[s])]", "ws = w[s, :int(counts[s])][:-1]"),       # last word lost
    ("out[hit] = out[hit] + v[hit]", "out = out + v"),                     # touches unsent elements
])
def test_decode_multi_pins_reject(old, new):
    import tests.test_oracle_gtc as pins
    mod = _mutant("gtc.py", old, new)
    saved = oracle.grad_threshold_decode_multi
    oracle.grad_threshold_decode_multi = mod.grad_threshold_decode_multi
    try:
        failures = 0
        for call in (lambda: pins.test_decode_multi_single_stream_is_decode(False),
                     lambda: pins.test_decode_multi_single_stream_is_decode(True),
                     pins.test_decode_multi_equals_sum_of_single_decodes,
                     pins.test_decode_multi_conserves_across_workers,
                     pins.test_decode_multi_cancelling_signs):
            try:
                call()
            except AssertionError:
                failures += 1
        assert failures > 0, (old, new)
    finally:
        oracle.grad_threshold_decode_multi = saved


# ---- input features and delayed targets ---------------------------------------

@pytest.mark.parametrize("old,new", [
    ("out[t, k * D:(k + 1) * D] = raw[offset + skip * t + k]",
     "out[t, k * D:(k + 1) * D] = raw[offset + skip * t + (stack - 1 - k)]"),      # newest frame first
    ("        run = run + y[t]\n        z[t] = y[t] - run / (t + 1)",
     "        z[t] = y[t] - run / max(t, 1)\n        run = run + y[t]"),           # mean of the past only
    ("                src = int(offs[t - delay]) + b", "                src = int(offs[t - delay + 1]) + b"),  # off by one
    ("    return max(0, (U - offset - stack) // skip + 1)", "    return max(0, (U - offset + skip - 1) // skip)"),  # partial stacks
])
def test_feature_pins_reject(old, new):
    import tests.test_oracle_features as pins
    mod = _mutant("features.py", old, new)
    saved = {k: getattr(oracle, k) for k in ("lfr_stack", "lfr_frames", "causal_mean_subtract", "delay_targets")}
    for k in saved:
        setattr(oracle, k, getattr(mod, k))
    try:
        failures = 0
        calls = [lambda o=o: pins.test_stacked_layout(o) for o in (0, 1, 2)]
        calls += [lambda a=a: pins.test_frame_counts(*a) for a in ((5, 2, 1), (4, 2, 0), (2, 0, 0))]
        calls += [pins.test_causal_mean_closed_forms]
        calls += [lambda l=l, d=d: pins.test_delayed_targets(l, d) for l in (None, [9, 7, 7, 3, 2, 0]) for d in (1, 3)]
        for call in calls:
            try:
                call()
            except (AssertionError, IndexError, ValueError):
                failures += 1
        assert failures > 0, (old, new)
    finally:
        for k, v in saved.items():
            setattr(oracle, k, v)


# ---- teacher -------------------------------------------------------------------

@pytest.mark.parametrize("old,new", [
    ("out[r, H:] = _lstm_sequence(xs[::-1], dirs[1], H)[::-1]",
     "out[r, H:] = _lstm_sequence(xs[::-1], dirs[1], H)"),              # not reversed back
    ("out[r, H:] = _lstm_sequence(xs[::-1], dirs[1], H)[::-1]",
     "out[r, H:] = _lstm_sequence(xs, dirs[1], H)"),                    # backward runs forward
    ("order = np.argsort(-z, axis=1, kind=\"stable\")[:, :k]",
     "order = np.argsort(z, axis=1, kind=\"stable\")[:, ::-1][:, :k]"),  # ties: higher index first
])
def test_teacher_pins_reject(old, new):
    import tests.test_oracle_teacher as pins
    mod = _mutant("teacher.py", old, new)
    saved = (oracle.teacher_forward, oracle.topk_logits)
    oracle.teacher_forward, oracle.topk_logits = mod.teacher_forward, mod.topk_logits
    try:
        failures = 0
        for call in (lambda: pins.test_matches_torch_bidirectional_lstm(None),
                     lambda: pins.test_matches_torch_bidirectional_lstm([7, 7, 5, 2, 1]),
                     pins.test_time_reversal_swaps_the_directions,
                     pins.test_topk_against_repeated_maximum):
            try:
                call()
            except AssertionError:
                failures += 1
        assert failures > 0, (old, new)
    finally:
        oracle.teacher_forward, oracle.topk_logits = saved
