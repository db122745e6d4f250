"""Pins of the oracle's LSTM acoustic model against things other than itself:
central finite differences, torch.nn.LSTM in fp64 (a library routine with the
same cell), closed forms, and batch independence.  CPU only."""

import numpy as np
import pytest
import torch

import oracle
from oracle import ModelDims, param_count, unpack_params

TINY = ModelDims(layers=2, input_dim=3, hidden=4, classes=5)


def _rand_problem(d, T, B, lengths=None, seed=0, scale=0.6, with_state=False):
    rng = np.random.default_rng(seed)
    n = param_count(d)
    params = rng.uniform(-scale, scale, size=n)
    counts, offs = oracle.batch_schedule(T, B, lengths)
    N = int(offs[-1])
    x = rng.standard_normal((N, d.input_dim))
    h0 = c0 = None
    if with_state:
        h0 = rng.uniform(-0.5, 0.5, size=(d.layers, B, d.hidden))
        c0 = rng.uniform(-0.5, 0.5, size=(d.layers, B, d.hidden))
    return params, x, h0, c0, N


def test_param_count_matches_paper_model():
    # five layers of 768 cells, 192-dim input, 3000 senones: "about 24 M"
    assert param_count(ModelDims(5, 192, 768, 3000)) == 24_145_848
    assert param_count(ModelDims(2, 64, 64, 500)) == 98_548
    offs = oracle.param_offsets(ModelDims(5, 192, 768, 3000))
    assert len(offs) == 17 and offs[0] == 0
    assert offs[-1] == 24_145_848 - 3000


def _loss_of(params, d, x, T, B, lengths, h0, c0, W):
    logits, _ = oracle.lstm_am_forward(params, d, x, T, B, lengths, h0, c0)
    return float((W * logits).sum())


@pytest.mark.parametrize("lengths,with_state", [
    (None, False), (np.array([5, 3, 0]), False), (np.array([5, 5, 2]), True)])
def test_backward_matches_central_differences(lengths, with_state):
    d, T, B = TINY, 5, 3
    params, x, h0, c0, N = _rand_problem(d, T, B, lengths, seed=1, with_state=with_state)
    W = np.random.default_rng(7).standard_normal((N, d.classes))
    _, cache = oracle.lstm_am_forward(params, d, x, T, B, lengths, h0, c0)
    grad = oracle.lstm_am_backward(params, d, cache, W)
    eps = 1e-6
    fd = np.zeros_like(params)
    for i in range(params.shape[0]):
        p = params.copy()
        p[i] += eps
        lp = _loss_of(p, d, x, T, B, lengths, h0, c0, W)
        p[i] -= 2 * eps
        lm = _loss_of(p, d, x, T, B, lengths, h0, c0, W)
        fd[i] = (lp - lm) / (2 * eps)
    gl, go = unpack_params(grad, d)
    fl, fo = unpack_params(fd, d)
    pairs = [(go["Wo"], fo["Wo"]), (go["bo"], fo["bo"])]
    for a, b in zip(gl, fl):
        pairs += [(a["Wx"], b["Wx"]), (a["Wh"], b["Wh"]), (a["b"], b["b"])]
    for a, b in pairs:
        assert np.linalg.norm(a - b) <= 1e-6 * max(np.linalg.norm(b), 1e-12)


def _torch_witness(params, d, x, T, B, lengths, W):
    """Logits and d<W, logits>/dparams from torch.nn.LSTM (fp64, CPU).

    torch's LSTM uses the same cell and gate order (i, f, g, o); its second
    bias is set to zero.  Variable-length batches are run one sequence at a
    time so that no packing code is shared with the oracle."""
    layers, out = unpack_params(params, d)
    lstm = torch.nn.LSTM(d.input_dim, d.hidden, num_layers=d.layers, dtype=torch.float64)
    with torch.no_grad():
        for l, p in enumerate(layers):
            getattr(lstm, f"weight_ih_l{l}").copy_(torch.from_numpy(p["Wx"]))
            getattr(lstm, f"weight_hh_l{l}").copy_(torch.from_numpy(p["Wh"]))
            getattr(lstm, f"bias_ih_l{l}").copy_(torch.from_numpy(p["b"]))
            getattr(lstm, f"bias_hh_l{l}").zero_()
    Wo = torch.tensor(out["Wo"], requires_grad=True)
    bo = torch.tensor(out["bo"], requires_grad=True)
    counts, offs = oracle.batch_schedule(T, B, lengths)
    lens = [T] * B if lengths is None else list(lengths)
    logits = torch.zeros((int(offs[-1]), d.classes), dtype=torch.float64)
    total = 0.0
    for b in range(B):
        if lens[b] == 0:
            continue
        rows = [int(offs[t]) + b for t in range(lens[b])]
        xb = torch.from_numpy(x[rows]).unsqueeze(1)
        hb, _ = lstm(xb)
        zb = hb[:, 0, :] @ Wo.T + bo
        total = total + (torch.from_numpy(W[rows]) * zb).sum()
        logits[rows] = zb.detach()
    total.backward()
    g = np.zeros_like(params)
    gl, go = unpack_params(g, d)
    for l in range(d.layers):
        gl[l]["Wx"][...] = getattr(lstm, f"weight_ih_l{l}").grad.numpy()
        gl[l]["Wh"][...] = getattr(lstm, f"weight_hh_l{l}").grad.numpy()
        gl[l]["b"][...] = getattr(lstm, f"bias_ih_l{l}").grad.numpy()
    go["Wo"][...] = Wo.grad.numpy()
    go["bo"][...] = bo.grad.numpy()
    return logits.numpy(), g


@pytest.mark.parametrize("lengths", [None, np.array([7, 7, 4, 1])])
def test_forward_backward_match_torch_lstm(lengths):
    d = ModelDims(layers=3, input_dim=6, hidden=5, classes=7)
    T, B = 7, 4
    params, x, _, _, N = _rand_problem(d, T, B, lengths, seed=3)
    W = np.random.default_rng(11).standard_normal((N, d.classes))
    logits, cache = oracle.lstm_am_forward(params, d, x, T, B, lengths)
    grad = oracle.lstm_am_backward(params, d, cache, W)
    t_logits, t_grad = _torch_witness(params, d, x, T, B, lengths, W)
    np.testing.assert_allclose(logits, t_logits, rtol=0, atol=1e-12)
    np.testing.assert_allclose(grad, t_grad, rtol=1e-10, atol=1e-12)


def test_final_state_is_state_after_last_frame():
    d, T, B = TINY, 6, 3
    lengths = np.array([6, 4, 0])
    params, x, h0, c0, _ = _rand_problem(d, T, B, lengths, seed=5, with_state=True)
    _, cache = oracle.lstm_am_forward(params, d, x, T, B, lengths, h0, c0)
    counts, offs = oracle.batch_schedule(T, B, lengths)
    for l in range(d.layers):
        for b, L in enumerate(lengths):
            if L == 0:
                np.testing.assert_array_equal(cache["hT"][l, b], h0[l, b])
                np.testing.assert_array_equal(cache["cT"][l, b], c0[l, b])
            else:
                row = int(offs[L - 1]) + b
                np.testing.assert_array_equal(cache["hT"][l, b], cache["layers"][l]["H"][row])
                np.testing.assert_array_equal(cache["cT"][l, b], cache["layers"][l]["C"][row])


def test_zero_weights_closed_form():
    # all weights zero: every gate is 1/2 or 0, so c = h = 0 and logits = bo;
    # with bo = 0 the student posterior is uniform and the per-frame loss is
    # M_f * ln C.
    d, T, B = ModelDims(2, 8, 6, 11), 4, 3
    params = np.zeros(param_count(d))
    x = np.random.default_rng(0).standard_normal((T * B, d.input_dim))
    logits, cache = oracle.lstm_am_forward(params, d, x, T, B)
    assert np.all(logits == 0.0)
    for cl in cache["layers"]:
        assert np.all(cl["H"] == 0.0) and np.all(cl["C"] == 0.0)
    idx = np.tile(np.array([[3, 0, 9]]), (T * B, 1))
    prob = np.tile(np.array([[0.5, 0.25, 0.2]]), (T * B, 1))
    loss, dz = oracle.sparse_soft_ce(logits, idx, prob)
    assert loss == pytest.approx(0.95 * np.log(11), rel=1e-14)


def test_chunks_are_independent():
    d, T, B = TINY, 5, 4
    params, x, _, _, N = _rand_problem(d, T, B, seed=9)
    W = np.random.default_rng(2).standard_normal((N, d.classes))
    logits, cache = oracle.lstm_am_forward(params, d, x, T, B)
    grad = oracle.lstm_am_backward(params, d, cache, W)
    gsum = np.zeros_like(grad)
    for b in range(B):
        rows = [t * B + b for t in range(T)]
        lb, cb = oracle.lstm_am_forward(params, d, x[rows], T, 1)
        np.testing.assert_allclose(lb, logits[rows], rtol=0, atol=1e-14)
        gsum += oracle.lstm_am_backward(params, d, cb, W[rows])
    np.testing.assert_allclose(gsum, grad, rtol=1e-12, atol=1e-13)
