"""Pins of the oracle's teacher target generation (§V-A, §V-C): the
bidirectional LSTM against torch's bidirectional LSTM in fp64 (fixed and
variable length), the time-reversal symmetry of the two directions, the
k best logits against repeated selection of the maximum, and the rebuilt
posterior against a full softmax (k = C, and the paper's large negative
fill).  CPU only."""

import numpy as np
import pytest
import torch

import oracle
from oracle import TeacherDims, teacher_param_count, teacher_param_offsets


def _params(d, seed):
    return np.random.default_rng(seed).uniform(-0.3, 0.3, teacher_param_count(d))


def _torch_teacher(p, d, x, T, B, lengths):
    offs = teacher_param_offsets(d)
    G, H = 4 * d.hidden, d.hidden
    lstm = torch.nn.LSTM(d.input_dim, H, num_layers=d.layers, bidirectional=True, dtype=torch.float64)
    with torch.no_grad():
        for l in range(d.layers):
            D = d.layer_input(l)
            for k, suf in enumerate(("", "_reverse")):
                o = offs[6 * l + 3 * k: 6 * l + 3 * k + 3]
                getattr(lstm, f"weight_ih_l{l}{suf}").copy_(torch.from_numpy(p[o[0]:o[0] + G * D].reshape(G, D)))
                getattr(lstm, f"weight_hh_l{l}{suf}").copy_(torch.from_numpy(p[o[1]:o[1] + G * H].reshape(G, H)))
                getattr(lstm, f"bias_ih_l{l}{suf}").copy_(torch.from_numpy(p[o[2]:o[2] + G]))
                getattr(lstm, f"bias_hh_l{l}{suf}").zero_()
    Wo = torch.from_numpy(p[offs[-2]:offs[-2] + d.classes * 2 * H].reshape(d.classes, 2 * H))
    bo = torch.from_numpy(p[offs[-1]:offs[-1] + d.classes])
    counts, poffs = oracle.batch_schedule(T, B, lengths)
    lens = [T] * B if lengths is None else list(lengths)
    pad = np.zeros((T, B, d.input_dim))
    for t in range(T):
        for b in range(int(counts[t])):
            pad[t, b] = x[int(poffs[t]) + b]
    packed = torch.nn.utils.rnn.pack_padded_sequence(torch.from_numpy(pad), torch.tensor(lens))
    out, _ = lstm(packed)
    out, _ = torch.nn.utils.rnn.pad_packed_sequence(out)
    z = (out @ Wo.T + bo).detach().numpy()
    res = np.zeros((int(poffs[-1]), d.classes))
    for t in range(T):
        for b in range(int(counts[t])):
            res[int(poffs[t]) + b] = z[t, b]
    return res


@pytest.mark.parametrize("lengths", [None, [7, 7, 5, 2, 1]])
def test_matches_torch_bidirectional_lstm(lengths):
    d = TeacherDims(3, 5, 6, 9)
    T, B = 7, 5
    p = _params(d, 1)
    counts, offs = oracle.batch_schedule(T, B, lengths)
    x = np.random.default_rng(2).standard_normal((int(offs[-1]), d.input_dim))
    got = oracle.teacher_forward(p, d, x, T, B, lengths)
    np.testing.assert_allclose(got, _torch_teacher(p, d, x, T, B, lengths), rtol=1e-12, atol=1e-12)


def test_time_reversal_swaps_the_directions():
    # one layer: reversing every sequence and swapping the directions'
    # weights reverses the hidden outputs in time and swaps their halves
    d = TeacherDims(1, 4, 5, 3)
    T, B = 6, 1
    p = _params(d, 3)
    offs = teacher_param_offsets(d)
    q = p.copy()
    half = offs[3] - offs[0]
    q[offs[0]:offs[3]], q[offs[3]:offs[3] + half] = p[offs[3]:offs[3] + half], p[offs[0]:offs[3]]
    # output layer: swap the column halves of Wo
    H, C = d.hidden, d.classes
    Wo = p[offs[-2]:offs[-2] + C * 2 * H].reshape(C, 2 * H)
    q[offs[-2]:offs[-2] + C * 2 * H] = np.concatenate([Wo[:, H:], Wo[:, :H]], axis=1).ravel()
    x = np.random.default_rng(4).standard_normal((T, d.input_dim))
    a = oracle.teacher_forward(p, d, x, T, B)
    b = oracle.teacher_forward(q, d, x[::-1].copy(), T, B)
    np.testing.assert_allclose(b[::-1], a, rtol=1e-12, atol=1e-12)


def _topk_brute(z, k):
    idx = np.zeros((z.shape[0], k), np.int32)
    val = np.zeros((z.shape[0], k))
    for r in range(z.shape[0]):
        left = list(range(z.shape[1]))
        for j in range(k):
            best = left[0]
            for c in left:
                if z[r, c] > z[r, best]:
                    best = c            # strictly greater: the lower index wins ties
            idx[r, j], val[r, j] = best, z[r, best]
            left.remove(best)
    return idx, val


def test_topk_against_repeated_maximum():
    rng = np.random.default_rng(5)
    z = rng.integers(-4, 5, (40, 17)).astype(np.float64)  # many ties
    i1, v1 = oracle.topk_logits(z, 6)
    i2, v2 = _topk_brute(z, 6)
    np.testing.assert_array_equal(i1, i2)
    np.testing.assert_array_equal(v1, v2)


def test_rebuilt_posterior():
    rng = np.random.default_rng(6)
    z = rng.standard_normal((30, 50)) * 4
    # k = C: the full softmax
    _, v = oracle.topk_logits(z, 50)
    full = torch.softmax(torch.from_numpy(v), dim=1).numpy()
    np.testing.assert_allclose(oracle.kbest_posteriors(v), full, rtol=1e-13, atol=1e-15)
    # the paper's recipe: a full vector, missing logits filled with a large
    # negative value, softmax over all C
    idx, v = oracle.topk_logits(z, 8)
    filled = np.full_like(z, -1e4)
    np.put_along_axis(filled, idx, v, axis=1)
    rebuilt = torch.softmax(torch.from_numpy(filled), dim=1).numpy()
    np.testing.assert_allclose(np.take_along_axis(rebuilt, idx, axis=1), oracle.kbest_posteriors(v),
                               rtol=1e-13, atol=1e-15)
    np.testing.assert_allclose(oracle.kbest_posteriors(v).sum(axis=1), 1.0, rtol=1e-14)
    np.testing.assert_allclose(oracle.kbest_posteriors(v + 3.5), oracle.kbest_posteriors(v), rtol=1e-13)
