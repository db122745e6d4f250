"""Teacher target generation (§V-A, §V-C, §VII).

TEST INFRASTRUCTURE ONLY (see the package docstring).

The teacher is a stack of bidirectional LSTM layers (five, each direction of
each layer 768 cells) over the same input frames as the student, followed by
a senone layer.  For each frame it emits senone logits; only the k largest
(k = 20) are stored, and at student training time the full posterior is
rebuilt with the missing logits filled by large negative values.

Readings (the paper names the layer type and sizes only):
  * each direction is the student's LSTM cell (no peepholes, no projection,
    one bias of 4H, gates i, f, g, o); the backward direction runs over each
    sequence from its last frame to its first, from a zero state;
  * a layer's output is [h_forward, h_backward] (2H), the next layer's input;
  * flat parameters: per layer, forward Wx [4H][D_l], Wh [4H][H], b [4H],
    then the same for the backward direction (D_0 = input_dim, D_l = 2H),
    then Wo [C][2H], bo [C].  (The paper's "78 M" is not reached by this cell:
    five such layers at 768 cells with 192 inputs and 3000 or 3183 senones
    hold about 67 M parameters; the count is unpinned);
  * the k largest logits of a frame are listed in descending order, equal
    values by ascending senone index;
  * the rebuilt posterior uses a fill of -infinity, i.e. it is the softmax
    over the k stored logits (a finite large negative fill differs from it
    by about exp(fill - max)).
Arithmetic: fp64.  Batch layout: as the student's (packed time-major rows,
sequences sorted by non-increasing length).
"""

from dataclasses import dataclass

import numpy as np

from .lstm_am import batch_schedule


@dataclass(frozen=True)
class TeacherDims:
    layers: int
    input_dim: int
    hidden: int      # cells per direction
    classes: int

    def layer_input(self, l):
        return self.input_dim if l == 0 else 2 * self.hidden


def teacher_param_offsets(d: TeacherDims):
    """Start offsets: per layer Wx_f, Wh_f, b_f, Wx_b, Wh_b, b_b; then Wo, bo."""
    offs, pos, G = [], 0, 4 * d.hidden
    for l in range(d.layers):
        for _ in range(2):
            for size in (G * d.layer_input(l), G * d.hidden, G):
                offs.append(pos)
                pos += size
    offs.append(pos)
    pos += d.classes * 2 * d.hidden
    offs.append(pos)
    return offs


def teacher_param_count(d: TeacherDims):
    return teacher_param_offsets(d)[-1] + d.classes


def _unpack(params, d):
    offs = teacher_param_offsets(d)
    G, H = 4 * d.hidden, d.hidden
    p = np.asarray(params, dtype=np.float64)
    layers = []
    for l in range(d.layers):
        D = d.layer_input(l)
        dirs = []
        for k in range(2):
            o = offs[6 * l + 3 * k: 6 * l + 3 * k + 3]
            dirs.append({"Wx": p[o[0]:o[0] + G * D].reshape(G, D),
                         "Wh": p[o[1]:o[1] + G * H].reshape(G, H),
                         "b": p[o[2]:o[2] + G]})
        layers.append(dirs)
    Wo = p[offs[-2]:offs[-2] + d.classes * 2 * H].reshape(d.classes, 2 * H)
    bo = p[offs[-1]:offs[-1] + d.classes]
    return layers, Wo, bo


def _sigm(x):
    return 1.0 / (1.0 + np.exp(-x))


def _lstm_sequence(xs, p, H):
    """One direction over one sequence xs [L][D] from a zero state."""
    h, c = np.zeros(H), np.zeros(H)
    out = np.zeros((xs.shape[0], H))
    for t in range(xs.shape[0]):
        a = p["Wx"] @ xs[t] + p["Wh"] @ h + p["b"]
        i, f = _sigm(a[0:H]), _sigm(a[H:2 * H])
        g, o = np.tanh(a[2 * H:3 * H]), _sigm(a[3 * H:4 * H])
        c = f * c + i * g
        h = o * np.tanh(c)
        out[t] = h
    return out


def teacher_forward(params, dims, x, T, B, lengths=None):
    """Teacher logits [N][C] for packed frames x [N][input_dim]."""
    layers, Wo, bo = _unpack(params, dims)
    counts, offs = batch_schedule(T, B, lengths)
    N = int(offs[-1])
    lens = [T] * B if lengths is None else [int(v) for v in lengths]
    rows = [[int(offs[t]) + b for t in range(lens[b])] for b in range(B)]
    inp = np.asarray(x, dtype=np.float64)
    assert inp.shape == (N, dims.input_dim)
    H = dims.hidden
    for dirs in layers:
        out = np.zeros((N, 2 * H))
        for b in range(B):
            r = rows[b]
            if not r:
                continue
            xs = inp[r]
            out[r, :H] = _lstm_sequence(xs, dirs[0], H)
            out[r, H:] = _lstm_sequence(xs[::-1], dirs[1], H)[::-1]
        inp = out
    return inp @ Wo.T + bo


def topk_logits(z, k):
    """The k largest logits of each row, descending (ties: lower index first).
    Returns (idx int32 [N][k], val [N][k])."""
    z = np.asarray(z)
    order = np.argsort(-z, axis=1, kind="stable")[:, :k]
    return order.astype(np.int32), np.take_along_axis(z, order, axis=1)


def kbest_posteriors(val):
    """Posterior rebuilt from k stored logits with -inf fill: the softmax over
    the k values of each row, fp64."""
    v = np.asarray(val, dtype=np.float64)
    m = v.max(axis=1, keepdims=True)
    e = np.exp(v - m)
    return e / e.sum(axis=1, keepdims=True)
