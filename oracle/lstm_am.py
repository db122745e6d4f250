"""Student LSTM acoustic model: forward and back-propagation through time.

Plain fp64 loops over layers and time steps; one matrix product per step is
the only library primitive used.  References are to Parthasarathi et al.,
"Realizing Petabyte Scale Acoustic Modeling".

Model (§II-B, §V-A): L unidirectional LSTM layers, then a linear senone layer
whose softmax is the student's posterior.  Cell, per layer and time step t
(the standard LSTM without peepholes or projection; the paper names the layer
type and sizes only):

    a_t = Wx x_t + Wh h_{t-1} + b,        a_t split as [a_i, a_f, a_g, a_o]
    i = sigm(a_i), f = sigm(a_f), g = tanh(a_g), o = sigm(a_o)
    c_t = f * c_{t-1} + i * g
    h_t = o * tanh(c_t)

with h_{-1} = h0, c_{-1} = c0 (zero unless given).  Logits z_t = Wo h^{L-1}_t + bo.

Batch layout.  Training runs on chunks of utterances (chunked BPTT, §II-B and
§V-D): B independent sequences of up to T frames.  Sequences are sorted by
non-increasing length, so the sequences active at step t are a prefix
0..B_t-1.  Frames are packed time-major: the frame (t, b), b < B_t, is row
off_t + b, with off_t = B_0 + ... + B_{t-1}.  Padding does not exist.  With
no lengths every sequence has T frames and row = t * B + b.
"""

import numpy as np

from .layout import unpack_params


def batch_schedule(T, B, lengths=None):
    """Active-sequence counts B_t and row offsets off_t (len T+1)."""
    if lengths is None:
        counts = np.full(T, B, dtype=np.int64)
    else:
        lengths = np.asarray(lengths, dtype=np.int64)
        assert lengths.shape == (B,)
        assert np.all(lengths >= 0) and np.all(lengths <= T)
        assert np.all(np.diff(lengths) <= 0), "lengths must be non-increasing"
        counts = np.array([(lengths > t).sum() for t in range(T)], dtype=np.int64)
    offs = np.zeros(T + 1, dtype=np.int64)
    offs[1:] = np.cumsum(counts)
    return counts, offs


def _sigm(x):
    return 1.0 / (1.0 + np.exp(-x))


def lstm_am_forward(params, dims, x, T, B, lengths=None, h0=None, c0=None):
    """Forward pass.

    params : flat parameter vector (any float dtype; used as fp64)
    x      : [N][input_dim] packed frames
    h0, c0 : [L][B][H] initial states or None (zeros)
    Returns (logits [N][C] fp64, cache).  ``cache`` holds what BPTT needs and
    the final states ``hT``/``cT`` [L][B][H]: the state after each sequence's
    last frame (h0/c0 for an empty sequence).
    """
    layers, out = unpack_params(np.asarray(params, dtype=np.float64), dims)
    H = dims.hidden
    counts, offs = batch_schedule(T, B, lengths)
    N = int(offs[-1])
    x = np.asarray(x, dtype=np.float64)
    assert x.shape == (N, dims.input_dim)

    cache = {"T": T, "B": B, "counts": counts, "offs": offs, "layers": []}
    hT = np.zeros((dims.layers, B, H))
    cT = np.zeros((dims.layers, B, H))
    inp = x
    for l, p in enumerate(layers):
        h = np.zeros((B, H)) if h0 is None else np.array(h0[l], dtype=np.float64)
        c = np.zeros((B, H)) if c0 is None else np.array(c0[l], dtype=np.float64)
        Hs = np.zeros((N, H))       # h_{t-1} seen by frame row
        Cs = np.zeros((N, H))       # c_{t-1} seen by frame row
        Hout = np.zeros((N, H))
        Cout = np.zeros((N, H))
        gates = np.zeros((N, 4 * H))
        for t in range(T):
            nb = int(counts[t])
            rows = slice(int(offs[t]), int(offs[t]) + nb)
            a = inp[rows] @ p["Wx"].T + h[:nb] @ p["Wh"].T + p["b"]
            gi = _sigm(a[:, 0:H])
            gf = _sigm(a[:, H:2 * H])
            gg = np.tanh(a[:, 2 * H:3 * H])
            go = _sigm(a[:, 3 * H:4 * H])
            Hs[rows] = h[:nb]
            Cs[rows] = c[:nb]
            c_new = gf * c[:nb] + gi * gg
            h_new = go * np.tanh(c_new)
            gates[rows] = np.concatenate([gi, gf, gg, go], axis=1)
            Cout[rows] = c_new
            Hout[rows] = h_new
            c[:nb] = c_new
            h[:nb] = h_new
        hT[l] = h
        cT[l] = c
        cache["layers"].append({"X": inp, "Hs": Hs, "Cs": Cs, "H": Hout,
                                "C": Cout, "gates": gates})
        inp = Hout
    logits = inp @ out["Wo"].T + out["bo"]
    cache["hT"] = hT
    cache["cT"] = cT
    return logits, cache


def lstm_am_backward(params, dims, cache, dlogits):
    """Back-propagation through time, given dL/dlogits [N][C].

    Returns the gradient as a flat fp64 vector in the parameter layout.  The
    gradient with respect to the input frames of layer 0 is not formed.
    Chunks are independent and every chunk's state gradient starts at zero
    after its last frame (truncated BPTT within the chunk, §II-B).
    """
    params = np.asarray(params, dtype=np.float64)
    layers, out = unpack_params(params, dims)
    grad = np.zeros_like(params)
    glayers, gout = unpack_params(grad, dims)
    H = dims.hidden
    T, B = cache["T"], cache["B"]
    counts, offs = cache["counts"], cache["offs"]
    dZ = np.asarray(dlogits, dtype=np.float64)

    top = cache["layers"][-1]["H"]
    gout["Wo"][...] = dZ.T @ top
    gout["bo"][...] = dZ.sum(axis=0)
    dH = dZ @ out["Wo"]                      # gradient reaching the top layer's h

    for l in range(dims.layers - 1, -1, -1):
        p = layers[l]
        cl = cache["layers"][l]
        g = cl["gates"]
        dA = np.zeros_like(g)
        dh_next = np.zeros((B, H))            # recurrent gradient into h_t
        dc_next = np.zeros((B, H))            # gradient into c_t from step t+1
        for t in range(T - 1, -1, -1):
            nb = int(counts[t])
            rows = slice(int(offs[t]), int(offs[t]) + nb)
            gi = g[rows, 0:H]
            gf = g[rows, H:2 * H]
            gg = g[rows, 2 * H:3 * H]
            go = g[rows, 3 * H:4 * H]
            c = cl["C"][rows]
            c_prev = cl["Cs"][rows]
            tc = np.tanh(c)
            dh = dH[rows] + dh_next[:nb]
            d_o = dh * tc
            dc = dh * go * (1.0 - tc * tc) + dc_next[:nb]
            d_i = dc * gg
            d_g = dc * gi
            d_f = dc * c_prev
            da = np.concatenate([d_i * gi * (1.0 - gi),
                                 d_f * gf * (1.0 - gf),
                                 d_g * (1.0 - gg * gg),
                                 d_o * go * (1.0 - go)], axis=1)
            dA[rows] = da
            dh_next[:nb] = da @ p["Wh"]
            dc_next[:nb] = dc * gf
        glayers[l]["Wx"][...] = dA.T @ cl["X"]
        glayers[l]["Wh"][...] = dA.T @ cl["Hs"]
        glayers[l]["b"][...] = dA.sum(axis=0)
        if l > 0:
            dH = dA @ p["Wx"]
    return grad
