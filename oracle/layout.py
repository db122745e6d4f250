"""Flat parameter layout of the student LSTM acoustic model (oracle side).

The student (§II-B) is a stack of ``layers`` unidirectional LSTM layers of
``hidden`` cells over ``input_dim``-dimensional feature frames, followed by a
softmax layer over ``classes`` senones.  The paper fixes five layers of 768
cells and "about 24 M" parameters; an LSTM with no projection layer and no
peepholes, one bias vector per layer, 192-dim input and 3000 outputs has
exactly 24,145,848, which is the reading taken here.

All parameters live in one flat vector so that the whole gradient can be
quantised in a single pass (§VI-A).  Order, per layer l = 0..L-1:

    Wx_l [4H][D_l]   input weights   (D_0 = input_dim, D_l = H for l >= 1)
    Wh_l [4H][H]     recurrent weights
    b_l  [4H]        bias

then ``Wo [C][H]`` and ``bo [C]``.  Gate blocks inside every 4H axis are in the
order input, forget, cell-candidate, output (i, f, g, o).
"""

from dataclasses import dataclass

import numpy as np


@dataclass(frozen=True)
class ModelDims:
    layers: int
    input_dim: int
    hidden: int
    classes: int

    def layer_input(self, l):
        return self.input_dim if l == 0 else self.hidden


def param_offsets(d: ModelDims):
    """Offsets of every tensor in the flat vector.

    Returns a list of ``3 * layers + 2`` start offsets, in the order
    Wx_0, Wh_0, b_0, Wx_1, ..., b_{L-1}, Wo, bo.
    """
    offs = []
    pos = 0
    G = 4 * d.hidden
    for l in range(d.layers):
        for size in (G * d.layer_input(l), G * d.hidden, G):
            offs.append(pos)
            pos += size
    offs.append(pos)
    pos += d.classes * d.hidden
    offs.append(pos)
    return offs


def param_count(d: ModelDims) -> int:
    G = 4 * d.hidden
    n = 0
    for l in range(d.layers):
        n += G * d.layer_input(l) + G * d.hidden + G
    return n + d.classes * d.hidden + d.classes


def unpack_params(flat, d: ModelDims):
    """Views (no copies) of the flat vector as named 2-D/1-D tensors."""
    flat = np.asarray(flat)
    assert flat.ndim == 1 and flat.shape[0] == param_count(d)
    offs = param_offsets(d)
    G = 4 * d.hidden
    layers = []
    for l in range(d.layers):
        ox, oh, ob = offs[3 * l: 3 * l + 3]
        Dl = d.layer_input(l)
        layers.append({
            "Wx": flat[ox: ox + G * Dl].reshape(G, Dl),
            "Wh": flat[oh: oh + G * d.hidden].reshape(G, d.hidden),
            "b": flat[ob: ob + G],
        })
    oo, obo = offs[-2], offs[-1]
    out = {
        "Wo": flat[oo: oo + d.classes * d.hidden].reshape(d.classes, d.hidden),
        "bo": flat[obo: obo + d.classes],
    }
    return layers, out
