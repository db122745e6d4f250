"""Blockwise model update filtering with Nesterov block momentum (BMUF-NBM),
the global step that ends every block of local SGD (§VI-B, eqs. (2)-(6)).

TEST INFRASTRUCTURE ONLY (see the package docstring).

Each of N workers trains its own copy W^i of the model with mini-batch SGD
for a block of mini-batches; the global model W_g then moves as follows,
written in the paper's notation:

    (2)  Wbar(t)  = (1/N) sum_i W(t)^i             model average
    (3)  G(t)     = Wbar(t) - W_g(t-1)             block-level update
    (4)  Delta(t) = eta_t Delta(t-1) + zeta_t G(t) block momentum
    (5)  W_g(t)   = W_g(t-1) + Delta(t) + eta_{t+1} Delta(t)
                                                   Nesterov look-ahead
    (6)  zeta / (N (1 - eta)) = C, C >= 1          how eta and zeta are set

(the paper's numbering: its eq. (1) is the decoding rule of the recogniser)

Readings (the paper gives the equations, not their arithmetic):
  * eq. (5) is taken literally, as printed: W_g(t) is the model broadcast to
    the workers for the next block, one line that adds Delta(t) and the
    look-ahead eta_{t+1} Delta(t) to W_g(t-1);
  * the model average may arrive as the N models (one GPU holding them) or
    already summed by an all-reduce: ``count`` addends are summed and the sum
    is divided by ``workers``;
  * W_g and Delta are fp32 state; each step evaluates (2)-(5) in fp64 from the
    fp32 inputs, in the order written (the sum of (2) left to right over the
    addends, then the division; (4) and (5) left to right with no fused
    multiply-add), and rounds once to fp32 per output;
  * the workers restart from W_g(t); its bf16 working copy is the
    round-to-nearest-even image of the new fp32 value.
"""

import numpy as np

from .numerics import bf16_bits


def bmuf_zeta(C, workers, eta):
    """Block learning rate from eq. (6): zeta = C N (1 - eta)."""
    return float(C) * float(workers) * (1.0 - float(eta))


def bmuf_block_update(models, workers, global_w, delta, eta, eta_next, zeta):
    """One BMUF-NBM step.

    models   [count][n] fp32: the addends of the model average (the N local
             models, or one all-reduced sum)
    workers  N, the divisor of the model average
    global_w W_g(t-1) [n] fp32;  delta Delta(t-1) [n] fp32
    eta, eta_next, zeta: eta_t, eta_{t+1}, zeta_t (fp32 scalars)
    Returns (W_g(t) fp32, Delta(t) fp32, bf16 bits of W_g(t)).
    """
    m = np.asarray(models, dtype=np.float32)
    if m.ndim == 1:
        m = m[None, :]
    wg = np.asarray(global_w, dtype=np.float32).astype(np.float64)
    d0 = np.asarray(delta, dtype=np.float32).astype(np.float64)
    assert m.shape[1] == wg.shape[0] == d0.shape[0] and workers >= 1
    eta = np.float64(np.float32(eta))
    eta_next = np.float64(np.float32(eta_next))
    zeta = np.float64(np.float32(zeta))
    s = np.zeros_like(wg)
    for i in range(m.shape[0]):                    # (2): fixed order
        s = s + m[i].astype(np.float64)
    wbar = s / np.float64(workers)
    g = wbar - wg                                  # (3)
    d = eta * d0 + zeta * g                        # (4)
    new_w = (wg + d) + eta_next * d                # (5)
    new_w32 = new_w.astype(np.float32)
    return new_w32, d.astype(np.float32), bf16_bits(new_w32)
