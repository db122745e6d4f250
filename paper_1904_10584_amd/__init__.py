"""MI355X (gfx950) student training step of "Realizing Petabyte Scale Acoustic
Modeling": stacked-LSTM acoustic model forward/backward, sparse soft-target
cross-entropy, SGD and gradient threshold compression, as hand-written HIP
kernels behind a C ABI (``include/mi355am.h``).

Importing the package is cheap; the native library is loaded on first use by
``paper_1904_10584_amd.binding`` and its absence is an error, never a fallback.
"""

__all__ = ["binding", "synth"]
