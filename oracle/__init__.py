"""CPU oracle for the per-GPU student training step.

TEST INFRASTRUCTURE ONLY.  Nothing on the product path may import, call or
execute anything in this package: it is used by ``tests/``, by the smoke check
of ``__graft_entry__`` and by the CPU-baseline leg of ``bench.py``.  It shares
no code with the HIP path (no kernels, headers, helpers, tables or generators)
and imports nothing from it.

What it computes, in the order the training step runs it
(Parthasarathi et al., "Realizing Petabyte Scale Acoustic Modeling"):

* ``lstm_am``  -- the student acoustic model: a stack of unidirectional LSTM
  layers followed by a senone output layer (§II-B; the student is the same
  network, §V-A), trained by chunked back-propagation through time (§II-B,
  §V-D).  Forward and backward are explicit loops over time in fp64.
* ``soft_ce``  -- cross-entropy between the teacher's sparse k-best posterior
  and the student's softmax (§II-C, §V-A, §V-C), with its logit gradient.
* ``sgd``      -- the local mini-batch SGD update (§VI, §VI-B) and the
  round-to-nearest-even bf16 copy of the updated fp32 master weights.
* ``gtc``      -- Gradient Threshold Compression (§VI-A): residual error
  feedback, +-tau one-bit quantisation and 32-bit index/sign packing, the
  matching decode, and the aggregate of several workers' sparse updates.
* ``bmuf``     -- the BMUF-NBM global step that ends a block of local SGD
  (§VI-B, eqs. (2)-(6)).
* ``features`` -- the student's input frames (three 10 ms frames stacked at a
  30 ms advance, causal mean subtraction, global normalisation) and the
  targets delayed by the model's look-ahead (§II-B).
* ``teacher``  -- target generation: the bidirectional LSTM teacher's logits,
  the k best logits per frame and the posterior rebuilt from them (§V-A,
  §V-C, §VII).

Floating point: the model, loss and their gradients are computed in fp64;
the quantiser and SGD use the exact fp32 operation order that the method
states (they are compared bit for bit).  Where the paper is silent the
readings are the ones listed in the design notes of this repository; each
function repeats the reading it relies on.
"""

from .layout import ModelDims, param_count, param_offsets, unpack_params
from .numerics import bf16_round, bf16_bits, bf16_bits_to_f32
from .lstm_am import batch_schedule, lstm_am_forward, lstm_am_backward
from .soft_ce import sparse_soft_ce
from .sgd import sgd_apply
from .gtc import grad_threshold_encode, grad_threshold_decode, grad_threshold_decode_multi
from .bmuf import bmuf_block_update, bmuf_zeta
from .features import (lfr_frames, lfr_stack, causal_mean_subtract, global_mvn, lfr_features,
                       delay_targets)
from .teacher import (TeacherDims, teacher_param_count, teacher_param_offsets, teacher_forward,
                      topk_logits, kbest_posteriors)

__all__ = [
    "ModelDims", "param_count", "param_offsets", "unpack_params",
    "bf16_round", "bf16_bits", "bf16_bits_to_f32",
    "batch_schedule", "lstm_am_forward", "lstm_am_backward",
    "sparse_soft_ce", "sgd_apply",
    "grad_threshold_encode", "grad_threshold_decode", "grad_threshold_decode_multi",
    "bmuf_block_update", "bmuf_zeta",
    "lfr_frames", "lfr_stack", "causal_mean_subtract", "global_mvn", "lfr_features",
    "delay_targets",
    "TeacherDims", "teacher_param_count", "teacher_param_offsets", "teacher_forward",
    "topk_logits", "kbest_posteriors",
]
