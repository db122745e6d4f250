"""One GPU's student training step: buffers plus the C-ABI launch sequence.

forward (lstm_am_forward) -> loss and logit gradient (sparse_soft_ce) ->
BPTT (lstm_am_backward) -> [threshold encode of the gradient with residual
error feedback -> decode] -> SGD on the fp32 master weights with a fresh bf16
copy (with threshold compression, decode and SGD run as one pass:
grad_threshold_decode_sgd).  Every step runs on the current HIP stream without host
synchronisation; this module only owns buffers and orders the calls.

A recurrence whose step barrier timed out (its workgroups were not all
resident, or the device stalled) leaves the pass invalid: lstm_am_backward
then writes a zero gradient on the device, so a step that is encoded and
applied before anyone looks adds nothing to the residual or the weights.
check() synchronises and raises for such a pass; call it before relying on
the loss or logits of a step.
"""

import torch

from . import binding as am


class StudentStep:
    def __init__(self, model: am.Model, T, B, K, lengths=None, lr=0.01, tau=1e-4, gtc=True,
                 device="cuda"):
        self.model, self.T, self.B, self.K = model, T, B, K
        self.lengths = None if lengths is None else [int(v) for v in lengths]
        self.N = T * B if lengths is None else int(sum(self.lengths))
        self.lr, self.tau, self.gtc = lr, tau, gtc
        self.n = am.param_count(model)
        dev = torch.device(device)
        f32 = torch.float32
        self.bf16 = model.dtype == am.BF16
        self.master = torch.zeros(self.n, dtype=f32, device=dev)
        self.weights = torch.zeros(self.n, dtype=torch.bfloat16, device=dev) if self.bf16 else None
        self.grads = torch.zeros(self.n, dtype=f32, device=dev)
        self.residual = torch.zeros(self.n, dtype=f32, device=dev)
        self.words = torch.zeros(self.n, dtype=torch.int32, device=dev)
        self.count = torch.zeros(1, dtype=torch.int64, device=dev)
        self.x = torch.zeros((self.N, model.input_dim), dtype=model.torch_dtype, device=dev)
        self.idx = torch.zeros((self.N, K), dtype=torch.int32, device=dev)
        self.prob = torch.zeros((self.N, K), dtype=f32, device=dev)
        self.logits = torch.zeros((self.N, model.classes), dtype=f32, device=dev)
        self.dlogits = torch.zeros((self.N, model.classes), dtype=model.torch_dtype, device=dev)
        self.loss = torch.zeros(1, dtype=f32, device=dev)
        self.ws = torch.zeros(am.workspace_bytes(model, T, B, self.N), dtype=torch.uint8, device=dev)
        self.ce_ws = torch.zeros(am.ce_workspace_bytes(self.N), dtype=torch.uint8, device=dev)
        self.enc_ws = torch.zeros(am.encode_workspace_bytes(self.n), dtype=torch.uint8, device=dev)

    @property
    def params(self):
        """The parameter copy the kernels read (bf16 working copy or fp32)."""
        return self.weights if self.bf16 else self.master

    def load_params(self, master):
        self.master.copy_(torch.as_tensor(master, dtype=torch.float32))
        if self.bf16:
            am.cast_f32_to_bf16(self.master, self.weights)

    def load_batch(self, x, idx, prob):
        x = torch.as_tensor(x, dtype=torch.float32)
        if self.bf16:
            xf = x.to(self.x.device)
            am.cast_f32_to_bf16(xf, self.x)
        else:
            self.x.copy_(x)
        self.idx.copy_(torch.as_tensor(idx, dtype=torch.int32))
        self.prob.copy_(torch.as_tensor(prob, dtype=torch.float32))

    def forward(self):
        am.lstm_am_forward(self.model, self.params, self.x, self.T, self.B, self.logits, self.ws,
                           lengths=self.lengths)

    def loss_and_grad(self):
        am.sparse_soft_ce(self.logits, self.idx, self.prob, self.loss, self.dlogits, self.ce_ws)

    def backward(self):
        am.lstm_am_backward(self.model, self.params, self.x, self.T, self.B, self.dlogits,
                            self.ws, self.grads, lengths=self.lengths)

    def apply(self):
        if self.gtc:
            am.grad_threshold_encode(self.grads, self.residual, self.tau, self.words, self.count,
                                     self.enc_ws)
            # decode + SGD in one pass (the same bits as the two calls)
            am.grad_threshold_decode_sgd(self.words, self.count, self.tau, self.master, self.lr,
                                         self.weights)
        else:
            am.sgd_apply(self.master, self.grads, self.lr, self.weights)

    def check(self):
        """Synchronise; raise if a recurrence step barrier of the last pass
        timed out (the pass's outputs are then invalid)."""
        am.workspace_check(self.ws)

    def step(self):
        self.forward()
        self.loss_and_grad()
        self.backward()
        self.apply()
