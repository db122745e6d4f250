"""Helpers for the GPU parity tests: run the HIP path through the C ABI on
numpy inputs, run the oracle on the same inputs, and compare per tensor.

Every float comparison applies two bounds to each tensor: the relative L2
error ||x - ref|| / ||ref|| and the element-wise bound
max|x - ref| <= tol * max|ref|, so that an error confined to one unit, one
tile edge or one row of a large tensor cannot hide inside the norm.  With
PARITY_LOG=<path> in the environment every comparison is appended to that
file as a JSON line (test, tensor, both errors, tolerance)."""

import json
import os
import sys

import numpy as np
import torch

import oracle
from paper_1904_10584_amd import binding as am


def say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def rel_l2(a, ref):
    a = np.asarray(a, np.float64)
    ref = np.asarray(ref, np.float64)
    den = np.linalg.norm(ref)
    return float(np.linalg.norm(a - ref) / den) if den > 0 else float(np.linalg.norm(a))


def max_ratio(a, ref):
    """max|a - ref| / max|ref| (element-wise error against the tensor's scale)."""
    a = np.asarray(a, np.float64)
    ref = np.asarray(ref, np.float64)
    if a.size == 0:
        return 0.0
    den = float(np.max(np.abs(ref)))
    num = float(np.max(np.abs(a - ref)))
    return num / den if den > 0 else num


def _log(name, rl2, mr, tol):
    path = os.environ.get("PARITY_LOG")
    if not path:
        return
    test = os.environ.get("PYTEST_CURRENT_TEST", "").split(" ")[0]
    with open(path, "a") as fh:
        fh.write(json.dumps({"test": test, "tensor": name, "rel_l2": rl2, "max_ratio": mr,
                             "tol": tol}) + "\n")


def assert_close(name, got, ref, tol):
    """Both bounds on one tensor; returns (rel_l2, max_ratio)."""
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    assert got.shape == ref.shape, (name, got.shape, ref.shape)
    assert np.all(np.isfinite(got)), f"{name}: non-finite values"
    rl2, mr = rel_l2(got, ref), max_ratio(got, ref)
    _log(name, rl2, mr, tol)
    assert rl2 <= tol, f"{name}: rel L2 {rl2:.3e} > {tol:g}"
    if mr > tol:
        i = int(np.argmax(np.abs(got - ref)))
        where = np.unravel_index(i, ref.shape)
        raise AssertionError(f"{name}: max|err| / max|ref| = {mr:.3e} > {tol:g} at {where} "
                             f"(got {got.flat[i]!r}, ref {ref.flat[i]!r})")
    return rl2, mr


def to_dev(a, dtype=None):
    t = torch.from_numpy(np.ascontiguousarray(a))
    if dtype is not None:
        t = t.to(dtype)
    return t.cuda()


def bf16_dev(a32):
    """fp32 numpy -> bf16 GPU tensor, cast by the library's kernel."""
    src = to_dev(np.asarray(a32, np.float32))
    dst = torch.empty(src.shape, dtype=torch.bfloat16, device="cuda")
    am.cast_f32_to_bf16(src, dst)
    return dst


def gpu_forward_backward(m, master, x, T, B, idx, prob, lengths=None, h0=None, c0=None,
                         dlogits=None, want_state=False):
    """HIP path: forward, soft CE (unless dlogits is given), backward."""
    bf = m.dtype == am.BF16
    N = x.shape[0]
    if bf:
        params = bf16_dev(master)
        xd = bf16_dev(x)
    else:
        params = to_dev(np.asarray(master, np.float32))
        xd = to_dev(np.asarray(x, np.float32))
    logits = torch.empty((N, m.classes), dtype=torch.float32, device="cuda")
    ws = torch.empty(am.workspace_bytes(m, T, B, N), dtype=torch.uint8, device="cuda")
    h0d = to_dev(np.asarray(h0, np.float32)) if h0 is not None else None
    c0d = to_dev(np.asarray(c0, np.float32)) if c0 is not None else None
    hT = cT = None
    if want_state:
        hT = torch.empty((m.layers, B, m.hidden), dtype=torch.float32, device="cuda")
        cT = torch.empty_like(hT)
    am.lstm_am_forward(m, params, xd, T, B, logits, ws, lengths=lengths, h0=h0d, c0=c0d, hT=hT, cT=cT)
    out = {}
    if dlogits is None:
        dz = torch.empty((N, m.classes), dtype=m.torch_dtype, device="cuda")
        loss = torch.zeros(1, dtype=torch.float32, device="cuda")
        cws = torch.empty(am.ce_workspace_bytes(N), dtype=torch.uint8, device="cuda")
        am.sparse_soft_ce(logits, to_dev(idx.astype(np.int32)), to_dev(prob.astype(np.float32)),
                          loss, dz, cws)
        out["loss"] = float(loss.cpu()[0])
    else:
        dz = to_dev(np.asarray(dlogits, np.float32))
        if bf:
            dz = dz.to(torch.bfloat16)
    grads = torch.empty(am.param_count(m), dtype=torch.float32, device="cuda")
    am.lstm_am_backward(m, params, xd, T, B, dz, ws, grads, lengths=lengths)
    am.workspace_check(ws)
    torch.cuda.synchronize()
    out["logits"] = logits.cpu().numpy()
    out["dlogits"] = dz.float().cpu().numpy()
    out["grads"] = grads.cpu().numpy()
    if want_state:
        out["hT"] = hT.cpu().numpy()
        out["cT"] = cT.cpu().numpy()
    return out


def oracle_forward_backward(dims, master, x, T, B, idx, prob, lengths=None, h0=None, c0=None,
                            bf16=False, dlogits=None):
    p = oracle.bf16_round(master) if bf16 else np.asarray(master, np.float32)
    xe = oracle.bf16_round(x) if bf16 else np.asarray(x, np.float32)
    logits, cache = oracle.lstm_am_forward(p, dims, xe, T, B, lengths, h0, c0)
    out = {"logits": logits, "hT": cache["hT"], "cT": cache["cT"]}
    if dlogits is None:
        loss, dz = oracle.sparse_soft_ce(logits, idx, prob)
        out["loss"] = loss
    else:
        dz = np.asarray(dlogits, np.float64)
    out["dlogits"] = dz
    out["grads"] = oracle.lstm_am_backward(p, dims, cache, dz)
    return out


def grad_tensors(grads, dims):
    """Named parameter tensors of a flat gradient."""
    gl, go = oracle.unpack_params(np.asarray(grads, np.float64), dims)
    out = {"Wo": go["Wo"], "bo": go["bo"]}
    for l, a in enumerate(gl):
        for k in ("Wx", "Wh", "b"):
            out[f"{k}{l}"] = a[k]
    return out


def check_grads(grads, ref, dims, tol, label="grad"):
    """Both bounds on every parameter tensor of the gradient; returns the
    largest rel L2 and the largest element-wise ratio."""
    g, r = grad_tensors(grads, dims), grad_tensors(ref, dims)
    worst_l2 = worst_mr = 0.0
    for k in r:
        rl2, mr = assert_close(f"{label}.{k}", g[k], r[k], tol)
        worst_l2, worst_mr = max(worst_l2, rl2), max(worst_mr, mr)
    return worst_l2, worst_mr


def per_tensor_errors(grads, ref, dims):
    gl, go = oracle.unpack_params(np.asarray(grads, np.float64), dims)
    rl, ro = oracle.unpack_params(np.asarray(ref, np.float64), dims)
    errs = {"Wo": rel_l2(go["Wo"], ro["Wo"]), "bo": rel_l2(go["bo"], ro["bo"])}
    for l, (a, b) in enumerate(zip(gl, rl)):
        for k in ("Wx", "Wh", "b"):
            errs[f"{k}{l}"] = rel_l2(a[k], b[k])
    return errs
