"""Host-side checks of the C ABI (no GPU needed): the library loads, exports
every entry point the header declares, agrees with the oracle on the
parameter layout, and rejects invalid arguments before enqueuing anything."""

import ctypes
import os
import re

import numpy as np
import pytest

import oracle
from paper_1904_10584_amd import binding as am

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "mi355am.h")


def _declared_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    names = re.findall(r"^[A-Za-z_][\w \*]*?\b(\w+)\s*\(", src, flags=re.M)
    return sorted(set(n for n in names if n not in ("if", "while")))


@pytest.fixture(scope="module")
def L():
    return am.lib()


def test_library_exports_every_declared_function(L):
    declared = _declared_functions()
    assert len(declared) >= 17
    for name in declared:
        assert hasattr(L, name), name
    assert sorted(declared) == sorted(am.exported_symbols())


@pytest.mark.parametrize("dims", [(2, 64, 64, 500), (5, 192, 768, 3000), (5, 192, 1536, 6000), (1, 8, 16, 8)])
def test_param_layout_matches_oracle(dims):
    m = am.Model(*dims, dtype=am.F32)
    d = oracle.ModelDims(*dims)
    assert am.param_count(m) == oracle.param_count(d)
    assert am.param_offsets(m) == oracle.param_offsets(d)


def test_paper_model_size():
    assert am.param_count(am.Model(5, 192, 768, 3000)) == 24_145_848


def _m(L_=2, D=64, H=64, C=500, dt=am.F32):
    return am._Model(L_, D, H, C, dt)


def _status(L, fn, *args):
    st = getattr(L, fn)(*args)
    return st, L.am_last_error().decode()


def test_invalid_models_rejected(L):
    for bad, code in [((2, 64, 20, 500, am.F32), -3), ((0, 64, 64, 500, am.F32), -1),
                      ((2, 64, 64, 500, 7), -1), ((2, 64, 64, 500, am.BF16), -3),
                      ((2, 60, 64, 504, am.BF16), -3)]:
        m = am._Model(*bad)
        assert L.am_param_count(ctypes.byref(m)) == -1
        off = (ctypes.c_int64 * 64)()
        st, msg = _status(L, "am_param_offsets", ctypes.byref(m), off)
        assert st == code and msg


def test_forward_argument_checks_enqueue_nothing(L):
    m = _m()
    fake = ctypes.c_void_p(0x100000)   # never dereferenced: validation fails first
    ws_need = L.am_workspace_bytes(ctypes.byref(m), 5, 3, 15)
    assert ws_need > 0
    lens_bad = (ctypes.c_int32 * 3)(2, 5, 1)       # not non-increasing
    st, msg = _status(L, "lstm_am_forward", ctypes.byref(m), fake, fake, lens_bad, None, None, 5, 3,
                      fake, None, None, fake, ws_need, None)
    assert st == -1 and "non-increasing" in msg
    lens_long = (ctypes.c_int32 * 3)(9, 5, 1)       # longer than T
    st, _ = _status(L, "lstm_am_forward", ctypes.byref(m), fake, fake, lens_long, None, None, 5, 3,
                    fake, None, None, fake, ws_need, None)
    assert st == -1
    st, msg = _status(L, "lstm_am_forward", ctypes.byref(m), fake, fake, None, None, None, 5, 3,
                      fake, None, None, fake, ws_need - 1, None)
    assert st == -5
    st, _ = _status(L, "lstm_am_forward", ctypes.byref(m), fake, fake, None, None, None, 5, 0,
                    fake, None, None, fake, ws_need, None)
    assert st == -1
    misaligned = ctypes.c_void_p(0x100004)
    st, _ = _status(L, "lstm_am_forward", ctypes.byref(m), fake, misaligned, None, None, None, 5, 3,
                    fake, None, None, fake, ws_need, None)
    assert st == -1
    st, _ = _status(L, "lstm_am_backward", ctypes.byref(m), fake, fake, None, 5, 3, fake, fake,
                    ws_need, None, None)
    assert st == -1


def test_encode_decode_ce_sgd_argument_checks(L):
    fake = ctypes.c_void_p(0x100000)
    n = 1000
    ws = L.am_encode_workspace_bytes(n)
    st, _ = _status(L, "grad_threshold_encode", n, fake, fake, ctypes.c_float(1e-3), fake, n - 1, fake, fake, ws, None)
    assert st == -2
    st, _ = _status(L, "grad_threshold_encode", n, fake, fake, ctypes.c_float(0.0), fake, n, fake, fake, ws, None)
    assert st == -1
    st, _ = _status(L, "grad_threshold_encode", n, fake, fake, ctypes.c_float(1e-3), fake, n, fake, fake, ws - 1, None)
    assert st == -5
    st, _ = _status(L, "grad_threshold_encode", 1 << 31, fake, fake, ctypes.c_float(1e-3), fake, 1 << 31, fake, fake, ws, None)
    assert st == -1
    st, _ = _status(L, "grad_threshold_decode", fake, fake, 10, ctypes.c_float(1e-3), n, fake, 2, None)
    assert st == -1
    cws = L.am_ce_workspace_bytes(16)
    st, _ = _status(L, "sparse_soft_ce", 16, 10000, 5, fake, fake, fake, None, 0, fake, fake, 0, fake, cws, None)
    assert st == -3   # more classes than the register-resident row holds
    st, _ = _status(L, "sparse_soft_ce", 16, 502, 5, fake, fake, fake, None, 0, fake, fake, 0, fake, cws, None)
    assert st == -3   # C not a multiple of 4
    st, _ = _status(L, "sparse_soft_ce", 16, 500, 5, fake, fake, fake, None, 3, fake, fake, 0, fake, cws, None)
    assert st == -1
    st, _ = _status(L, "sgd_apply", -1, fake, None, fake, ctypes.c_float(0.1), None)
    assert st == -1
    f = ctypes.c_float
    st, _ = _status(L, "grad_threshold_decode_sgd", fake, fake, 10, f(1e-3), 1 << 31, f(0.1), fake, None, None)
    assert st == -1   # n outside [0, 2^31)
    st, _ = _status(L, "grad_threshold_decode_sgd", fake, fake, -1, f(1e-3), n, f(0.1), fake, None, None)
    assert st == -1   # negative capacity
    st, _ = _status(L, "grad_threshold_decode_sgd", fake, None, 10, f(1e-3), n, f(0.1), fake, None, None)
    assert st == -1   # no count
    st, _ = _status(L, "grad_threshold_decode_sgd", fake, fake, 10, f(1e-3), n, f(0.1), None, None, None)
    assert st == -1   # no master
    st, _ = _status(L, "grad_threshold_decode_sgd", None, fake, 10, f(1e-3), n, f(0.1), fake, None, None)
    assert st == -1   # words missing for a positive capacity
    for s in (0, -1, -2, -3, -4, -5, -6):
        assert L.am_status_string(s)
    assert b"timed out" in L.am_status_string(-6)
    # the time-out query validates before it touches the stream
    st, _ = _status(L, "am_workspace_check", None, 1 << 20, None)
    assert st == -1
    st, _ = _status(L, "am_workspace_check", ctypes.c_void_p(0x100010), 1 << 20, None)
    assert st == -1   # not 256-byte aligned
    st, _ = _status(L, "am_workspace_check", fake, 4096, None)
    assert st == -5   # smaller than the sync region


def test_workspace_queries_are_monotone(L):
    m = _m(5, 192, 768, 3000, am.BF16)
    a = L.am_workspace_bytes(ctypes.byref(m), 64, 256, 64 * 256)
    b = L.am_workspace_bytes(ctypes.byref(m), 64, 256, 64 * 128)
    assert a > b > 0 and a % 256 == 0
    assert L.am_workspace_bytes(ctypes.byref(m), 64, 256, 64 * 256 + 1) == -1
    assert L.am_encode_workspace_bytes(24_145_848) > L.am_encode_workspace_bytes(1000) > 0


def test_bmuf_and_multi_decode_argument_checks(L):
    fake = ctypes.c_void_p(0x100000)
    f = ctypes.c_float
    # bmuf: counts, stride, NULLs
    st, _ = _status(L, "bmuf_block_update", 100, 0, 1, fake, 100, fake, fake, f(0.5), f(0.5), f(1.0), None, None, None)
    assert st == -1
    st, _ = _status(L, "bmuf_block_update", 100, 2, 2, fake, 99, fake, fake, f(0.5), f(0.5), f(1.0), None, None, None)
    assert st == -1
    st, _ = _status(L, "bmuf_block_update", 100, 1, 0, fake, 100, fake, fake, f(0.5), f(0.5), f(1.0), None, None, None)
    assert st == -1
    st, _ = _status(L, "bmuf_block_update", 100, 1, 1, None, 100, fake, fake, f(0.5), f(0.5), f(1.0), None, None, None)
    assert st == -1
    # multi-stream decode: stream count, workspace, NULLs, accumulate flag
    n = 50_000
    ws = L.am_decode_multi_workspace_bytes(4, n)
    assert ws >= 4 * ((n + 4095) // 4096 + 1) * 4 and ws % 256 == 0
    assert L.am_decode_multi_workspace_bytes(-1, n) == -1
    st, _ = _status(L, "grad_threshold_decode_multi", 40000, fake, n, fake, f(1e-3), n, fake, 0, fake, 1 << 30, None)
    assert st == -1
    st, _ = _status(L, "grad_threshold_decode_multi", 4, fake, n, fake, f(1e-3), n, fake, 0, fake, ws - 1, None)
    assert st == -5
    st, _ = _status(L, "grad_threshold_decode_multi", 4, fake, n, None, f(1e-3), n, fake, 0, fake, ws, None)
    assert st == -1
    st, _ = _status(L, "grad_threshold_decode_multi", 4, fake, n, fake, f(1e-3), n, fake, 2, fake, ws, None)
    assert st == -1
    st, _ = _status(L, "grad_threshold_decode_multi", 4, fake, n, fake, f(1e-3), 1 << 31, fake, 0, fake, ws, None)
    assert st == -1


@pytest.mark.parametrize("dims", [(2, 64, 64, 500), (5, 192, 768, 3000), (1, 8, 16, 8)])
def test_teacher_layout_matches_oracle(dims):
    L_, D, H, C = dims
    m = am.Model(L_, D, H, C, am.BF16 if D % 8 == 0 and C % 8 == 0 else am.F32)
    td = oracle.TeacherDims(L_, D, H, C)
    assert am.teacher_param_count(m) == oracle.teacher_param_count(td)
    assert am.teacher_param_offsets(m) == oracle.teacher_param_offsets(td)


def test_teacher_argument_checks(L):
    fake = ctypes.c_void_p(0x100000)
    m = _m(2, 64, 64, 520, am.BF16)
    ws = L.am_teacher_workspace_bytes(ctypes.byref(m), 10, 4, 40)
    assert ws > 0 and ws % 256 == 0
    st, _ = _status(L, "blstm_teacher_forward", ctypes.byref(m), fake, fake, None, 10, 4, fake, fake, ws - 1, None)
    assert st == -5
    st, _ = _status(L, "blstm_teacher_forward", ctypes.byref(m), fake, fake, None, 10, 2000, fake, fake, ws, None)
    assert st == -3
    st, _ = _status(L, "kbest_logits", 10, 100, 101, fake, fake, fake, None)
    assert st == -1   # K > C
    st, _ = _status(L, "kbest_logits", 10, 100, 65, fake, fake, fake, None)
    assert st == -3   # K > 64
    st, _ = _status(L, "kbest_logits", 10, 9000, 20, fake, fake, fake, None)
    assert st == -3   # C > 8192
    st, _ = _status(L, "kbest_posteriors", -1, 20, fake, fake, None)
    assert st == -1


def test_recurrence_path_query(monkeypatch):
    # host logic only: the XCD-local kernels are built for bf16 H = 768 with
    # B <= 256; variable lengths hold 16-bit lengths, so T > 65535 must not
    # take them (the per-step kernels use the host's 64-bit schedule)
    monkeypatch.delenv("AM_RECURRENCE", raising=False)
    monkeypatch.delenv("AM_STEP_KERNELS", raising=False)
    paper = am.Model(5, 192, 768, 3000, am.BF16)
    for fwd in (True, False):
        assert am.recurrence_path(paper, 64, 256, False, fwd) == am.PATH_XCD
        assert am.recurrence_path(paper, 1500, 128, True, fwd) == am.PATH_XCD
        assert am.recurrence_path(paper, 65535, 128, True, fwd) == am.PATH_XCD
        assert am.recurrence_path(paper, 65536, 128, True, fwd) != am.PATH_XCD
        assert am.recurrence_path(paper, 70000, 128, False, fwd) == am.PATH_XCD
        # fp32 models never take the XCD-local kernels
        assert am.recurrence_path(am.Model(5, 192, 768, 3000, am.F32), 64, 256, False, fwd) != am.PATH_XCD
    monkeypatch.setenv("AM_RECURRENCE", "step")
    assert am.recurrence_path(paper, 64, 256) == am.PATH_STEP
    with pytest.raises(am.AmError):
        am.recurrence_path(am.Model(5, 192, 770, 3000, am.BF16), 64, 256)


def test_profile_sampling_interval(L):
    # host logic only (no launch is recorded): the interval must be >= 1
    assert L.am_profile_sample_every(0) == am.EINVAL
    assert L.am_profile_sample_every(-3) == am.EINVAL
    assert L.am_profile_sample_every(7) == am.OK
    assert L.am_profile_sample_every(1) == am.OK
