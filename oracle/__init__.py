"""ctypes wrapper of the CPU oracle (oracle.c) -- TEST INFRASTRUCTURE ONLY.

Only tests/, the smoke check and the benchmark's CPU-baseline leg import this
package.  The library under paper_2609_34162_amd never does.
"""
import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
# ORACLE_LIB names another build of oracle.c (the sanitizer run's)
LIB_PATH = os.environ.get("ORACLE_LIB") or os.path.join(_HERE, "liboracle.so")
CFLAGS = ["-O2", "-fopenmp", "-fPIC", "-shared", "-std=c11",
          "-ffp-contract=off", "-fno-fast-math"]

ORC_OK, ORC_NONFINITE, ORC_INVALID = 0, 1, -1
MAX_RANKS = 64


def build(force: bool = True, src: str = None, out: str = None) -> str:
    """Compile oracle.c with gcc.  ``src``/``out`` let a test build a copy."""
    src = src or os.path.join(_HERE, "oracle.c")
    out = out or LIB_PATH
    if force or not os.path.exists(out):
        tmp = out + ".tmp"
        subprocess.check_call(["gcc", *CFLAGS, "-I", _HERE, "-o", tmp, src, "-lm"])
        os.replace(tmp, out)
    return out


class Segment(ctypes.Structure):
    _fields_ = [("master", ctypes.c_void_p), ("exp_avg", ctypes.c_void_p),
                ("exp_avg_sq", ctypes.c_void_p), ("param_bf16", ctypes.c_void_p),
                ("grads", ctypes.c_void_p), ("numel", ctypes.c_int64)]


class HParams(ctypes.Structure):
    _fields_ = [("lr", ctypes.c_double), ("beta1", ctypes.c_double),
                ("beta2", ctypes.c_double), ("eps", ctypes.c_double),
                ("weight_decay", ctypes.c_double),
                ("max_grad_norm", ctypes.c_double), ("step", ctypes.c_int64)]


def hparams(lr=1e-5, beta1=0.9, beta2=0.999, eps=1e-8, weight_decay=0.01,
            max_grad_norm=1.0, step=1) -> HParams:
    return HParams(lr, beta1, beta2, eps, weight_decay, max_grad_norm, step)


def _declare(L):
    vp, i64, i32, dbl = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32, ctypes.c_double
    L.orc_bf16_from_f32.restype = ctypes.c_uint16
    L.orc_bf16_from_f32.argtypes = [ctypes.c_float]
    L.orc_bf16_array.restype = None
    L.orc_bf16_array.argtypes = [vp, vp, i64]
    L.orc_mean_grads.restype = None
    L.orc_mean_grads.argtypes = [vp, i32, i64, vp]
    L.orc_grad_norm.restype = dbl
    L.orc_grad_norm.argtypes = [vp, i32, i32]
    L.orc_sum_squares_f32.restype = dbl
    L.orc_sum_squares_f32.argtypes = [vp, i64]
    L.orc_clip_coef.restype = dbl
    L.orc_clip_coef.argtypes = [dbl, dbl]
    L.orc_adamw_f64.restype = None
    L.orc_adamw_f64.argtypes = [i64, vp, vp, vp, vp, ctypes.POINTER(HParams), vp, vp, vp]
    L.orc_step.restype = ctypes.c_int
    L.orc_step.argtypes = [vp, i32, i32, ctypes.POINTER(HParams), ctypes.POINTER(dbl)]
    L.orc_step_fmt.restype = ctypes.c_int
    L.orc_step_fmt.argtypes = [vp, i32, i32, ctypes.POINTER(HParams), i32, ctypes.POINTER(dbl)]
    L.orc_update_points_fmt.restype = None
    L.orc_update_points_fmt.argtypes = [i64, vp, vp, vp, vp, i32, dbl,
                                        ctypes.POINTER(HParams), i32, vp, vp, vp, vp]
    L.orc_update_points.restype = None
    L.orc_update_points.argtypes = [i64, vp, vp, vp, vp, i32, dbl,
                                    ctypes.POINTER(HParams), vp, vp, vp, vp]
    L.orc_update_given_clip.restype = None
    L.orc_update_given_clip.argtypes = [i64, vp, vp, vp, vp, vp, i32, dbl, ctypes.POINTER(HParams), i32]
    L.orc_num_threads.restype = ctypes.c_int
    L.orc_num_threads.argtypes = []
    L.orc_set_num_threads.restype = None
    L.orc_set_num_threads.argtypes = [ctypes.c_int]
    return L


_lib = None


def load(path: str = None):
    """Load the oracle library (building it if nothing is built)."""
    global _lib
    if path is not None:
        return _declare(ctypes.CDLL(path))
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            build(force=False)
        _lib = _declare(ctypes.CDLL(LIB_PATH))
    return _lib


def _ptr(a: np.ndarray, dtype) -> int:
    assert a.dtype == dtype and a.flags.c_contiguous, (a.dtype, dtype)
    return a.ctypes.data


class State:
    """Host copies of one call's segments: FP32 master/m/v, BF16 params and
    the R BF16 gradient arrays of each segment (numpy arrays)."""

    def __init__(self, masters, exp_avgs=None, exp_avg_sqs=None, params=None):
        self.master = [np.ascontiguousarray(m, dtype=np.float32).copy() for m in masters]
        n = [m.size for m in self.master]
        self.exp_avg = ([np.zeros(k, np.float32) for k in n] if exp_avgs is None
                        else [np.ascontiguousarray(a, dtype=np.float32).copy() for a in exp_avgs])
        self.exp_avg_sq = ([np.zeros(k, np.float32) for k in n] if exp_avg_sqs is None
                           else [np.ascontiguousarray(a, dtype=np.float32).copy() for a in exp_avg_sqs])
        self.param_bf16 = ([np.zeros(k, np.uint16) for k in n] if params is None
                           else [np.ascontiguousarray(a, dtype=np.uint16).copy() for a in params])

    def copy(self) -> "State":
        return State(self.master, self.exp_avg, self.exp_avg_sq, self.param_bf16)


def _segments(state: State, grads):
    """Build the ctypes segment array; grads[s] is a list of R uint16 arrays."""
    keep = []
    segs = (Segment * len(state.master))()
    R = None
    for s in range(len(state.master)):
        gs = grads[s]
        if R is None:
            R = len(gs)
        assert len(gs) == R
        ptrs = (ctypes.c_void_p * R)(*[_ptr(g, np.uint16) for g in gs])
        for g in gs:
            assert g.size == state.master[s].size
        keep.append(ptrs)
        segs[s] = Segment(_ptr(state.master[s], np.float32),
                          _ptr(state.exp_avg[s], np.float32),
                          _ptr(state.exp_avg_sq[s], np.float32),
                          _ptr(state.param_bf16[s], np.uint16),
                          ctypes.cast(ptrs, ctypes.c_void_p), state.master[s].size)
    return segs, R, keep


def step(state: State, grads, hp: HParams, lib=None, gbar_bf16=False):
    """One oracle step in place.  Returns (status, norm).  gbar_bf16: the
    update consumes the mean gradient rounded to BF16 (the norm does not)."""
    L = lib or load()
    segs, R, keep = _segments(state, grads)
    norm = ctypes.c_double(0.0)
    rc = L.orc_step_fmt(ctypes.cast(segs, ctypes.c_void_p), len(state.master), R,
                        ctypes.byref(hp), int(bool(gbar_bf16)), ctypes.byref(norm))
    del keep
    return rc, norm.value


def grad_norm(grads, lib=None) -> float:
    """Global norm of the mean gradient; grads[s] is a list of R arrays."""
    L = lib or load()
    n = [g[0].size for g in grads]
    dummy = State([np.zeros(0, np.float32) for _ in n])
    segs = (Segment * len(grads))()
    keep = []
    R = len(grads[0])
    for s, gs in enumerate(grads):
        ptrs = (ctypes.c_void_p * R)(*[_ptr(g, np.uint16) for g in gs])
        keep.append(ptrs)
        segs[s] = Segment(0, 0, 0, 0, ctypes.cast(ptrs, ctypes.c_void_p), n[s])
    del dummy
    return L.orc_grad_norm(ctypes.cast(segs, ctypes.c_void_p), len(grads), R)


def mean_grads(gs, lib=None) -> np.ndarray:
    L = lib or load()
    R = len(gs)
    ptrs = (ctypes.c_void_p * R)(*[_ptr(g, np.uint16) for g in gs])
    out = np.empty(gs[0].size, np.float32)
    L.orc_mean_grads(ctypes.cast(ptrs, ctypes.c_void_p), R, out.size, out.ctypes.data)
    return out


def sum_squares(x: np.ndarray, lib=None) -> float:
    """Correctly rounded sum of the squares of FP32 values."""
    x = np.ascontiguousarray(x, np.float32)
    return (lib or load()).orc_sum_squares_f32(x.ctypes.data, x.size)


def clip_coef(norm: float, max_grad_norm: float, lib=None) -> float:
    return (lib or load()).orc_clip_coef(norm, max_grad_norm)


def bf16(x: np.ndarray, lib=None) -> np.ndarray:
    x = np.ascontiguousarray(x, dtype=np.float32)
    out = np.empty(x.size, np.uint16)
    (lib or load()).orc_bf16_array(x.ctypes.data, out.ctypes.data, x.size)
    return out


def adamw_f64(p, m, v, g, hp: HParams, lib=None):
    L = lib or load()
    arrs = [np.ascontiguousarray(a, dtype=np.float64) for a in (p, m, v, g)]
    n = arrs[0].size
    po, mo, vo = (np.empty(n, np.float64) for _ in range(3))
    L.orc_adamw_f64(n, *[a.ctypes.data for a in arrs], ctypes.byref(hp),
                    po.ctypes.data, mo.ctypes.data, vo.ctypes.data)
    return po, mo, vo


def update_points(p, m, v, g_rows, clip_c: float, hp: HParams, lib=None, gbar_bf16=False):
    """Update independent points; g_rows has shape (n, R) of uint16."""
    L = lib or load()
    p = np.ascontiguousarray(p, np.float32)
    m = np.ascontiguousarray(m, np.float32)
    v = np.ascontiguousarray(v, np.float32)
    g_rows = np.ascontiguousarray(g_rows, np.uint16)
    n, R = g_rows.shape
    po, mo, vo = (np.empty(n, np.float32) for _ in range(3))
    pb = np.empty(n, np.uint16)
    L.orc_update_points_fmt(n, p.ctypes.data, m.ctypes.data, v.ctypes.data,
                            g_rows.ctypes.data, R, clip_c, ctypes.byref(hp), int(bool(gbar_bf16)),
                            po.ctypes.data, mo.ctypes.data, vo.ctypes.data, pb.ctypes.data)
    return po, mo, vo, pb


def update_given_clip(p, m, v, pb, gs, clip_c: float, hp: HParams, lib=None, gbar_bf16=False):
    """Update the arrays p, m, v, pb in place from the R gradient arrays gs
    with a known clip coefficient (no norm pass)."""
    L = lib or load()
    n = p.size
    for a, dt in ((p, np.float32), (m, np.float32), (v, np.float32), (pb, np.uint16)):
        assert a.size == n
        _ptr(a, dt)
    for g in gs:
        assert g.size == n
    ptrs = (ctypes.c_void_p * len(gs))(*[_ptr(g, np.uint16) for g in gs])
    L.orc_update_given_clip(n, p.ctypes.data, m.ctypes.data, v.ctypes.data, pb.ctypes.data,
                            ctypes.cast(ptrs, ctypes.c_void_p), len(gs), clip_c, ctypes.byref(hp),
                            int(bool(gbar_bf16)))


def num_threads(lib=None) -> int:
    return (lib or load()).orc_num_threads()


def set_num_threads(n: int, lib=None) -> None:
    (lib or load()).orc_set_num_threads(n)
