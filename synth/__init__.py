"""Seeded synthetic inputs shared by the oracle and the HIP path.

Values come from the counter-based generator in ``gen.c``; gradients are
rounded to BF16 with torch's CPU cast (a library conversion, so this package
holds none of the update's arithmetic).
"""
import ctypes
import os
import subprocess

import numpy as np

from .configs import NORM_TILE, WORKLOADS, Workload, workload  # noqa: F401

_HERE = os.path.dirname(os.path.abspath(__file__))
# SYNTH_LIB names another build of gen.c (the sanitizer run's)
LIB_PATH = os.environ.get("SYNTH_LIB") or os.path.join(_HERE, "libsynth.so")
KIND_MASTER = 0
KIND_GRAD = 1

_lib = None


def build(force: bool = True) -> str:
    """Compile gen.c with gcc into libsynth.so (host code, OpenMP)."""
    if force or not os.path.exists(LIB_PATH):
        src = os.path.join(_HERE, "gen.c")
        tmp = LIB_PATH + ".tmp"
        subprocess.check_call(["gcc", "-O2", "-fopenmp", "-fPIC", "-shared",
                               "-std=c11", "-o", tmp, src, "-lm"])
        os.replace(tmp, LIB_PATH)
    return LIB_PATH


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            build(force=False)
        L = ctypes.CDLL(LIB_PATH)
        i64, u64, dbl = ctypes.c_int64, ctypes.c_uint64, ctypes.c_double
        vp = ctypes.c_void_p
        L.synth_seed.restype = u64
        L.synth_seed.argtypes = [vp, ctypes.c_int]
        L.synth_splitmix64.restype = u64
        L.synth_splitmix64.argtypes = [u64]
        L.synth_philox4x32_10.restype = None
        L.synth_philox4x32_10.argtypes = [u64, u64, vp]
        L.synth_normal_f32.restype = None
        L.synth_normal_f32.argtypes = [u64, i64, i64, dbl, dbl, dbl, vp]
        L.synth_normal_f32_at.restype = None
        L.synth_normal_f32_at.argtypes = [u64, vp, i64, dbl, dbl, dbl, vp]
        L.synth_raw_u32.restype = None
        L.synth_raw_u32.argtypes = [u64, i64, i64, vp]
        _lib = L
    return _lib


def seed(*fields: int) -> int:
    arr = np.asarray(fields, dtype=np.int64)
    return int(lib().synth_seed(arr.ctypes.data, len(fields)))


def philox(key: int, ctr: int) -> np.ndarray:
    out = np.zeros(4, dtype=np.uint32)
    lib().synth_philox4x32_10(key, ctr, out.ctypes.data)
    return out


def raw_u32(s: int, start_block: int, n_blocks: int) -> np.ndarray:
    out = np.empty(4 * n_blocks, dtype=np.uint32)
    lib().synth_raw_u32(s, start_block, n_blocks, out.ctypes.data)
    return out


def normal_f32(s: int, n: int, sigma: float, start: int = 0,
               outlier_p: float = 0.0, outlier_scale: float = 1.0,
               out: np.ndarray = None) -> np.ndarray:
    if out is None:
        out = np.empty(n, dtype=np.float32)
    assert out.dtype == np.float32 and out.size == n and out.flags.c_contiguous
    lib().synth_normal_f32(s, start, n, sigma, outlier_p, outlier_scale,
                           out.ctypes.data)
    return out


def normal_f32_at(s: int, idx: np.ndarray, sigma: float,
                  outlier_p: float = 0.0, outlier_scale: float = 1.0) -> np.ndarray:
    idx = np.ascontiguousarray(idx, dtype=np.int64)
    out = np.empty(idx.size, dtype=np.float32)
    lib().synth_normal_f32_at(s, idx.ctypes.data, idx.size, sigma, outlier_p,
                              outlier_scale, out.ctypes.data)
    return out


def to_bf16_bits(x: np.ndarray, out: np.ndarray = None,
                 block: int = 1 << 26) -> np.ndarray:
    """BF16 bit patterns of FP32 values, by torch's CPU cast."""
    import torch
    x = np.ascontiguousarray(x, dtype=np.float32)
    if out is None:
        out = np.empty(x.size, dtype=np.uint16)
    ot = torch.from_numpy(out.view(np.int16)).view(torch.bfloat16)
    for a in range(0, x.size, block):
        b = min(a + block, x.size)
        ot[a:b].copy_(torch.from_numpy(x[a:b]))
    return out


# ---- workload streams -------------------------------------------------------

def master_seed(w: Workload, seg: int) -> int:
    return seed(w.cid, seg, 0, 0, KIND_MASTER)


def grad_seed(w: Workload, seg: int, step: int, rank: int) -> int:
    return seed(w.cid, seg, step, rank, KIND_GRAD)


def master(w: Workload, seg: int, out: np.ndarray = None) -> np.ndarray:
    n = w.segments[seg].numel
    return normal_f32(master_seed(w, seg), n, w.master_sigma, out=out)


def grad_bf16(w: Workload, seg: int, step: int, rank: int,
              out: np.ndarray = None, block: int = 1 << 26) -> np.ndarray:
    """BF16 gradient of one rank, segment and step (step counts from 1)."""
    n = w.segments[seg].numel
    if out is None:
        out = np.empty(n, dtype=np.uint16)
    s = grad_seed(w, seg, step, rank)
    tmp = np.empty(min(block, n), dtype=np.float32)
    for a in range(0, n, block):
        b = min(a + block, n)
        t = tmp[:b - a]
        normal_f32(s, b - a, w.sigma, start=a, outlier_p=w.outlier_p,
                   outlier_scale=w.outlier_scale, out=t)
        to_bf16_bits(t, out=out[a:b])
    return out


def grad_bf16_at(w: Workload, seg: int, step: int, rank: int,
                 idx: np.ndarray) -> np.ndarray:
    f = normal_f32_at(grad_seed(w, seg, step, rank), idx, w.sigma,
                      w.outlier_p, w.outlier_scale)
    return to_bf16_bits(f)


def master_at(w: Workload, seg: int, idx: np.ndarray) -> np.ndarray:
    return normal_f32_at(master_seed(w, seg), idx, w.master_sigma)
