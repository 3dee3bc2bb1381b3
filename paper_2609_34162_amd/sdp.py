"""ctypes binding of libsdp (include/sdp.h): argument marshalling only.

Every function here has the name of the C entry point it calls and does
nothing but convert arguments, call it and turn a negative status into an
exception.  All computation runs in the HIP library; if libsdp.so is not
built this module raises on import.
"""
import ctypes
import os
from typing import List, Optional, Sequence, Tuple

_HERE = os.path.dirname(os.path.abspath(__file__))
# SDP_LIB names another build of the same library (the sanitizer run's)
LIB_PATH = os.environ.get("SDP_LIB") or os.path.join(_HERE, "libsdp.so")

# status codes and constants, as in include/sdp.h
SDP_OK = 0
SDP_ERR_INVALID_ARGUMENT = -1
SDP_ERR_ALIGNMENT = -2
SDP_ERR_NOT_DEVICE_MEMORY = -3
SDP_ERR_NOT_PINNED = -4
SDP_ERR_CHUNK_TOO_LARGE = -5
SDP_ERR_OUT_OF_MEMORY = -6
SDP_ERR_HIP = -7
SDP_ERR_NONFINITE = -8
SDP_NORM_TILE = 65536
SDP_MAX_RANKS = 16
SDP_ALIGN = 16
SDP_FLAG_DEVICE_GBAR_NEVER = 0x1
SDP_FLAG_DEVICE_GBAR_ALWAYS = 0x2
SDP_FLAG_STREAM_GBAR_NEVER = 0x4
SDP_FLAG_DEBUG_POISON = 0x8
SDP_FLAG_STREAM_STAGED = 0x10
SDP_FLAG_HOST_PIN_THREADS = 0x20
SDP_FLAG_STREAM_HOST_CAST = 0x40
SDP_FLAG_DEBUG_JITTER = 0x80
SDP_NOALLOC_MAX_SEGMENTS = 64
SDP_NOALLOC_MAX_TILES = 16384
SDP_DELIVER_HOST_CAST = 0
SDP_DELIVER_DEVICE_CAST = 1
SDP_GBAR_F32 = 0
SDP_GBAR_BF16 = 1
SDP_SCHED_STREAMED = 0
SDP_SCHED_STREAMED_STAGED = 1
SDP_SCHED_HOST_ROUTE_F32 = 2
SDP_SCHED_HOST_ROUTE_BF16 = 3


class SdpError(RuntimeError):
    def __init__(self, status: int, name: str, detail: str):
        super().__init__(f"{name}: {detail}")
        self.status = status
        self.name = name
        self.detail = detail


class SdpNonFinite(SdpError):
    def __init__(self, status, name, detail, norm):
        super().__init__(status, name, detail)
        self.norm = norm


class sdp_adamw_params(ctypes.Structure):
    _fields_ = [("lr", ctypes.c_double), ("beta1", ctypes.c_double), ("beta2", ctypes.c_double),
                ("eps", ctypes.c_double), ("weight_decay", ctypes.c_double),
                ("max_grad_norm", ctypes.c_double), ("step", ctypes.c_int64)]


class sdp_segment(ctypes.Structure):
    _fields_ = [("master", ctypes.c_void_p), ("exp_avg", ctypes.c_void_p),
                ("exp_avg_sq", ctypes.c_void_p), ("param_bf16", ctypes.c_void_p),
                ("grads", ctypes.c_void_p), ("n_ranks", ctypes.c_int32), ("numel", ctypes.c_int64)]


class sdp_kernel_times(ctypes.Structure):
    _fields_ = [("norm_ms", ctypes.c_double), ("finalize_ms", ctypes.c_double),
                ("update_ms", ctypes.c_double), ("norm_launches", ctypes.c_int64),
                ("finalize_launches", ctypes.c_int64), ("update_launches", ctypes.c_int64),
                ("update_elems", ctypes.c_int64), ("gbar_ms", ctypes.c_double),
                ("gbar_launches", ctypes.c_int64), ("host_adam_ms", ctypes.c_double),
                ("host_wait_ms", ctypes.c_double), ("host_adam_elems", ctypes.c_int64),
                ("host_issue_ms", ctypes.c_double), ("host_issues", ctypes.c_int64)]


class sdp_rates(ctypes.Structure):
    _fields_ = [(n, ctypes.c_double) for n in ("h2d_gbs", "d2h_gbs", "both_gbs", "copy_cmd_us", "norm_gbs",
                                              "update_gbs", "launch_us", "sync_us", "host_gbs", "host_task_us",
                                              "host_adam_gbs", "dep_us", "dma_host_cost", "host_issue_us")]


class sdp_prediction(ctypes.Structure):
    _fields_ = [(n, ctypes.c_double) for n in ("predicted_ms", "bound_ms", "h2d_ms", "d2h_ms", "link_ms",
                                              "gpu_ms", "host_ms", "dram_ms")] + [("n_chunks", ctypes.c_int64)]


def _load():
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built; run __graft_entry__.build() first")
    L = ctypes.CDLL(LIB_PATH)
    vp, i32, i64, dbl = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_double
    P = ctypes.POINTER
    sig = {
        "sdp_ctx_create": (ctypes.c_int, [P(vp), ctypes.c_int, i64, i32, ctypes.c_uint32]),
        "sdp_ctx_destroy": (None, [vp]),
        "sdp_agg_adam_step": (ctypes.c_int, [vp, vp, i32, P(sdp_adamw_params), i64, vp, P(dbl)]),
        "sdp_stream_step": (ctypes.c_int, [vp, vp, i32, P(sdp_adamw_params), i64, P(dbl)]),
        "sdp_grad_norm": (ctypes.c_int, [vp, vp, i32, ctypes.c_int, i64, vp, P(dbl)]),
        "sdp_ctx_last_norm": (ctypes.c_int, [vp, P(dbl), P(dbl), P(ctypes.c_int)]),
        "sdp_cast_bf16": (ctypes.c_int, [vp, vp, vp, i64, vp]),
        "sdp_deliver_params": (ctypes.c_int, [vp, vp, vp, i64, i64, ctypes.c_int]),
        "sdp_cast_bf16_host": (ctypes.c_int, [vp, vp, vp, i64]),
        "sdp_deliver_params_async": (ctypes.c_int, [vp, vp, vp, i64, i64, ctypes.c_int, vp]),
        "sdp_host_update_step": (ctypes.c_int, [vp, vp, i32, P(sdp_adamw_params), i64, ctypes.c_int, P(dbl)]),
        "sdp_host_adamw": (ctypes.c_int, [vp, vp, vp, vp, vp, vp, ctypes.c_int, i64, dbl,
                                           P(sdp_adamw_params)]),
        "sdp_ctx_set_host_threads": (ctypes.c_int, [vp, i32]),
        "sdp_predict_step": (ctypes.c_int, [ctypes.c_int, vp, i32, i32, i64, ctypes.c_uint32, P(sdp_rates),
                                            P(sdp_prediction)]),
        "sdp_tune_chunk": (ctypes.c_int, [ctypes.c_int, vp, i32, i32, ctypes.c_uint32, P(sdp_rates), vp, i32,
                                          P(i64), P(dbl)]),
        "sdp_probe_host_copy": (ctypes.c_int, [vp, vp, vp, i64, i32, P(dbl)]),
        "sdp_ctx_host_threads": (ctypes.c_int, [vp, P(i32)]),
        "sdp_plan": (ctypes.c_int, [vp, i32, i64, P(i64), P(i64)]),
        "sdp_bytes_per_elem": (ctypes.c_int, [ctypes.c_int, i32, ctypes.c_uint32, P(dbl), P(dbl)]),
        "sdp_ctx_set_timing": (ctypes.c_int, [vp, ctypes.c_int]),
        "sdp_ctx_get_timing": (ctypes.c_int, [vp, P(sdp_kernel_times)]),
        "sdp_probe_copy": (ctypes.c_int, [vp, vp, vp, i64, vp]),
        "sdp_probe_update_pattern": (ctypes.c_int, [vp, vp, vp]),
        "sdp_probe_norm_pattern": (ctypes.c_int, [vp, vp, vp]),
        "sdp_probe_link": (ctypes.c_int, [vp, vp, vp, vp, vp, i64, i64, i32, P(dbl)]),
        "sdp_probe_link_kernel": (ctypes.c_int, [vp, vp, vp, vp, vp, i64, i64, i32, P(dbl)]),
        "sdp_probe_memcpy": (ctypes.c_int, [vp, vp, vp, i64, vp]),
        "sdp_agg_adam_step_noalloc": (ctypes.c_int, [vp, i32, vp, vp, P(dbl)]),
        "sdp_host_alloc": (ctypes.c_int, [P(vp), ctypes.c_size_t]),
        "sdp_host_free": (ctypes.c_int, [vp]),
        "sdp_status_string": (ctypes.c_char_p, [ctypes.c_int]),
        "sdp_last_error": (ctypes.c_char_p, []),
    }
    for name, (res, args) in sig.items():
        f = getattr(L, name)
        f.restype = res
        f.argtypes = args
    return L


_lib = _load()


def _check(rc: int, norm: Optional[float] = None) -> None:
    if rc == SDP_OK:
        return
    name = _lib.sdp_status_string(rc).decode()
    detail = _lib.sdp_last_error().decode()
    if rc == SDP_ERR_NONFINITE:
        raise SdpNonFinite(rc, name, detail, norm)
    raise SdpError(rc, name, detail)


def _stream(stream) -> Optional[int]:
    if stream is None:
        return None
    if hasattr(stream, "cuda_stream"):
        return stream.cuda_stream or None
    return int(stream) or None


class Segments:
    """A marshalled array of sdp_segment (keeps the pointer arrays alive).

    Each entry is (master, exp_avg, exp_avg_sq, param_bf16, [grad ptrs], numel)
    with integer addresses."""

    def __init__(self, entries: Sequence[Tuple[int, int, int, int, Sequence[int], int]]):
        self.n = len(entries)
        self.arr = (sdp_segment * max(self.n, 1))()
        self._keep = []
        for k, (p, m, v, pb, grads, numel) in enumerate(entries):
            g = (ctypes.c_void_p * len(grads))(*grads)
            self._keep.append(g)
            self.arr[k] = sdp_segment(p, m, v, pb, ctypes.cast(g, ctypes.c_void_p), len(grads), numel)

    @property
    def ptr(self):
        return ctypes.cast(self.arr, ctypes.c_void_p)


def segments_from_tensors(tensor_sets) -> Segments:
    """tensor_sets: iterable of (master, exp_avg, exp_avg_sq, param_bf16, grads)
    torch tensors (contiguous; FP32 states, 16-bit params and gradients)."""
    entries = []
    for master, m, v, pb, grads in tensor_sets:
        for t in (master, m, v, pb, *grads):
            if not t.is_contiguous():
                raise ValueError("tensors must be contiguous")
        entries.append((master.data_ptr(), m.data_ptr(), v.data_ptr(), pb.data_ptr(),
                        [g.data_ptr() for g in grads], master.numel()))
    return Segments(entries)


def make_params(lr=1e-5, beta1=0.9, beta2=0.999, eps=1e-8, weight_decay=0.01,
                max_grad_norm=1.0, step=1) -> sdp_adamw_params:
    return sdp_adamw_params(lr, beta1, beta2, eps, weight_decay, max_grad_norm, step)


# ---- entry points ---------------------------------------------------------

def sdp_ctx_create(device: int = 0, max_chunk_elems: int = 0, max_ranks: int = SDP_MAX_RANKS,
                   flags: int = 0) -> ctypes.c_void_p:
    ctx = ctypes.c_void_p()
    _check(_lib.sdp_ctx_create(ctypes.byref(ctx), device, max_chunk_elems, max_ranks, flags))
    return ctx


def sdp_ctx_destroy(ctx) -> None:
    _lib.sdp_ctx_destroy(ctx)


def sdp_agg_adam_step(ctx, segs: Segments, hp: sdp_adamw_params, chunk_elems: int = 0,
                      stream=None, want_norm: bool = False) -> Optional[float]:
    norm = ctypes.c_double(float("nan"))
    rc = _lib.sdp_agg_adam_step(ctx, segs.ptr, segs.n, ctypes.byref(hp), chunk_elems,
                                _stream(stream), ctypes.byref(norm) if want_norm else None)
    _check(rc, norm.value)
    return norm.value if want_norm else None


def sdp_agg_adam_step_noalloc(segs: Segments, hp: sdp_adamw_params, stream=None,
                              want_norm: bool = False) -> Optional[float]:
    norm = ctypes.c_double(float("nan"))
    rc = _lib.sdp_agg_adam_step_noalloc(segs.ptr, segs.n, ctypes.byref(hp), _stream(stream),
                                        ctypes.byref(norm) if want_norm else None)
    _check(rc, norm.value)
    return norm.value if want_norm else None


def sdp_stream_step(ctx, segs: Segments, hp: sdp_adamw_params, chunk_elems: int) -> float:
    norm = ctypes.c_double(float("nan"))
    rc = _lib.sdp_stream_step(ctx, segs.ptr, segs.n, ctypes.byref(hp), chunk_elems, ctypes.byref(norm))
    _check(rc, norm.value)
    return norm.value


def sdp_grad_norm(ctx, segs: Segments, device_resident: bool, chunk_elems: int = 0,
                  stream=None) -> float:
    norm = ctypes.c_double(float("nan"))
    rc = _lib.sdp_grad_norm(ctx, segs.ptr, segs.n, int(bool(device_resident)), chunk_elems,
                            _stream(stream), ctypes.byref(norm))
    _check(rc, norm.value)
    return norm.value


def sdp_ctx_last_norm(ctx) -> Tuple[float, float, bool]:
    n, c, f = ctypes.c_double(), ctypes.c_double(), ctypes.c_int()
    _check(_lib.sdp_ctx_last_norm(ctx, ctypes.byref(n), ctypes.byref(c), ctypes.byref(f)))
    return n.value, c.value, bool(f.value)


def sdp_cast_bf16(ctx, src: int, dst: int, n: int, stream=None) -> None:
    _check(_lib.sdp_cast_bf16(ctx, src, dst, n, _stream(stream)))


def sdp_deliver_params(ctx, host_master: int, dev_bf16: int, n: int, chunk_elems: int,
                       mode: int = SDP_DELIVER_HOST_CAST) -> None:
    _check(_lib.sdp_deliver_params(ctx, host_master, dev_bf16, n, chunk_elems, mode))


def sdp_deliver_params_async(ctx, host_master: int, dev_bf16: int, n: int, chunk_elems: int,
                             mode: int = SDP_DELIVER_HOST_CAST, consumer_stream=None) -> None:
    _check(_lib.sdp_deliver_params_async(ctx, host_master, dev_bf16, n, chunk_elems, mode,
                                         _stream(consumer_stream)))


def sdp_cast_bf16_host(ctx, src: int, dst: int, n: int) -> None:
    _check(_lib.sdp_cast_bf16_host(ctx, src, dst, n))


def sdp_host_update_step(ctx, segs: Segments, hp: sdp_adamw_params, chunk_elems: int,
                         gbar_format: int = SDP_GBAR_F32) -> float:
    norm = ctypes.c_double(float("nan"))
    rc = _lib.sdp_host_update_step(ctx, segs.ptr, segs.n, ctypes.byref(hp), chunk_elems, gbar_format,
                                   ctypes.byref(norm))
    _check(rc, norm.value)
    return norm.value


def sdp_host_adamw(ctx, master: int, exp_avg: int, exp_avg_sq: int, param_bf16: int, gbar: int,
                   gbar_format: int, n: int, clip_coef: float, hp: sdp_adamw_params) -> None:
    _check(_lib.sdp_host_adamw(ctx, master, exp_avg, exp_avg_sq, param_bf16, gbar, gbar_format, n,
                               clip_coef, ctypes.byref(hp)))


def sdp_probe_host_copy(ctx, dst: int, src: int, nbytes: int, reps: int) -> float:
    g = ctypes.c_double()
    _check(_lib.sdp_probe_host_copy(ctx, dst, src, nbytes, reps, ctypes.byref(g)))
    return g.value


def sdp_ctx_set_host_threads(ctx, threads: int) -> None:
    _check(_lib.sdp_ctx_set_host_threads(ctx, threads))


def sdp_ctx_host_threads(ctx) -> int:
    t = ctypes.c_int32()
    _check(_lib.sdp_ctx_host_threads(ctx, ctypes.byref(t)))
    return t.value


def make_rates(**kw) -> sdp_rates:
    r = sdp_rates()
    r.dma_host_cost = 1.0
    for k, v in kw.items():
        if not hasattr(r, k):
            raise TypeError(f"unknown rate {k}")
        setattr(r, k, float(v))
    return r


def sdp_predict_step(schedule: int, numels: Sequence[int], n_ranks: int, chunk_elems: int, flags: int,
                     rates: sdp_rates) -> sdp_prediction:
    arr = (ctypes.c_int64 * len(numels))(*numels)
    out = sdp_prediction()
    _check(_lib.sdp_predict_step(schedule, ctypes.cast(arr, ctypes.c_void_p), len(numels), n_ranks, chunk_elems,
                                 flags, ctypes.byref(rates), ctypes.byref(out)))
    return out


def sdp_tune_chunk(schedule: int, numels: Sequence[int], n_ranks: int, flags: int, rates: sdp_rates,
                   candidates: Sequence[int]) -> Tuple[int, List[float]]:
    arr = (ctypes.c_int64 * len(numels))(*numels)
    cand = (ctypes.c_int64 * len(candidates))(*candidates)
    ms = (ctypes.c_double * len(candidates))()
    best = ctypes.c_int64()
    _check(_lib.sdp_tune_chunk(schedule, ctypes.cast(arr, ctypes.c_void_p), len(numels), n_ranks, flags,
                               ctypes.byref(rates), ctypes.cast(cand, ctypes.c_void_p), len(candidates),
                               ctypes.byref(best), ms))
    return best.value, list(ms)


def sdp_plan(numels: Sequence[int], chunk_elems: int) -> Tuple[int, int]:
    arr = (ctypes.c_int64 * len(numels))(*numels)
    ch, ti = ctypes.c_int64(), ctypes.c_int64()
    _check(_lib.sdp_plan(ctypes.cast(arr, ctypes.c_void_p), len(numels), chunk_elems,
                         ctypes.byref(ch), ctypes.byref(ti)))
    return ch.value, ti.value


def sdp_bytes_per_elem(streamed: bool, n_ranks: int, flags: int = 0) -> Tuple[float, float]:
    a, b = ctypes.c_double(), ctypes.c_double()
    _check(_lib.sdp_bytes_per_elem(int(bool(streamed)), n_ranks, flags, ctypes.byref(a), ctypes.byref(b)))
    return a.value, b.value


def sdp_ctx_set_timing(ctx, enable: bool) -> None:
    _check(_lib.sdp_ctx_set_timing(ctx, int(bool(enable))))


def sdp_ctx_get_timing(ctx) -> sdp_kernel_times:
    t = sdp_kernel_times()
    _check(_lib.sdp_ctx_get_timing(ctx, ctypes.byref(t)))
    return t


def sdp_probe_copy(ctx, dst: int, src: int, nbytes: int, stream=None) -> None:
    _check(_lib.sdp_probe_copy(ctx, dst, src, nbytes, _stream(stream)))


def sdp_probe_memcpy(ctx, dst: int, src: int, nbytes: int, stream=None) -> None:
    _check(_lib.sdp_probe_memcpy(ctx, dst, src, nbytes, _stream(stream)))


def sdp_probe_norm_pattern(ctx, segs: Segments, stream=None) -> None:
    if segs.n != 1:
        raise ValueError("sdp_probe_norm_pattern takes one segment")
    _check(_lib.sdp_probe_norm_pattern(ctx, segs.ptr, _stream(stream)))


def sdp_probe_update_pattern(ctx, segs: Segments, stream=None) -> None:
    if segs.n != 1:
        raise ValueError("sdp_probe_update_pattern takes one segment")
    _check(_lib.sdp_probe_update_pattern(ctx, segs.ptr, _stream(stream)))


def sdp_probe_link(ctx, host_a: int, host_b: int, dev_a: int, dev_b: int, nbytes: int,
                   chunk_bytes: int, reps: int) -> List[float]:
    out = (ctypes.c_double * 3)()
    _check(_lib.sdp_probe_link(ctx, host_a, host_b, dev_a, dev_b, nbytes, chunk_bytes, reps,
                               ctypes.cast(out, ctypes.POINTER(ctypes.c_double))))
    return list(out)


def sdp_probe_link_kernel(ctx, host_a: int, host_b: int, dev_a: int, dev_b: int, nbytes: int,
                          chunk_bytes: int, reps: int) -> List[float]:
    out = (ctypes.c_double * 3)()
    _check(_lib.sdp_probe_link_kernel(ctx, host_a, host_b, dev_a, dev_b, nbytes, chunk_bytes, reps,
                                      ctypes.cast(out, ctypes.POINTER(ctypes.c_double))))
    return list(out)


def sdp_host_alloc(nbytes: int) -> int:
    p = ctypes.c_void_p()
    _check(_lib.sdp_host_alloc(ctypes.byref(p), nbytes))
    return p.value


def sdp_host_free(ptr: int) -> None:
    _check(_lib.sdp_host_free(ptr))


def sdp_status_string(status: int) -> str:
    return _lib.sdp_status_string(status).decode()


def sdp_last_error() -> str:
    return _lib.sdp_last_error().decode()


class _Region:
    """A byte range of a HostBuffer exposed to numpy; keeps the buffer alive."""

    def __init__(self, owner: "HostBuffer", ptr: int, nbytes: int):
        self.owner = owner
        self.__array_interface__ = {"data": (ptr, False), "shape": (nbytes,), "typestr": "|u1", "version": 3}


class HostBuffer:
    """Pinned host memory from sdp_host_alloc, viewable as numpy arrays.
    The memory is freed by close() or when neither the buffer nor any view
    of it is referenced any more."""

    def __init__(self, nbytes: int):
        self.nbytes = nbytes
        self.ptr = sdp_host_alloc(nbytes)

    def view(self, dtype, count: int, offset: int = 0):
        import numpy as np
        dt = np.dtype(dtype)
        if offset < 0 or offset + count * dt.itemsize > self.nbytes:
            raise ValueError("view outside the buffer")
        return np.asarray(_Region(self, self.ptr + offset, count * dt.itemsize)).view(dt)

    def close(self):
        if self.ptr:
            sdp_host_free(self.ptr)
            self.ptr = 0

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
