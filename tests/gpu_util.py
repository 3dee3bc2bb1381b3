"""Helpers for the GPU parity tests: device states in torch tensors, pinned
host states, and the parity criteria against the oracle."""
import ctypes
import os
import subprocess
import sys
import time

import numpy as np
import pytest

import oracle
import synth

torch = pytest.importorskip("torch")


def need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU visible")
    from paper_2609_34162_amd import sdp  # fails loudly if libsdp.so is missing
    return sdp


def log(msg):
    """A progress line that shows even while pytest captures the test's output."""
    import progress
    progress.say(msg)


DEV = "cuda:0"


def to_dev_f32(a):
    return torch.from_numpy(np.ascontiguousarray(a, np.float32)).to(DEV)


def to_dev_u16(a):
    return torch.from_numpy(np.ascontiguousarray(a, np.uint16).view(np.int16)).to(DEV)


def from_dev_f32(t):
    return t.cpu().numpy().astype(np.float32)


def from_dev_u16(t):
    return t.cpu().numpy().view(np.uint16)


class DevState:
    """FP32 master/m/v, BF16 params and R BF16 gradient buffers per segment, on the GPU."""

    def __init__(self, masters, R, exp_avgs=None, exp_avg_sqs=None):
        self.R = R
        self.p = [to_dev_f32(m) for m in masters]
        self.m = ([torch.zeros_like(p) for p in self.p] if exp_avgs is None else [to_dev_f32(a) for a in exp_avgs])
        self.v = ([torch.zeros_like(p) for p in self.p] if exp_avg_sqs is None else [to_dev_f32(a) for a in exp_avg_sqs])
        self.pb = [torch.zeros(p.numel(), dtype=torch.int16, device=DEV) for p in self.p]
        self.g = [[torch.zeros(p.numel(), dtype=torch.int16, device=DEV) for _ in range(R)] for p in self.p]

    def set_grads(self, grads):
        for s, gs in enumerate(grads):
            for r, g in enumerate(gs):
                self.g[s][r].copy_(torch.from_numpy(np.ascontiguousarray(g).view(np.int16)))

    def segments(self, sdp):
        return sdp.segments_from_tensors(
            [(self.p[s], self.m[s], self.v[s], self.pb[s], self.g[s]) for s in range(len(self.p))])

    def host(self):
        st = oracle.State([from_dev_f32(p) for p in self.p], [from_dev_f32(m) for m in self.m],
                          [from_dev_f32(v) for v in self.v], [from_dev_u16(b) for b in self.pb])
        return st

    def clone(self):
        h = self.host()
        c = DevState(h.master, self.R, h.exp_avg, h.exp_avg_sq)
        for s in range(len(c.pb)):
            c.pb[s].copy_(self.pb[s])
            for r in range(self.R):
                c.g[s][r].copy_(self.g[s][r])
        return c


class HostState:
    """The same state in pinned host memory (sdp_host_alloc), viewed as numpy."""

    def __init__(self, sdp, masters, R, exp_avgs=None, exp_avg_sqs=None):
        self.sdp = sdp
        self.R = R
        self.bufs = []
        self.p, self.m, self.v, self.pb, self.g = [], [], [], [], []
        for s, mst in enumerate(masters):
            n = mst.size

            def alloc(dtype):
                b = sdp.HostBuffer(max(n * np.dtype(dtype).itemsize, 16))
                self.bufs.append(b)
                return b.view(dtype, n)
            p = alloc(np.float32)
            p[:] = mst
            m = alloc(np.float32)
            m[:] = 0 if exp_avgs is None else exp_avgs[s]
            v = alloc(np.float32)
            v[:] = 0 if exp_avg_sqs is None else exp_avg_sqs[s]
            pb = alloc(np.uint16)
            pb[:] = 0
            self.p.append(p)
            self.m.append(m)
            self.v.append(v)
            self.pb.append(pb)
            self.g.append([alloc(np.uint16) for _ in range(R)])

    @classmethod
    def allocate(cls, sdp, sizes, R):
        """Pinned arrays of the given segment sizes, contents not initialised."""
        self = cls.__new__(cls)
        self.sdp, self.R, self.bufs = sdp, R, []
        self.p, self.m, self.v, self.pb, self.g = [], [], [], [], []

        def alloc(dtype, n):
            b = sdp.HostBuffer(max(n * np.dtype(dtype).itemsize, 16))
            self.bufs.append(b)
            return b.view(dtype, n)
        for n in sizes:
            self.p.append(alloc(np.float32, n))
            self.m.append(alloc(np.float32, n))
            self.v.append(alloc(np.float32, n))
            self.pb.append(alloc(np.uint16, n))
            self.g.append([alloc(np.uint16, n) for _ in range(R)])
        return self

    def set_grads(self, grads):
        for s, gs in enumerate(grads):
            for r, g in enumerate(gs):
                self.g[s][r][:] = g

    def segments(self):
        return self.sdp.Segments([(self.p[s].ctypes.data, self.m[s].ctypes.data, self.v[s].ctypes.data,
                                   self.pb[s].ctypes.data, [g.ctypes.data for g in self.g[s]], self.p[s].size)
                                  for s in range(len(self.p))])

    def host(self):
        return oracle.State([x.copy() for x in self.p], [x.copy() for x in self.m],
                            [x.copy() for x in self.v], [x.copy() for x in self.pb])

    def close(self):
        """Views keep their buffers alive; dropping the list frees the rest."""
        self.bufs = []


class PageableState(HostState):
    """The same state in ordinary (pageable) numpy arrays, for the staged mode."""

    def __init__(self, sdp, masters, R):
        self.sdp, self.R, self.bufs = sdp, R, []
        self.p = [np.ascontiguousarray(m, np.float32).copy() for m in masters]
        self.m = [np.zeros(x.size, np.float32) for x in self.p]
        self.v = [np.zeros(x.size, np.float32) for x in self.p]
        self.pb = [np.zeros(x.size, np.uint16) for x in self.p]
        self.g = [[np.zeros(x.size, np.uint16) for _ in range(R)] for x in self.p]

    @classmethod
    def allocate(cls, sdp, sizes, R):
        self = cls.__new__(cls)
        self.sdp, self.R, self.bufs = sdp, R, []
        self.p = [np.empty(n, np.float32) for n in sizes]
        self.m = [np.empty(n, np.float32) for n in sizes]
        self.v = [np.empty(n, np.float32) for n in sizes]
        self.pb = [np.empty(n, np.uint16) for n in sizes]
        self.g = [[np.empty(n, np.uint16) for _ in range(R)] for n in sizes]
        return self


# ---------------------------------------------------------------------------
# parity criteria

RTOL = 1e-5          # FP32 master / exp_avg / exp_avg_sq, per element, strict
NORM_RTOL = 1e-6     # gradient norm
BF16_MISMATCH = 1e-4  # fraction of BF16 params that may differ from bf16(oracle master)


_HERE = os.path.dirname(os.path.abspath(__file__))
_PC_LIB = os.path.join(_HERE, "libparity_check.so")
_pc = None


def build_parity_check(force=True):
    if force or not os.path.exists(_PC_LIB):
        tmp = _PC_LIB + ".tmp"
        subprocess.check_call(["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-std=c11", "-o", tmp,
                               os.path.join(_HERE, "parity_check.c"), "-lm"])
        os.replace(tmp, _PC_LIB)
    return _PC_LIB


def pc():
    global _pc
    if _pc is None:
        if not os.path.exists(_PC_LIB):
            build_parity_check(force=False)
        L = ctypes.CDLL(_PC_LIB)
        vp, i64 = ctypes.c_void_p, ctypes.c_int64
        L.pc_compare_f32.restype = None
        L.pc_compare_f32.argtypes = [vp, vp, i64] + [vp] * 5
        L.pc_compare_bf16.restype = None
        L.pc_compare_bf16.argtypes = [vp, vp, i64, vp, vp, vp]
        L.pc_equal.restype = ctypes.c_int
        L.pc_equal.argtypes = [vp, vp, i64]
        _pc = L
    return _pc


def check_f32(got, ref, name):
    """Strict per-element relative error (an oracle zero needs a GPU zero)."""
    got = np.ascontiguousarray(got, np.float32)
    ref = np.ascontiguousarray(ref, np.float32)
    assert got.shape == ref.shape
    worst = ctypes.c_double()
    wi, zm, fm, be = (ctypes.c_int64() for _ in range(4))
    pc().pc_compare_f32(got.ctypes.data, ref.ctypes.data, got.size, ctypes.byref(worst), ctypes.byref(wi),
                        ctypes.byref(zm), ctypes.byref(fm), ctypes.byref(be))
    assert fm.value == 0, f"{name}: finiteness differs on {fm.value} elements"
    assert zm.value == 0, f"{name}: oracle value is 0 but the GPU's is not on {zm.value} elements"
    assert worst.value <= RTOL, (f"{name}: max relative error {worst.value:.3e} > {RTOL} at {wi.value} "
                                 f"(gpu {got[wi.value]!r}, oracle {ref[wi.value]!r})")
    return worst.value, be.value / max(got.size, 1)


def check_bf16(gpu_pb, gpu_master, ref_pb):
    """ref_pb: the oracle's BF16 params, i.e. bf16(oracle master)."""
    gpu_pb = np.ascontiguousarray(gpu_pb, np.uint16)
    own = oracle.bf16(gpu_master)
    assert arrays_equal(gpu_pb, own), "param_bf16 != bf16(GPU master)"
    ref = np.ascontiguousarray(ref_pb, np.uint16)
    d, sg, far = (ctypes.c_int64() for _ in range(3))
    pc().pc_compare_bf16(gpu_pb.ctypes.data, ref.ctypes.data, gpu_pb.size, ctypes.byref(d), ctypes.byref(sg),
                         ctypes.byref(far))
    assert sg.value == 0, "BF16 sign differs"
    assert far.value == 0, "BF16 differs by more than 1 ulp"
    frac = d.value / max(gpu_pb.size, 1)
    assert frac <= BF16_MISMATCH, f"BF16 params differ from bf16(oracle master) on {frac:.2e} of elements"
    return frac


def arrays_equal(a, b) -> bool:
    a = np.ascontiguousarray(a)
    b = np.ascontiguousarray(b)
    if a.nbytes != b.nbytes:
        return False
    return bool(pc().pc_equal(a.ctypes.data, b.ctypes.data, a.nbytes))


def check_norm(got, ref):
    assert abs(got - ref) <= NORM_RTOL * abs(ref), f"norm {got!r} vs oracle {ref!r}"


def check_state(gpu_host: oracle.State, ref: oracle.State):
    stats = {}
    for s in range(len(ref.master)):
        stats[f"master{s}"] = check_f32(gpu_host.master[s], ref.master[s], f"seg{s}.master")
        stats[f"exp_avg{s}"] = check_f32(gpu_host.exp_avg[s], ref.exp_avg[s], f"seg{s}.exp_avg")
        stats[f"exp_avg_sq{s}"] = check_f32(gpu_host.exp_avg_sq[s], ref.exp_avg_sq[s], f"seg{s}.exp_avg_sq")
        stats[f"bf16_{s}"] = check_bf16(gpu_host.param_bf16[s], gpu_host.master[s], ref.param_bf16[s])
    return stats


def states_equal(a: oracle.State, b: oracle.State) -> bool:
    for x, y in ((a.master, b.master), (a.exp_avg, b.exp_avg), (a.exp_avg_sq, b.exp_avg_sq),
                 (a.param_bf16, b.param_bf16)):
        for s in range(len(x)):
            if not arrays_equal(x[s], y[s]):
                return False
    return True


def rand_inputs(sizes, R, steps, seed, sigma=1e-3, outlier_p=0.01):
    masters = [synth.normal_f32(synth.seed(seed, 1, k), n, 0.02) for k, n in enumerate(sizes)]
    grads = [[[synth.to_bf16_bits(synth.normal_f32(synth.seed(seed, 2, t, k, r), n, sigma,
                                                   outlier_p=outlier_p, outlier_scale=100.0))
               for r in range(R)] for k, n in enumerate(sizes)] for t in range(1, steps + 1)]
    return masters, grads


def hp_pair(sdp, **kw):
    return sdp.make_params(**kw), oracle.hparams(**kw)
