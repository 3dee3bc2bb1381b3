"""The seeded input generator: determinism, slicing, distribution (no GPU)."""
import os
import subprocess
import sys

import numpy as np

import synth
from synth import configs


def test_slices_regenerate_bit_identically():
    s = synth.seed(1, 0, 3, 2, synth.KIND_GRAD)
    full = synth.normal_f32(s, 100003, 1e-3, outlier_p=0.01, outlier_scale=100.0)
    for a, b in ((0, 1), (1, 2), (5, 1000), (99999, 100003), (4096, 70001)):
        part = synth.normal_f32(s, b - a, 1e-3, start=a, outlier_p=0.01, outlier_scale=100.0)
        assert np.array_equal(part.view(np.uint32), full[a:b].view(np.uint32))
    idx = np.array([0, 1, 2, 77, 100002, 5000, 5000])
    at = synth.normal_f32_at(s, idx, 1e-3, 0.01, 100.0)
    assert np.array_equal(at.view(np.uint32), full[idx].view(np.uint32))


def test_thread_count_independent(tmp_path):
    code = ("import sys; sys.path.insert(0, %r); import synth, numpy as np;"
            "x = synth.normal_f32(synth.seed(4, 4), 200001, 0.02);"
            "sys.stdout.write(str(int(np.bitwise_xor.reduce(x.view(np.uint32)))))"
            % os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
    outs = set()
    for nt in ("1", "3", "8"):
        env = dict(os.environ, OMP_NUM_THREADS=nt)
        outs.add(subprocess.check_output([sys.executable, "-c", code], env=env).decode())
    assert len(outs) == 1


def test_distribution():
    x = synth.normal_f32(synth.seed(2, 2), 1 << 22, 1.0).astype(np.float64)
    n = x.size
    assert abs(x.mean()) < 5 / np.sqrt(n)
    assert abs(x.var() - 1) < 5 * np.sqrt(2 / n)
    assert abs(np.mean(x ** 4) - 3) < 0.05          # normal kurtosis
    assert abs(np.mean(np.abs(x) > 3) - 0.0026998) < 0.0003
    u = synth.raw_u32(synth.seed(2, 3), 0, 1 << 18)
    counts = np.bincount(u >> 24, minlength=256)
    expected = u.size / 256
    chi2 = np.sum((counts - expected) ** 2 / expected)
    assert chi2 < 255 + 6 * np.sqrt(2 * 255)


def test_outlier_fraction():
    s = synth.seed(9, 9)
    base = synth.normal_f32(s, 1 << 20, 1e-3)
    scaled = synth.normal_f32(s, 1 << 20, 1e-3, outlier_p=0.01, outlier_scale=100.0)
    ratio = scaled.astype(np.float64) / np.where(base == 0, 1, base)
    frac = np.mean(np.abs(ratio - 100.0) < 1e-3)
    assert abs(frac - 0.01) < 0.001
    assert np.all((np.abs(ratio - 1.0) < 1e-6) | (np.abs(ratio - 100.0) < 1e-3) | (base == 0))


def test_seeds_differ_per_field():
    seen = set()
    for f in [(0, 0, 1, 0, 1), (0, 0, 1, 1, 1), (0, 0, 2, 0, 1), (0, 1, 1, 0, 1),
              (1, 0, 1, 0, 1), (0, 0, 1, 0, 0)]:
        seen.add(synth.seed(*f))
    assert len(seen) == 6


def test_workload_shapes():
    """Parameter counts of the five layer-shaped workloads."""
    n = [w.numel for w in configs.WORKLOADS]
    assert n == [1048576, 192946176, 330311680, 14768291840, 877674496]
    assert [w.ranks for w in configs.WORKLOADS] == [2, 4, 4, 2, 8]
    assert [len(w.segments) for w in configs.WORKLOADS] == [1, 1, 1, 42, 1]
    for w in configs.WORKLOADS:
        assert w.chunk % configs.NORM_TILE == 0


def test_bf16_gradients_use_library_cast():
    w = configs.workload(0)
    g = synth.grad_bf16(w, 0, 1, 0)
    import torch
    f = synth.normal_f32(synth.grad_seed(w, 0, 1, 0), w.numel, w.sigma)
    t = torch.from_numpy(f).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(g, t)
