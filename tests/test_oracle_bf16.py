"""The oracle's BF16 rounding over every FP32 bit pattern, against torch's
CPU float32 -> bfloat16 cast (NaNs compared by class: torch returns one
canonical NaN, the oracle keeps the payload's top bits and sets the quiet bit)."""
import numpy as np
import torch


def test_bf16_exhaustive_vs_torch(orc):
    chunk = 1 << 27
    base = np.arange(chunk, dtype=np.uint32)
    u = np.empty(chunk, np.uint32)
    out = np.empty(chunk, np.uint16)
    mismatches = 0
    nan_bad = 0
    for a in range(0, 1 << 32, chunk):
        np.add(base, np.uint32(a), out=u)
        f = u.view(np.float32)
        orc.orc_bf16_array(f.ctypes.data, out.ctypes.data, chunk)
        t = torch.from_numpy(f).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
        diff = np.flatnonzero(out != t)
        if diff.size:
            du = u[diff]
            is_nan = ((du & 0x7f800000) == 0x7f800000) & ((du & 0x007fffff) != 0)
            mismatches += int((~is_nan).sum())
            o = out[diff][is_nan].astype(np.uint32)
            nan_bad += int(np.sum(((o & 0x7f80) != 0x7f80) | ((o & 0x0040) == 0)))
    assert mismatches == 0
    assert nan_bad == 0
