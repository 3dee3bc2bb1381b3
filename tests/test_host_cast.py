"""The library's host-side BF16 rounding (the parameter-delivery lane) over
every FP32 bit pattern, against the oracle -- bit for bit, NaNs included.
Host code only: runs without a GPU."""
import numpy as np
import pytest


@pytest.fixture(scope="module")
def sdp():
    from paper_2609_34162_amd import sdp as mod
    return mod


def test_host_cast_exhaustive_vs_oracle(orc, sdp):
    chunk = 1 << 27
    base = np.arange(chunk, dtype=np.uint32)
    u = np.empty(chunk, np.uint32)
    got = np.empty(chunk, np.uint16)
    want = np.empty(chunk, np.uint16)
    bad = 0
    for a in range(0, 1 << 32, chunk):
        np.add(base, np.uint32(a), out=u)
        sdp.sdp_cast_bf16_host(None, u.ctypes.data, got.ctypes.data, chunk)
        orc.orc_bf16_array(u.ctypes.data, want.ctypes.data, chunk)
        bad += int(np.count_nonzero(got != want))
    assert bad == 0


def test_host_cast_ragged_and_errors(orc, sdp):
    import oracle
    rng = np.random.default_rng(4)
    for n in (1, 2, 7, 8, 9, 1000003):
        with np.errstate(over="ignore"):   # some values overflow to infinity, on purpose
            x = (rng.normal(0, 1, n) * np.exp2(rng.integers(-130, 128, n))).astype(np.float32)
        y = np.empty(n, np.uint16)
        sdp.sdp_cast_bf16_host(None, x.ctypes.data, y.ctypes.data, n)
        assert np.array_equal(y, oracle.bf16(x))
    with pytest.raises(sdp.SdpError):
        sdp.sdp_cast_bf16_host(None, 0, 0, 5)
