"""The gfx950 kernels' register and scratch use, from the compiler's own
resource report (hipcc cross-compiles here; no GPU needed).

Every kernel must run without scratch memory: a call stack or a spill puts
the kernel's waves on scratch, which caps the waves in flight, and such a
build of the norm pass and the fused update ran three to four times slower.
The norm passes of the workloads' rank counts must keep full occupancy
(8 waves per SIMD); the fused update runs under a residency cap of 10
one-wave blocks per compute unit, so its limit is 4 waves per SIMD.
"""
import os
import re
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "paper_2609_34162_amd", "csrc", "sdp_kernels.hip")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")


@pytest.fixture(scope="module")
def report(tmp_path_factory):
    if not os.path.exists(HIPCC) and not shutil.which("hipcc"):
        pytest.skip("hipcc not available")
    out = tmp_path_factory.mktemp("kres") / "k.o"
    cmd = [HIPCC, "--offload-arch=gfx950", "-O3", "-std=c++17", "-Xclang", "-target-feature", "-Xclang",
           "-packed-fp32-ops", "-I", os.path.join(ROOT, "include"), "-I", os.path.dirname(SRC), "-c", SRC,
           "-o", str(out), "-Rpass-analysis=kernel-resource-usage"]
    text = subprocess.run(cmd, capture_output=True, text=True, check=True).stderr
    kernels = {}
    name = None
    for line in text.splitlines():
        m = re.search(r"Function Name: (\S+)", line)
        if m:
            name = m.group(1)
            kernels[name] = {}
            continue
        m = re.search(r"(VGPRs|ScratchSize \[bytes/lane\]|Occupancy \[waves/SIMD\]): (\d+)", line)
        if m and name:
            kernels[name][m.group(1).split()[0]] = int(m.group(2))
    assert kernels, "no resource report"
    return kernels


def test_no_kernel_uses_scratch(report):
    bad = {k: v["ScratchSize"] for k, v in report.items() if v.get("ScratchSize", 0) != 0}
    assert not bad, f"kernels with scratch: {bad}"


@pytest.mark.parametrize("R", [1, 2, 4, 8])
@pytest.mark.parametrize("store", [0, 1])
def test_norm_pass_full_occupancy(report, R, store):
    name = f"_ZN3sdp12_GLOBAL__N_115k_norm_partialsILi{R}ELb{store}EEEvNS_8NormArgsE"
    assert report[name]["Occupancy"] == 8, report[name]


@pytest.mark.parametrize("R,cached", [(1, 1), (2, 0), (4, 0), (8, 0)])
def test_update_fits_its_residency_cap(report, R, cached):
    name = f"_ZN3sdp12_GLOBAL__N_18k_updateILi{R}ELb{cached}EEEvNS_10UpdateArgsE"
    assert report[name]["Occupancy"] >= 4, report[name]
