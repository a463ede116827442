"""Every gfx950 kernel must run without private (scratch) memory or VGPR
spills: a local array left in scratch turned the expert kernels' stores
into tens of MB of extra HBM writes per launch.  SGPR spills are allowed
while the scratch size stays zero: the compiler then parks them in VGPR
lanes, which costs no memory traffic.  Compiles each HIP source with
hipcc's resource-usage remarks (CPU only, no GPU needed)."""
import os
import re
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2609_33614_amd", "csrc")
HIPCC = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
SOURCES = sorted(f for f in os.listdir(CSRC)
                 if f.endswith(".hip") and "__global__" in open(os.path.join(CSRC, f)).read())


@pytest.mark.skipif(not os.path.exists(HIPCC), reason="hipcc missing")
@pytest.mark.parametrize("src", SOURCES)
def test_no_scratch_or_spills(src, tmp_path):
    cmd = [HIPCC, "--offload-arch=gfx950", "-O3", "-std=c++17", "-Xclang", "-target-feature", "-Xclang",
           "-packed-fp32-ops", "-I", os.path.join(ROOT, "include"), "--cuda-device-only", "-c",
           os.path.join(CSRC, src), "-o", str(tmp_path / "k.o"), "-Rpass-analysis=kernel-resource-usage"]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-2000:]
    kernels, cur = {}, None
    for line in r.stderr.splitlines():
        m = re.search(r"remark: (.*?) \[-Rpass", line)
        if not m:
            continue
        t = m.group(1)
        if t.startswith("Function Name:"):
            cur = t.split(":", 1)[1].strip()
            kernels[cur] = {}
        elif cur and ":" in t:
            k, v = t.split(":", 1)
            kernels[cur][k.strip()] = v.strip()
    assert kernels, "no kernels reported"
    for name, info in kernels.items():
        assert info.get("ScratchSize [bytes/lane]") == "0", f"{name} uses scratch: {info}"
        assert info.get("VGPRs Spill") == "0", f"{name} spills VGPRs: {info}"
