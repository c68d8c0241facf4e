"""Build-time guards for the kernels that hand registers between inline asm and compiled code.

The grouped GEMMs load their token-row fragments into registers with inline asm the compiler does
not track and read them only after an explicit wait; that is sound only while the compiler keeps the
values in the registers the loads write, i.e. while the kernels neither spill nor use scratch.  The
resource report of the gfx950 build must show no scratch and no spilled registers for them.
"""
import os
import re
import shutil
import subprocess

import pytest

from paper_2606_21868_amd import build


@pytest.mark.skipif(not (shutil.which(build.HIPCC) or os.path.exists(build.HIPCC)), reason="hipcc not installed")
def test_grouped_gemm_kernels_keep_their_registers(tmp_path):
    src = os.path.join(build.CSRC, "grouped_gemm.hip")
    r = subprocess.run([build.HIPCC, *build.HIP_FLAGS, "--cuda-device-only", "-c", src, "-o", str(tmp_path / "g.o"),
                        "-Rpass-analysis=kernel-resource-usage"], stdout=subprocess.PIPE, stderr=subprocess.STDOUT,
                       text=True, timeout=600)
    assert r.returncode == 0, r.stdout[-2000:]
    # remarks come in blocks: "Function Name: <kernel>" then its resource lines
    blocks = re.split(r"remark: Function Name: ", r.stdout)[1:]
    seen = 0
    for b in blocks:
        name = b.split()[0]
        if "grouped_kernel" not in name:
            continue
        seen += 1
        fields = dict(re.findall(r"remark:\s+([A-Za-z ]+?)(?: \[[^\]]*\])?: (\d+)", b))
        assert int(fields["ScratchSize"]) == 0, (name, fields)
        assert int(fields["VGPRs Spill"]) == 0 and int(fields["SGPRs Spill"]) == 0, (name, fields)
        assert int(fields["VGPRs"]) <= 256, (name, fields)
    assert seen == 2, r.stdout[-2000:]
