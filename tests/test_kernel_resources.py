"""Register budgets of the GEMM kernels, from the compiler's own report.

Every prefill and decode kernel the library builds must fit its registers
without spilling vector registers to scratch memory: a spill turns the
K loop's register-held accumulators and fragments into memory traffic (one
flavour of the 320 x 256 prefill tile once spilled 150 registers after an
epilogue change, and its step ran 14 % slower).  The sources are compiled for
gfx950 to device assembly (no GPU needed) and the kernel descriptors'
vgpr_spill_count read back."""
import os
import re
import subprocess

import pytest

from paper_2406_18832_amd import build_lib

CSRC = build_lib.CSRC


def kernel_resources(src, tmp_path):
    out = tmp_path / (os.path.basename(src) + ".s")
    cmd = [build_lib.hipcc(), *[f for f in build_lib.HIPCC_FLAGS if f not in ("-shared", "-fPIC")],
           "--cuda-device-only", "-S", src, "-o", str(out)]
    run = subprocess.run(cmd, capture_output=True, text=True, timeout=600)
    assert run.returncode == 0, run.stderr[-3000:]
    text = out.read_text()
    res = {}
    for m in re.finditer(r"\.name:\s+(\S+)\n(.*?)(?=\n  - |\n\.end_amdgpu_metadata)", text, re.S):
        body = m.group(2)

        def field(key):
            f = re.search(r"\." + key + r":\s+(\d+)", body)
            return int(f.group(1)) if f else None
        res[m.group(1)] = dict(vgpr=field("vgpr_count"), spill=field("vgpr_spill_count"))
    return res


@pytest.mark.timeout(900)
@pytest.mark.parametrize("src", ["ot_prefill.hip", "ot_decode.hip"])
def test_gemm_kernels_do_not_spill(src, tmp_path):
    res = kernel_resources(os.path.join(CSRC, src), tmp_path)
    gemm = {k: v for k, v in res.items() if "qgemm" in k}
    assert gemm, f"no GEMM kernels found in {src}"
    spilled = {k: v for k, v in gemm.items() if v["spill"] is None or v["spill"] > 0}
    assert not spilled, f"kernels spilling vector registers: {spilled}"
