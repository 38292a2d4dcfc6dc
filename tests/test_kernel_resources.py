"""Register budget of the persistent kernels (CPU only: a compile, no launch).

The persistent GEMM and G^ kernels run one wave per SIMD and keep their
accumulators in the accumulation registers, the decompression runs four
workgroups per CU in at most 128 registers per lane; any VGPR spill or private
(scratch) array inside them turns into scratch-memory traffic whose waits
share the vector-memory counter with the operand copies, and each such wait
drains every copy in flight.  The unit is compiled as build.py compiles
it, with the compiler's resource-usage remarks, and every kernel of the unit
must use no scratch memory and spill no VGPR."""
import os
import re
import subprocess
import sys
import tempfile

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _remarks(unit):
    sys.path.insert(0, ROOT)
    from paper_2410_15352_amd import build as B
    try:
        hipcc = B.hipcc()
    except RuntimeError:
        pytest.skip("hipcc not available")
    extra = dict(B.UNITS)[unit]
    with tempfile.TemporaryDirectory(prefix="compact_res_") as d:
        cmd = [hipcc, *B.FLAGS, *extra, "-I", B.INCLUDE, "-c", os.path.join(B.CSRC, unit), "-o",
               os.path.join(d, "u.o"), "-Rpass-analysis=kernel-resource-usage"]
        res = subprocess.run(cmd, capture_output=True, text=True, cwd=d)
    assert res.returncode == 0, res.stderr[-2000:]
    kernels, cur = {}, None
    for line in res.stderr.splitlines():
        m = re.search(r"Function Name: (\S+)", line)
        if m:
            cur = m.group(1)
            kernels[cur] = {}
            continue
        m = re.search(r"remark:\s+([A-Za-z ]+?)(?: \[[^\]]*\])?: (\d+) \[", line)
        if m and cur is not None:
            kernels[cur][m.group(1).strip()] = int(m.group(2))
    return kernels


def test_persistent_kernels_use_no_scratch():
    kernels = _remarks("kernels_w4.hip")
    names = [k for k in kernels if "k_gemm_w4" in k or "k_ghat_w4" in k or "k_dec_w4" in k]
    assert len([k for k in names if "k_gemm_w4" in k]) == 16, sorted(kernels)
    assert len([k for k in names if "k_ghat_w4" in k]) == 3, sorted(kernels)
    for k in names:
        r = kernels[k]
        assert r.get("ScratchSize") == 0, (k, r)
        assert r.get("VGPRs Spill") == 0, (k, r)
