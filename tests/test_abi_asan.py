"""The host side of the C ABI under AddressSanitizer (CPU only).

The library is rebuilt with the sanitizer on its host code only (device code
is compiled as usual), loaded into a fresh Python process that preloads the
sanitizer runtime, and the CPU ABI tests (argument validation, workspace
sizing, seed schedule, status strings; no kernel launch) run against it there.
A heap or stack overrun, a use after free or an uninitialised read in the
validation and planning code ends that process with a sanitizer report."""
import glob
import os
import subprocess
import sys
import tempfile

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

# host-only instrumentation: every sanitizer flag is scoped to the host pass
HOST_ASAN = "-Xarch_host -fsanitize=address -Xarch_host -fno-omit-frame-pointer".split()


def _runtime():
    found = sorted(glob.glob("/opt/rocm/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so"))
    return found[-1] if found else None


def _build(out_dir):
    sys.path.insert(0, ROOT)
    from paper_2410_15352_amd import build as B
    objs = []
    for unit, extra in B.UNITS:
        obj = os.path.join(out_dir, unit + ".o")
        cmd = [B.hipcc(), *B.FLAGS, *HOST_ASAN, *extra, "-I", B.INCLUDE, "-c", os.path.join(B.CSRC, unit), "-o", obj]
        subprocess.run(cmd, check=True, capture_output=True)
        objs.append(obj)
    lib = os.path.join(out_dir, "libcompact_asan.so")
    subprocess.run([B.hipcc(), "--offload-arch=gfx950", "-shared", "-fPIC", *HOST_ASAN, *objs, "-o", lib], check=True,
                   capture_output=True)
    return lib


def test_abi_host_code_under_asan():
    rt = _runtime()
    if rt is None:
        pytest.skip("no AddressSanitizer runtime in this toolchain")
    from paper_2410_15352_amd import build as B
    try:
        B.hipcc()
    except RuntimeError:
        pytest.skip("hipcc not available")
    with tempfile.TemporaryDirectory(prefix="compact_asan_") as d:
        lib = _build(d)
        script = (
            "import sys; sys.path.insert(0, %r)\n"
            "from paper_2410_15352_amd import _lib\n"
            "_lib.load(%r)  # every later load() returns this library\n"
            "import pytest\n"
            "sys.exit(pytest.main(['-q', '-p', 'no:cacheprovider', '-m', 'not gpu', %r]))\n"
        ) % (ROOT, lib, os.path.join(ROOT, "tests", "test_abi_cpu.py"))
        env = dict(os.environ, LD_PRELOAD=rt,
                   ASAN_OPTIONS="detect_leaks=0:alloc_dealloc_mismatch=0:abort_on_error=0:exitcode=97")
        res = subprocess.run([sys.executable, "-c", script], cwd=ROOT, env=env, capture_output=True, text=True,
                             timeout=600)
        report = res.stdout[-3000:] + res.stderr[-3000:]
        assert "AddressSanitizer" not in res.stderr, report
        assert res.returncode == 0, report
        assert " passed" in res.stdout, report
