"""Pins for the oracle's Philox generator (Salmon et al., SC'11).

* The generic round code, instantiated at 4x64, must reproduce numpy's
  ``numpy.random.Philox`` (a library implementation of Philox4x64-10).
* The vectorised 4x32 generator must agree with the generic code, and with
  rocRAND's Philox4x32-10 engine (header-only library source compiled here and
  run on the host).
* Output words must be uniform (chi-square over the top byte) and the counter
  layout must give independent words for neighbouring counters.
"""
import os
import shutil
import subprocess

import numpy as np
import pytest

from oracle.pstream import philox4_generic, philox4x32_10

HERE = os.path.dirname(os.path.abspath(__file__))


@pytest.mark.parametrize("key,counter", [
    ((0, 0), (0, 0, 0, 0)),
    ((1, 2), (5, 0, 0, 0)),
    ((0xDEADBEEFCAFEF00D, 0x0123456789ABCDEF), (2**64 - 3, 7, 2**63, 11)),
    ((12345, 67890), (2**40 + 17, 2**33, 0, 2**62)),
])
def test_generic_philox4x64_matches_numpy(key, counter):
    bg = np.random.Philox(key=np.array(key, dtype=np.uint64),
                          counter=np.array(counter, dtype=np.uint64))
    got = [int(v) for v in bg.random_raw(8)]
    # numpy advances the 256-bit counter before each block
    c = sum(int(v) << (64 * i) for i, v in enumerate(counter))
    exp = []
    for blk in (1, 2):
        cc = (c + blk) % (1 << 256)
        words = [(cc >> (64 * i)) & (2**64 - 1) for i in range(4)]
        exp.extend(philox4_generic(words, key, wordbits=64))
    assert got == exp


def test_vectorised_philox4x32_matches_generic():
    rng = np.random.Generator(np.random.PCG64(99))
    c = rng.integers(0, 2**32, size=(4, 64), dtype=np.uint64).astype(np.uint32)
    k = rng.integers(0, 2**32, size=(2, 64), dtype=np.uint64).astype(np.uint32)
    vec = philox4x32_10(c[0], c[1], c[2], c[3], k[0], k[1])
    for t in range(64):
        g = philox4_generic([int(c[i, t]) for i in range(4)], [int(k[0, t]), int(k[1, t])], 32)
        assert tuple(int(vec[i][t]) for i in range(4)) == g


def _compile_rocrand_driver(tmp_path):
    hipcc = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    if not os.path.exists(hipcc) or not os.path.exists("/opt/rocm/include/rocrand/rocrand_kernel.h"):
        pytest.skip("hipcc / rocRAND headers not available")
    exe = str(tmp_path / "rocrand_philox_host")
    subprocess.run([hipcc, "-O1", os.path.join(HERE, "rocrand_philox_host.cpp"), "-o", exe],
                   check=True, capture_output=True)
    return exe


def test_philox4x32_matches_rocrand(tmp_path):
    exe = _compile_rocrand_driver(tmp_path)
    rng = np.random.Generator(np.random.PCG64(7))
    cases = [(1, 0, 0), (0, 0, 0), ((5 << 32) + 3, 0, 4 * 17)]
    for _ in range(40):
        seed = int(rng.integers(0, 2**63)) * 2 + int(rng.integers(0, 2))
        sub = int(rng.integers(0, 2**32))
        off = 4 * int(rng.integers(0, 2**32))
        cases.append((seed, sub, off))
    stdin = "".join(f"{s} {u} {o}\n" for s, u, o in cases)
    out = subprocess.run([exe], input=stdin, capture_output=True, text=True, check=True).stdout
    lines = out.strip().splitlines()
    assert len(lines) == len(cases)
    for (seed, sub, off), line in zip(cases, lines):
        got = tuple(int(v) for v in line.split())
        ctr = off // 4
        w = philox4x32_10(ctr & 0xFFFFFFFF, ctr >> 32, sub & 0xFFFFFFFF, sub >> 32,
                          seed & 0xFFFFFFFF, seed >> 32)
        assert tuple(int(v) for v in w) == got


def test_philox4x32_words_uniform():
    p = np.arange(1 << 16, dtype=np.uint32)[:, None]
    j = np.arange(4, dtype=np.uint32)[None, :]
    words = np.concatenate([w.ravel() for w in philox4x32_10(p, j, 0, 0, 0x1234, 0x5)])
    counts = np.bincount((words >> 24).astype(np.int64), minlength=256)
    expected = words.size / 256
    chi2 = float(((counts - expected) ** 2 / expected).sum())
    # 255 degrees of freedom: mean 255, sd ~22.6; 6 sd margin
    assert chi2 < 255 + 6 * 22.6
    # neighbouring counters give uncorrelated words
    a = philox4x32_10(p[:, 0], 0, 0, 0, 1, 0)[0].astype(np.float64)
    b = philox4x32_10(p[:, 0] + 1, 0, 0, 0, 1, 0)[0].astype(np.float64)
    assert abs(np.corrcoef(a, b)[0, 1]) < 5 / np.sqrt(a.size)
