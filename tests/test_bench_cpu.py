"""The benchmark's host arithmetic, without a GPU: the LLaMA-350M workload's
layer shapes (hidden 1024, FFN 2736, 24 blocks, r = n/8, 65536 tokens per
step), the input groups it forms, and the algorithmic flops and bytes per step
that its roofline figures divide by the measured time, each written out here
from the shapes rather than taken from the code under test."""
import pytest

import bench
from synthetic import input_groups, workload

T = 65536
BLOCKS = 24
H, F = 1024, 2736
R_H, R_F = H // 8, F // 8  # 128 and 342


def test_llama350m_layer_shapes():
    wl = workload("llama-350m")
    assert wl.tokens == T and wl.dtype == "bf16"
    assert len(wl.layers) == 7 * BLOCKS
    shapes = [(L.n, L.m, L.r) for L in wl.layers[:7]]
    assert shapes == [(H, H, R_H)] * 4 + [(H, F, R_H)] * 2 + [(F, H, R_F)]
    for b in range(BLOCKS):
        assert [(L.n, L.m, L.r) for L in wl.layers[7 * b:7 * b + 7]] == shapes
    # a distinct projection seed per layer
    assert len({L.seed for L in wl.layers}) == len(wl.layers)


def test_input_groups_share_the_input():
    wl = workload("llama-350m")
    groups = input_groups(wl)
    assert len(groups) == 4 * BLOCKS
    sizes = sorted(len(g) for g in groups[:4])
    assert sizes == [1, 1, 2, 3]  # q|k|v, o, gate|up, down
    for g in groups:
        assert len({wl.layers[i].n for i in g}) == 1
        assert len({wl.layers[i].block for i in g}) == 1
    assert sorted(i for g in groups for i in g) == list(range(len(wl.layers)))
    # without grouping every layer is its own launch
    assert len(input_groups(wl, False)) == len(wl.layers)


def test_algorithmic_work_per_step():
    wl = workload("llama-350m")
    f, b = bench.algorithmic(wl, input_groups(wl))
    # forward: [y | z] = x [W | P] per group, K = n
    fwd = 2 * T * (H * (3 * H + 3 * R_H) + H * (H + R_H) + H * (2 * F + 2 * R_H) + F * (H + R_F))
    dx = 2 * T * (H * 3 * H + H * H + H * 2 * F + F * H)
    ghat = 2 * T * (4 * R_H * H + 2 * R_H * F + R_F * H)
    dec = 2 * (4 * H * R_H * H + 2 * H * R_H * F + F * R_F * H)
    assert f["fwd"] == pytest.approx(BLOCKS * fwd, rel=1e-12)
    assert f["dx"] == pytest.approx(BLOCKS * dx, rel=1e-12)
    assert f["ghat"] == pytest.approx(BLOCKS * ghat, rel=1e-12)
    assert f["dec"] == pytest.approx(BLOCKS * dec, rel=1e-12)
    # the forward and dL/dx are about 90 TFLOP per step together at these shapes
    assert 85e12 < f["fwd"] + f["dx"] + f["ghat"] < 95e12

    # bytes: bf16 operands read once and outputs written once per launch
    def fwd_bytes(n, M, R):
        return 2 * (T * n + n * M + T * M + T * R)

    def dx_bytes(n, M):
        return 2 * (T * M + n * M + T * n)

    fb = fwd_bytes(H, 3 * H, 3 * R_H) + fwd_bytes(H, H, R_H) + fwd_bytes(H, 2 * F, 2 * R_H) + fwd_bytes(F, H, R_F)
    db = dx_bytes(H, 3 * H) + dx_bytes(H, H) + dx_bytes(H, 2 * F) + dx_bytes(F, H)
    assert b["fwd"] == pytest.approx(BLOCKS * fb, rel=1e-12)
    assert b["dx"] == pytest.approx(BLOCKS * db, rel=1e-12)
    # G^: z and dL/do read (bf16), G^ written (fp32); Adam: 22 bytes per r x m
    # element (G^, M, V read; M, V written; N written in bf16); decompression:
    # W read and written (bf16) and N read
    layers = [(H, H, R_H)] * 4 + [(H, F, R_H)] * 2 + [(F, H, R_F)]
    gb = sum(2 * T * (r + m) + 4 * r * m for n, m, r in layers)
    ab = sum(22 * r * m for n, m, r in layers)
    deb = sum(4 * n * m + 2 * r * m for n, m, r in layers)
    assert b["ghat"] == pytest.approx(BLOCKS * gb, rel=1e-12)
    assert b["adam"] == pytest.approx(BLOCKS * ab, rel=1e-12)
    assert b["dec"] == pytest.approx(BLOCKS * deb, rel=1e-12)


def test_more_than_one_gpu_is_refused():
    # the benchmark runs on exactly one GPU: --gpus N > 1 (or a multi-rank
    # launch) prints a JSON error line and exits with status 2 before any GPU work
    import json
    import os
    import subprocess
    import sys
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    for args, env in ((["--gpus", "2"], {}), ([], {"WORLD_SIZE": "4"})):
        p = subprocess.run([sys.executable, os.path.join(root, "bench.py"), *args], capture_output=True, text=True,
                           env={**os.environ, **env}, timeout=120)
        assert p.returncode == 2, p.stderr[-500:]
        line = json.loads(p.stdout.strip().splitlines()[-1])
        assert "one GPU" in line["error"]
