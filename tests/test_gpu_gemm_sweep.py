"""Seeded sweep of shapes through the persistent GEMM (forward and dL/dx),
every output element against the fp64 oracle (Alg. 1 and Alg. 2).

The shapes are drawn at random (fixed seed) over the ranges where the
kernel's structure changes: K from the smallest accepted (320) to a few
thousand, so that the K loop runs in 32-deep stages (fewer than 18 K tiles,
or an odd number below 41) or with A in 64-deep slots (an even number from
18 on, or an odd number from 41 on, padded by a zero K tile); K % 8 != 0
(the last 16-byte chunk of each row cleared past K, with NaN in the row
padding of the A operand, which must not reach the output); odd output
widths; and token counts from one row to eleven row tiles (one tile per
workgroup here; several per workgroup are covered by test_gpu_multitile).
Each element is held to the probabilistic accumulation bound of gpu_util."""
import numpy as np
import pytest

from oracle.pstream import projection
from synthetic import normal_bf16_blocked

from gpu_util import BF16_U, assert_elementwise, empty, ld_for, to_dev, to_np, workspace

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
cp = pytest.importorskip("paper_2410_15352_amd")


def _k_values():
    # every K-loop regime at least once, then random K
    fixed = [320, 321, 544, 545, 571, 576, 1053, 1280, 1300, 1311, 1312, 2055]
    rng = np.random.default_rng(20261202)
    return fixed + [int(k) for k in rng.integers(320, 2600, size=8)]


def _cases(kind):
    rng = np.random.default_rng({"fwd": 11, "dx": 12}[kind])
    out = []
    for i, K in enumerate(_k_values()):
        T = int(rng.choice([1, 37, 256, 700, 1333, 2600]))
        width = int(rng.integers(1, 1400))
        if i % 3 == 0:
            width |= 1  # odd output width
        r = int(rng.integers(1, min(K, 300) + 1))
        out.append((T, K, width, r))
    return out


def _ids(c):
    return "T{}-K{}-w{}-r{}".format(*c)


def _nan_padding(t, cols, ld):
    """Fill the row padding (columns cols .. ld - 1) of the view's buffer with NaN."""
    if ld > cols:
        full = t.as_strided((t.shape[0], ld), (ld, 1))
        full[:, cols:] = float("nan")


@pytest.mark.parametrize("case", _cases("fwd"), ids=_ids)
def test_forward_sweep(case):
    T, n, m, r = case
    x = normal_bf16_blocked(T, n, seed=1000 + n)
    W = normal_bf16_blocked(n, m, seed=2000 + m, scale=0.02)
    seed = (n << 20) | m
    xd = to_dev(x, "bf16", ld_for(n, "bf16"))
    _nan_padding(xd, n, ld_for(n, "bf16"))
    Wd = to_dev(W, "bf16", ld_for(m, "bf16"))
    y = empty(T, m, "bf16", ld_for(m, "bf16"), fill=float("nan"))
    z = empty(T, r, "bf16", ld_for(r, "bf16"), fill=float("nan"))
    ws = workspace(cp.fwd_workspace_bytes(n, m, r))
    ws.fill_(0xFF)
    cp.compact_fwd(xd, Wd, y, z, seed, ws=ws)
    torch.cuda.synchronize()
    x64 = x.astype(np.float64)
    ax = np.abs(x64)
    P = projection(seed, n, r)
    W64 = W.astype(np.float64)
    assert_elementwise(to_np(y), x64 @ W64, ax @ np.abs(W64), n, what="y")
    assert_elementwise(to_np(z), x64 @ P, ax @ np.abs(P), n, operand_rel=BF16_U * 1.001, what="z")


@pytest.mark.parametrize("case", _cases("dx"), ids=_ids)
def test_dx_sweep(case):
    # dx = dL/do W^T: K = m (the sweep's K), output width n
    T, m, n, r = case
    dy = normal_bf16_blocked(T, m, seed=3000 + m, scale=0.01)
    W = normal_bf16_blocked(n, m, seed=4000 + n, scale=0.02)
    dyd = to_dev(dy, "bf16", ld_for(m, "bf16"))
    _nan_padding(dyd, m, ld_for(m, "bf16"))
    Wd = to_dev(W, "bf16", ld_for(m, "bf16"))
    dx = empty(T, n, "bf16", ld_for(n, "bf16"), fill=float("nan"))
    ws = workspace(cp.bwd_group_workspace_bytes(T, n, (m,), (min(r, n),)))
    ws.fill_(0xFF)
    cp.compact_bwd_group(dyd, Wd, None, dx, None, (m,), (min(r, n),), ws=ws)
    torch.cuda.synchronize()
    dy64, W64 = dy.astype(np.float64), W.astype(np.float64)
    assert_elementwise(to_np(dx), dy64 @ W64.T, np.abs(dy64) @ np.abs(W64).T, m, what="dx")
