"""Every output element of the persistent GEMMs at sizes where each workgroup
walks several output tiles, against the fp64 oracle (Alg. 1 and Alg. 2).

With at least three 256 x 256 tiles per compute unit the persistent kernel runs
everything it does at full size: a finished tile's stores overlap the next
tile's K loop, the operand copies run ahead across tile boundaries, and the
walk covers several bands per XCD.  The token counts are not multiples of the
tile (a ragged last row of tiles), and the widths leave ragged last column
tiles (384 z columns, 5472 or 2736 output columns).  The shapes are those of
the LLaMA-350M layers (q|k|v and gate|up input groups, down alone) and the
LLaMA-1B layers of width 5461 (a K that is not a multiple of 8, whose last
16-byte chunk the kernel clears past K; odd output widths, whose last column
goes out alone).

Each element is held to a bound, beside the relative Frobenius error: the
output rounding plus a probabilistic accumulation bound (gpu_util); a wrong
tile, column or K tile anywhere fails it.  The G^ of the backward is checked
the same way on synthetic z (the oracle never sees a GPU value)."""
import numpy as np
import pytest

from oracle import compact as oc
from oracle.pstream import projection
from synthetic import normal_bf16_blocked

from gpu_util import BF16_U, assert_elementwise, dev, empty, ld_for, to_dev, to_np, workspace

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
cp = pytest.importorskip("paper_2410_15352_amd")

TOL = 2e-2
SEEDS = tuple(((k + 1) << 32) | 5 for k in range(3))
# (tokens, n, widths, ranks): the LLaMA-350M input groups
FWD = [
    (16384 + 77, 1024, (1024, 1024, 1024), (128, 128, 128)),
    (16384 + 77, 1024, (2736, 2736), (128, 128)),
    (32768 + 77, 2736, (1024,), (342,)),
    # LLaMA-1B widths of 5461: K % 8 != 0 (down), odd output widths (gate, z of down)
    (16384 + 77, 5461, (2048,), (1365,)),
    (8192 + 77, 2048, (5461,), (512,)),
]
# K edges of the K loop: from 18 32-deep K tiles on, an even number of them,
# or an odd number from 41 on (padded by a zero K tile), runs A in 64-deep
# slots, the rest in 32-deep stages; each with K % 8 != 0 and odd widths.
# (K = 5461 and 5472 above: 171 K tiles, padded.)
FWD_K = [
    (22016 + 77, 320, (2048,), (40,)),      # K = 320: the fewest K tiles (10, even)
    (22016 + 77, 352, (2048,), (45,)),      # 11 K tiles (odd), odd z width
    (22016 + 77, 571, (2048,), (72,)),      # K % 8 != 0, 18 K tiles: the fewest in 64-deep slots
    (32768 + 77, 1021, (1000,), (512,)),    # K % 8 != 0, 32 K tiles (even)
    (32768 + 77, 1053, (1000,), (257,)),    # K % 8 != 0, 33 K tiles (odd), odd z width
]
# dx = dL/do W^T has n output columns: more tokens for three tiles per CU
DX = [
    (49152 + 77, 1024, (1024, 1024, 1024), (128, 128, 128)),
    (32768 + 77, 2736, (1024,), (342,)),
    (49152 + 77, 1024, (2736, 2736), (128, 128)),
    (12288 + 77, 5461, (2048,), (1365,)),     # odd output width (dL/dx of down)
    (24576 + 77, 2048, (5461,), (512,)),      # K % 8 != 0 (dL/dx of gate)
    (49152 + 77, 1021, (1021,), (128,)),      # K % 8 != 0 with 32 K tiles (even), odd output width
    (24576 + 77, 2048, (1053,), (128,)),      # K % 8 != 0 with 33 K tiles (odd)
]


def _ids(c):
    return "T{}-n{}-m{}-r{}".format(c[0], c[1], "+".join(map(str, c[2])), "+".join(map(str, c[3])))


def _cus():
    return torch.cuda.get_device_properties(0).multi_processor_count


def _tiles(T, cols):
    return -(-T // 256) * sum(-(-c // 256) for c in cols)


def _rows_np(t, r0, r1):
    return to_np(t[r0:r1])


CHUNK = 8192


@pytest.mark.parametrize("case", FWD + FWD_K, ids=_ids)
def test_multitile_forward_every_element(case):
    T, n, ms, rs = case
    M, R = sum(ms), sum(rs)
    assert _tiles(T, (M, R)) >= 3 * _cus(), "the case must give every compute unit three tiles or more"
    x = normal_bf16_blocked(T, n, seed=71 + n)
    Ws = [normal_bf16_blocked(n, m, seed=72 + 10 * k + m, scale=0.02) for k, m in enumerate(ms)]
    xd = to_dev(x, "bf16", ld_for(n, "bf16"))
    Wd = to_dev(np.concatenate(Ws, axis=1), "bf16", ld_for(M, "bf16"))
    y = empty(T, M, "bf16", ld_for(M, "bf16"), fill=float("nan"))
    z = empty(T, R, "bf16", ld_for(R, "bf16"), fill=float("nan"))
    ws = workspace(cp.fwd_group_workspace_bytes(n, ms, rs))
    ws.fill_(0xFF)
    seeds = SEEDS[:len(ms)]
    if len(ms) > 1:
        cp.compact_fwd_group(xd, Wd, y, z, ms, rs, seeds, ws=ws)
    else:
        cp.compact_fwd(xd, Wd, y, z, seeds[0], ws=ws)
    torch.cuda.synchronize()
    Ps = [projection(s, n, r) for s, r in zip(seeds, rs)]
    num = {"y": 0.0, "z": 0.0}
    den = {"y": 0.0, "z": 0.0}
    for r0 in range(0, T, CHUNK):
        r1 = min(T, r0 + CHUNK)
        xc = x[r0:r1].astype(np.float64)
        ax = np.abs(xc)
        yc, zc = _rows_np(y, r0, r1), _rows_np(z, r0, r1)
        mo = ro = 0
        for k, (m, r) in enumerate(zip(ms, rs)):
            y_ref, z_ref = xc @ Ws[k].astype(np.float64), xc @ Ps[k]
            assert_elementwise(yc[:, mo:mo + m], y_ref, ax @ np.abs(Ws[k].astype(np.float64)), n,
                               what=f"y[{k}] rows {r0}..{r1}")
            # P is rounded to bf16 once before the product (one more 2^-8)
            assert_elementwise(zc[:, ro:ro + r], z_ref, ax @ np.abs(Ps[k]), n, operand_rel=BF16_U * 1.001,
                               what=f"z[{k}] rows {r0}..{r1}")
            num["y"] += float(np.sum((yc[:, mo:mo + m] - y_ref) ** 2))
            den["y"] += float(np.sum(y_ref ** 2))
            num["z"] += float(np.sum((zc[:, ro:ro + r] - z_ref) ** 2))
            den["z"] += float(np.sum(z_ref ** 2))
            mo += m
            ro += r
    for k in num:
        assert (num[k] / den[k]) ** 0.5 <= TOL


@pytest.mark.parametrize("case", DX, ids=_ids)
def test_multitile_dx_every_element(case):
    T, n, ms, rs = case
    M = sum(ms)
    assert _tiles(T, (n,)) >= 3 * _cus()
    dy = normal_bf16_blocked(T, M, seed=81 + M, scale=0.01)
    W = normal_bf16_blocked(n, M, seed=82 + n, scale=0.02)
    dyd = to_dev(dy, "bf16", ld_for(M, "bf16"))
    Wd = to_dev(W, "bf16", ld_for(M, "bf16"))
    dx = empty(T, n, "bf16", ld_for(n, "bf16"), fill=float("nan"))
    ws = workspace(cp.bwd_group_workspace_bytes(T, n, ms, rs))
    ws.fill_(0xFF)
    cp.compact_bwd_group(dyd, Wd, None, dx, None, ms, rs, ws=ws)
    torch.cuda.synchronize()
    W64 = W.astype(np.float64)
    aW = np.abs(W64)
    num = den = 0.0
    for r0 in range(0, T, CHUNK):
        r1 = min(T, r0 + CHUNK)
        dyc = dy[r0:r1].astype(np.float64)
        ref = dyc @ W64.T
        got = _rows_np(dx, r0, r1)
        assert_elementwise(got, ref, np.abs(dyc) @ aW.T, M, what=f"dx rows {r0}..{r1}")
        num += float(np.sum((got - ref) ** 2))
        den += float(np.sum(ref ** 2))
    assert (num / den) ** 0.5 <= TOL


# G^ cases: the forward groups, plus launches on the 384 x 128 tiles (every
# projection of the launch with 256 < r, no more padding than 128-row tiles
# and not a fit for 256-row ones): a group of two such projections; and on
# the 256 x 256 tiles: r = 512 and 256 (LLaMA-1B at n/4 and n/8), a group of
# both, r = 682 (LLaMA-1B's down at n/8), and r >= 1024 padded past what
# 128-row tiles would (1365 among the forward groups; 1100 with a ragged m)
GHAT = FWD + [
    (16384 + 77, 1024, (1024, 520), (344, 300)),
    (8192 + 77, 5461, (2048,), (682,)),
    (16384 + 77, 2048, (2048, 2048, 2048), (512, 512, 512)),
    (8192 + 77, 2048, (2048, 1000), (256, 512)),
    (4096 + 77, 2048, (700,), (1100,)),
]


@pytest.mark.parametrize("case", GHAT, ids=_ids)
def test_multitile_ghat_every_element(case):
    # G^_j = z_j^T dL/do_j over all tokens (split-K, fp32 partials summed in a
    # fixed order): every element against the exact sum
    T, n, ms, rs = case
    M, R = sum(ms), sum(rs)
    dy = normal_bf16_blocked(T, M, seed=91 + M, scale=0.01)
    z = normal_bf16_blocked(T, R, seed=92 + R, scale=float(np.sqrt(n / rs[0])))
    dyd = to_dev(dy, "bf16", ld_for(M, "bf16"))
    zd = to_dev(z, "bf16", ld_for(R, "bf16"))
    Gs = [torch.full((r, m), float("nan"), dtype=torch.float32, device=dev()) for m, r in zip(ms, rs)]
    ws = workspace(cp.bwd_group_workspace_bytes(T, n, ms, rs))
    ws.fill_(0xFF)
    cp.compact_bwd_group(dyd, None, zd, None, Gs, ms, rs, ws=ws)
    torch.cuda.synchronize()
    mo = ro = 0
    for k, (m, r) in enumerate(zip(ms, rs)):
        z64, dy64 = z[:, ro:ro + r].astype(np.float64), dy[:, mo:mo + m].astype(np.float64)
        G_ref = z64.T @ dy64
        got = Gs[k].cpu().numpy().astype(np.float64)
        # fp32 output: no output rounding; T products and up to 256 partials summed
        assert_elementwise(got, G_ref, np.abs(z64).T @ np.abs(dy64), T + 256, bf16_out=False, what=f"G^[{k}]")
        assert oc.rel_fro(got, G_ref) <= TOL
        mo += m
        ro += r
