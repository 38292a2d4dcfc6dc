"""GPU parity of the sparse Johnson-Lindenstrauss projection (the ablation's
sparse JL matrices, §5) against the fp64 oracle.

* The stream: compact_projection's integer matrix S equals the oracle's,
  entry for entry, for several (n, r, s) with ragged n, r = 1, odd s and
  s = 64; the Gaussian kind equals compact_pstream.
* Forward (Alg. 1) with P = S / sqrt(s): y and z against the oracle on the
  bf16 path (with and without the workspace) and the fp32 path; y is bitwise
  the Gaussian call's y (the projection only touches z); an input group is
  bitwise its per-projection calls.
* Alg. 3 with the sparse P: M, V and the update against the oracle, fp32 and
  bf16 weights; the batched step is bitwise the per-layer step.  Every
  element of the update on W = 0 against the oracle within the rounding of N
  to bf16, of the (at most s nonzero) terms' sum and of W, for ragged widths,
  rows padded past m (a column slice), wide rows and s = 64 with repeated
  columns.
* The gather-add forward (COMPACT_PROJ_GATHER): z against the oracle element
  by element for s = 1, 3, 8, 16, ragged T and n and r over several column
  chunks; y bitwise the flag-free y; deterministic; a group bitwise its
  per-projection calls; a NaN in x reaches exactly the columns its row of S
  draws; the flag ignored where the persistent GEMM does not run; one token,
  the smallest n of the persistent path, odd r, eight projections, r = n.
"""
import numpy as np
import pytest

from oracle import compact as oc
from oracle.pstream import sparse_jl_raw
from synthetic import bf16_round, fwd_inputs, step_inputs

from gpu_util import BF16_U, assert_elementwise, dev, empty, ld_for, to_dev, to_np, to_np_f32, workspace

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
cp = pytest.importorskip("paper_2410_15352_amd")

TOL = {"f32": 1e-5, "bf16": 2e-2}
CODE = {"f32": 0, "bf16": 1}


@pytest.mark.parametrize("n,r,s,seed", [(7, 5, 3, 1), (1024, 128, 8, (9 << 32) | 77), (2736, 342, 8, 5 << 32),
                                        (13, 1, 4, 2**64 - 1), (100, 37, 64, 123), (5461, 682, 1, 7 << 40),
                                        (333, 64, 2, 42)])
def test_projection_stream_bitwise(n, r, s, seed):
    out = torch.full((n, r), 9.0, dtype=torch.float32, device=dev())
    cp.compact_projection(seed, out, proj=f"sparse-jl:{s}")
    torch.cuda.synchronize()
    assert np.array_equal(out.cpu().numpy().astype(np.float64), sparse_jl_raw(seed, n, r, s))


def test_projection_default_draws_and_gaussian_kind():
    n, r, seed = 300, 48, (3 << 32) | 1
    out = torch.empty(n, r, dtype=torch.float32, device=dev())
    cp.compact_projection(seed, out, proj="sparse-jl")
    g1 = torch.empty(n, r, dtype=torch.float32, device=dev())
    g2 = torch.empty(n, r, dtype=torch.float32, device=dev())
    cp.compact_projection(seed, g1, proj="gaussian")
    cp.compact_pstream(seed, g2)
    torch.cuda.synchronize()
    assert np.array_equal(out.cpu().numpy().astype(np.float64), sparse_jl_raw(seed, n, r, 8))
    assert torch.equal(g1, g2)


SHAPES = [
    (256, 256, 512, 32, "f32"),
    (100, 36, 20, 12, "f32"),
    (300, 200, 136, 40, "bf16"),
    (1000, 1376, 512, 344, "bf16"),
    (513, 512, 1376, 128, "bf16"),
    (777, 1024, 2736, 128, "bf16"),
    (150, 200, 203, 24, "bf16"),
]


def _ids(s):
    return "T{}-n{}-m{}-r{}-{}".format(*s)


# (shape, workspace): the fp32 path has no workspace mode
FWD_CASES = [(sh, ws) for sh in SHAPES for ws in (True, False) if not (sh[4] == "f32" and ws)]


@pytest.mark.parametrize("shape,use_ws", FWD_CASES, ids=[f"{ws}-{_ids(sh)}" for sh, ws in FWD_CASES])
@pytest.mark.parametrize("s", [8, 3])
def test_forward_parity(shape, use_ws, s):
    T, n, m, r, dt = shape
    seed = (13 << 32) | 5
    x, W = fwd_inputs(T, n, m, dt, data_seed=T + n + 1)
    xd, Wd = to_dev(x, dt, ld_for(n, dt)), to_dev(W, dt, ld_for(m, dt))
    y, z = empty(T, m, dt, ld_for(m, dt)), empty(T, r, dt, ld_for(r, dt))
    yg, zg = empty(T, m, dt, ld_for(m, dt)), empty(T, r, dt, ld_for(r, dt))
    ws = workspace(cp.fwd_workspace_bytes(n, m, r, CODE[dt])) if use_ws else None
    cp.compact_fwd(xd, Wd, y, z, seed, proj=f"sparse-jl:{s}", ws=ws)
    cp.compact_fwd(xd, Wd, yg, zg, seed, proj="gaussian", ws=ws)
    torch.cuda.synchronize()
    y_ref, z_ref = oc.ref_fwd(x, W, seed, r, sparse_s=s)
    assert oc.rel_fro(to_np(y), y_ref) <= TOL[dt]
    assert oc.rel_fro(to_np(z), z_ref) <= TOL[dt]
    assert torch.equal(y.contiguous().view(torch.int32 if dt == "f32" else torch.int16),
                       yg.contiguous().view(torch.int32 if dt == "f32" else torch.int16))


def test_group_forward_equals_per_projection():
    T, n, ms, rs = 513, 512, (512, 512, 512), (64, 64, 64)
    seeds = [((j + 3) << 32) | 11 for j in range(3)]
    x, _ = fwd_inputs(T, n, 8, "bf16", data_seed=71)
    W = np.concatenate([fwd_inputs(8, n, m, "bf16", data_seed=72 + j)[1] for j, m in enumerate(ms)], axis=1)
    M, R = sum(ms), sum(rs)
    xd, Wd = to_dev(x, "bf16", ld_for(n, "bf16")), to_dev(W, "bf16", ld_for(M, "bf16"))
    y, z = empty(T, M, "bf16"), empty(T, R, "bf16")
    y1, z1 = empty(T, M, "bf16"), empty(T, R, "bf16")
    cp.compact_fwd_group(xd, Wd, y, z, ms, rs, seeds, proj="sparse-jl",
                         ws=workspace(cp.fwd_group_workspace_bytes(n, ms, rs)))
    mo = ro = 0
    for j, (m, r) in enumerate(zip(ms, rs)):
        cp.compact_fwd(xd, Wd[:, mo:mo + m], y1[:, mo:mo + m], z1[:, ro:ro + r], seeds[j], proj="sparse-jl",
                       ws=workspace(cp.fwd_workspace_bytes(n, m, r)))
        mo += m
        ro += r
    torch.cuda.synchronize()
    assert torch.equal(y.view(torch.int16), y1.view(torch.int16))
    assert torch.equal(z.view(torch.int16), z1.view(torch.int16))
    ro = 0
    for j, r in enumerate(rs):
        _, z_ref = oc.ref_fwd(x, W[:, :1], seeds[j], r, sparse_s=8)
        assert oc.rel_fro(to_np(z)[:, ro:ro + r], z_ref) <= TOL["bf16"]
        ro += r


@pytest.mark.parametrize("shape", SHAPES, ids=_ids)
@pytest.mark.parametrize("t", [1, 3])
def test_step_parity(shape, t):
    _, n, m, r, dt = shape
    s = 8
    seed, lr, b1, b2, eps, alpha = (6 << 32) | 2, 1e-3, 0.9, 0.999, 1e-8, 0.25
    W, G, M, V = step_inputs(n, m, r, dt, t=t, data_seed=n + r + 7)
    Wd = to_dev(W, "f32", ld_for(m, "f32"))
    Gd, Md, Vd = (torch.from_numpy(a.copy()).to(dev()) for a in (G, M, V))
    ws = workspace(cp.step_workspace_bytes(n, m, r, CODE[dt]))
    cp.compact_step(Wd, Gd, Md, Vd, seed, t, lr, b1, b2, eps, alpha, proj="sparse-jl", dtype=dt, ws=ws)
    torch.cuda.synchronize()
    W_ref, M_ref, V_ref, dW_ref = oc.ref_step(W, G, M, V, seed, r, t, lr, b1, b2, eps, alpha, sparse_s=s)
    dW = to_np_f32(Wd).astype(np.float64) - W.astype(np.float64)
    assert oc.rel_fro(Md.cpu().numpy(), M_ref) <= TOL[dt]
    assert oc.rel_fro(Vd.cpu().numpy(), V_ref) <= TOL[dt]
    assert oc.rel_fro(dW, dW_ref) <= (TOL[dt] if dt == "bf16" else 2e-4)
    if dt == "bf16":
        Wb = to_dev(W, "bf16", ld_for(m, "bf16"))
        Gd2, Md2, Vd2 = (torch.from_numpy(a.copy()).to(dev()) for a in (G, M, V))
        cp.compact_step(Wb, Gd2, Md2, Vd2, seed, t, lr, b1, b2, eps, alpha, proj="sparse-jl", dtype="bf16", ws=ws)
        torch.cuda.synchronize()
        assert np.array_equal(to_np_f32(Wb).view(np.uint32), bf16_round(to_np_f32(Wd)).view(np.uint32))


def test_step_batched_equals_per_layer():
    shapes = [(512, 512, 128), (512, 1376, 128), (1376, 512, 344), (300, 200, 40)] * 3
    layers_a, layers_b = [], []
    for i, (n, m, r) in enumerate(shapes):
        W, G, M, V = step_inputs(n, m, r, "bf16", t=2, data_seed=80 + i)
        for lst in (layers_a, layers_b):
            g, mm, v = (torch.from_numpy(a.copy()).to(dev()) for a in (G, M, V))
            lst.append(dict(W=to_dev(W, "bf16", ld_for(m, "bf16")), G=g, M=mm, V=v, seed=((i + 1) << 32) | 9,
                            alpha=0.25))
    cp.compact_step_batched(layers_a, 2, 1e-3, proj="sparse-jl:4",
                            ws=workspace(cp.step_batched_workspace_bytes(layers_a)))
    for L in layers_b:
        n, m = L["W"].shape
        r = L["G"].shape[0]
        cp.compact_step(L["W"], L["G"], L["M"], L["V"], L["seed"], 2, 1e-3, alpha=L["alpha"], proj="sparse-jl:4",
                        ws=workspace(cp.step_workspace_bytes(n, m, r)))
    torch.cuda.synchronize()
    for La, Lb in zip(layers_a, layers_b):
        assert torch.equal(La["M"], Lb["M"]) and torch.equal(La["V"], Lb["V"])
        assert torch.equal(La["W"].view(torch.int16), Lb["W"].view(torch.int16))


# (n, m, r, s, W dtype, ldw): ragged m; rows padded past m; m = 2736; s = 64
# over r = 5 (every row draws each column many times)
UPDATE = [
    (300, 203, 40, 8, "f32", 204),
    (300, 203, 40, 3, "bf16", 208),
    (256, 1000, 128, 8, "bf16", 1032),
    (1024, 2736, 128, 8, "f32", 2736),
    (2736, 1024, 342, 8, "bf16", 1024),
    (100, 37, 5, 64, "bf16", 40),
]


@pytest.mark.parametrize("case", UPDATE, ids=lambda c: "n{}-m{}-r{}-s{}-{}-ld{}".format(*c))
def test_step_update_every_element(case):
    n, m, r, s, wdt, ldw = case
    seed, t, lr, b1, b2, eps, alpha = (11 << 32) | 3, 2, 1e-2, 0.9, 0.999, 1e-8, 0.5
    _, G, M, V = step_inputs(n, m, r, "f32", t=t, data_seed=n + m + s)
    W0 = np.zeros((n, m), np.float32)
    Wd = to_dev(W0, wdt, ldw)
    Gd, Md, Vd = (torch.from_numpy(a.copy()).to(dev()) for a in (G, M, V))
    ws = workspace(cp.step_workspace_bytes(n, m, r, CODE["bf16"]))
    cp.compact_step(Wd, Gd, Md, Vd, seed, t, lr, b1, b2, eps, alpha, proj=f"sparse-jl:{s}", dtype="bf16", ws=ws)
    torch.cuda.synchronize()
    _, _, direction = oc.ref_adam(G, M, V, t, b1, b2, eps)
    _, _, _, change = oc.ref_step(W0, G, M, V, seed, r, t, lr, b1, b2, eps, alpha, sparse_s=s)
    P = oc.projection(seed, n, r, sparse_s=s)
    absprod = lr * alpha * (np.abs(P) @ np.abs(direction))
    # N is rounded to bf16 once (2^-8 of each term); at most s nonzero terms
    # are summed in fp32; the update rounds once more when W is bf16
    assert_elementwise(to_np(Wd), change, absprod, s, bf16_out=(wdt == "bf16"), operand_rel=BF16_U * 1.001,
                       what=f"dW {case}")
    # the columns past m of a padded row are untouched
    if ldw > m:
        full = Wd.as_strided((n, ldw), (Wd.stride(0), 1))
        assert not torch.any(full[:, m:].float() != 0)


# Gather-add forward (COMPACT_PROJ_GATHER): z = sum over features i, in order,
# of x[t][i] * bf16(S[i][c] / sqrt(s)) in fp32.  Shapes the persistent GEMM
# takes (n >= 320): token counts with a partial 64-token block, n with a
# partial 8-feature chunk (333), r over one, two and three 128-column chunks,
# and s = 1, 3 (odd), 8 and 16 (the largest the flag takes).
GATHER_SHAPES = [(300, 512, 512, 128), (1000, 1376, 512, 344), (777, 333, 136, 200), (65, 1024, 2736, 342),
                 (130, 2736, 1024, 342)]


def _bf(rows, cols):
    return empty(rows, cols, "bf16", ld_for(cols, "bf16"))


def _gather_ref(x, seed, r, s):
    P = sparse_jl_raw(seed, x.shape[1], r, s) / np.sqrt(s)
    return x.astype(np.float64) @ P, np.abs(x.astype(np.float64)) @ np.abs(P)


@pytest.mark.parametrize("shape", GATHER_SHAPES, ids=lambda sh: "T{}-n{}-m{}-r{}".format(*sh))
@pytest.mark.parametrize("s", [1, 3, 8, 16])
def test_gather_forward_parity(shape, s):
    T, n, m, r = shape
    seed = (21 << 32) | (n + s)
    x, W = fwd_inputs(T, n, m, "bf16", data_seed=T + 3 * s)
    xd, Wd = to_dev(x, "bf16", ld_for(n, "bf16")), to_dev(W, "bf16", ld_for(m, "bf16"))
    y, z, y2, z2 = _bf(T, m), _bf(T, r), _bf(T, m), _bf(T, r)
    yd, zd = _bf(T, m), _bf(T, r)
    ws = workspace(cp.fwd_workspace_bytes(n, m, r, 1))
    cp.compact_fwd(xd, Wd, y, z, seed, proj=f"sparse-jl:{s}:gather", ws=ws)
    cp.compact_fwd(xd, Wd, yd, zd, seed, proj=f"sparse-jl:{s}", ws=ws)
    cp.compact_fwd(xd, Wd, y2, z2, seed, proj=f"sparse-jl:{s}:gather", ws=ws)
    torch.cuda.synchronize()
    assert torch.equal(y.view(torch.int16), yd.view(torch.int16)), "the flag changed y"
    assert torch.equal(z.view(torch.int16), z2.view(torch.int16)), "gather-add z not deterministic"
    z_ref, absprod = _gather_ref(x, seed, r, s)
    # each term carries P rounded to bf16 (2^-8 of its share) and the sum at
    # most n terms of fp32 rounding
    assert_elementwise(to_np(z), z_ref, absprod, K=n, operand_rel=BF16_U, what="gather-add z")
    assert_elementwise(to_np(zd), z_ref, absprod, K=n, operand_rel=BF16_U, what="MFMA z")


def test_gather_group_equals_per_projection():
    T, n, ms, rs = 333, 1024, (512, 512, 512), (128, 136, 64)
    seeds = [((j + 5) << 32) | 13 for j in range(3)]
    x, _ = fwd_inputs(T, n, 8, "bf16", data_seed=91)
    W = np.concatenate([fwd_inputs(8, n, m, "bf16", data_seed=92 + j)[1] for j, m in enumerate(ms)], axis=1)
    M, R = sum(ms), sum(rs)
    xd, Wd = to_dev(x, "bf16", ld_for(n, "bf16")), to_dev(W, "bf16", ld_for(M, "bf16"))
    y, z = _bf(T, M), _bf(T, R)
    y1, z1 = _bf(T, M), _bf(T, R)
    proj = "sparse-jl:4:gather"
    cp.compact_fwd_group(xd, Wd, y, z, ms, rs, seeds, proj=proj,
                         ws=workspace(cp.fwd_group_workspace_bytes(n, ms, rs)))
    mo = ro = 0
    for j, (m, r) in enumerate(zip(ms, rs)):
        cp.compact_fwd(xd, Wd[:, mo:mo + m], y1[:, mo:mo + m], z1[:, ro:ro + r], seeds[j], proj=proj,
                       ws=workspace(cp.fwd_workspace_bytes(n, m, r)))
        mo += m
        ro += r
    torch.cuda.synchronize()
    assert torch.equal(y.view(torch.int16), y1.view(torch.int16))
    assert torch.equal(z.view(torch.int16), z1.view(torch.int16))
    ro = 0
    for j, r in enumerate(rs):
        z_ref, absprod = _gather_ref(x, seeds[j], r, 4)
        assert_elementwise(to_np(z)[:, ro:ro + r], z_ref, absprod, K=n, operand_rel=BF16_U, what=f"z_{j}")
        ro += r


def test_gather_nan_reaches_only_drawn_columns():
    # the gather path's own semantics: a NaN at x[t][i] reaches z[t][c] only
    # where S[i][c] != 0 (the MFMA path multiplies it by every P[i][c], zeros
    # included), so this also shows that the gather launch computed z
    T, n, m, r, s, seed = 200, 512, 256, 128, 8, (4 << 32) | 9
    x, W = fwd_inputs(T, n, m, "bf16", data_seed=5)
    t0, i0 = 70, 301
    x[t0, i0] = np.nan
    xd, Wd = to_dev(x, "bf16", ld_for(n, "bf16")), to_dev(W, "bf16", ld_for(m, "bf16"))
    y, z, zd = _bf(T, m), _bf(T, r), _bf(T, r)
    ws = workspace(cp.fwd_workspace_bytes(n, m, r, 1))
    cp.compact_fwd(xd, Wd, y, z, seed, proj=f"sparse-jl:{s}:gather", ws=ws)
    cp.compact_fwd(xd, Wd, y, zd, seed, proj=f"sparse-jl:{s}", ws=ws)
    torch.cuda.synchronize()
    zg, zm = to_np(z), to_np(zd)
    drawn = sparse_jl_raw(seed, n, r, s)[i0] != 0
    assert np.array_equal(np.isnan(zg[t0]), drawn)
    assert np.isnan(zm[t0]).all()
    assert np.isfinite(np.delete(zg, t0, axis=0)).all()
    assert np.isnan(to_np(y)[t0]).all()


@pytest.mark.parametrize("n,use_ws", [(200, True), (512, False)])
def test_gather_flag_ignored_off_the_persistent_path(n, use_ws):
    # n < 320 (the fused 8-wave GEMM) or no workspace: z as without the flag
    T, m, r, s, seed = 150, 136, 24, 8, (8 << 32) | 3
    x, W = fwd_inputs(T, n, m, "bf16", data_seed=n)
    xd, Wd = to_dev(x, "bf16", ld_for(n, "bf16")), to_dev(W, "bf16", ld_for(m, "bf16"))
    y, z, y2, z2 = _bf(T, m), _bf(T, r), _bf(T, m), _bf(T, r)
    ws = workspace(cp.fwd_workspace_bytes(n, m, r, 1)) if use_ws else None
    cp.compact_fwd(xd, Wd, y, z, seed, proj=f"sparse-jl:{s}:gather", ws=ws)
    cp.compact_fwd(xd, Wd, y2, z2, seed, proj=f"sparse-jl:{s}", ws=ws)
    torch.cuda.synchronize()
    assert torch.equal(y.view(torch.int16), y2.view(torch.int16))
    assert torch.equal(z.view(torch.int16), z2.view(torch.int16))


@pytest.mark.parametrize("T,ms,rs,s", [(1, (64,), (13,), 2),                       # one token, odd r
                                       (129, (64,) * 7 + (40,), (8,) * 7 + (13,), 5),  # 8 projections
                                       (64, (320,), (320,), 16)])                     # r = n, s at its maximum
def test_gather_edge_cases(T, ms, rs, s):
    n = 320  # the smallest n the persistent GEMM (and so the gather path) takes
    seeds = [((j + 11) << 32) | 7 for j in range(len(ms))]
    x, _ = fwd_inputs(T, n, 8, "bf16", data_seed=T + 5)
    W = np.concatenate([fwd_inputs(8, n, m, "bf16", data_seed=40 + j)[1] for j, m in enumerate(ms)], axis=1)
    M, R = sum(ms), sum(rs)
    xd, Wd = to_dev(x, "bf16", ld_for(n, "bf16")), to_dev(W, "bf16", ld_for(M, "bf16"))
    y, z, y2, z2 = _bf(T, M), _bf(T, R), _bf(T, M), _bf(T, R)
    ws = workspace(cp.fwd_group_workspace_bytes(n, list(ms), list(rs)))
    cp.compact_fwd_group(xd, Wd, y, z, list(ms), list(rs), seeds, proj=f"sparse-jl:{s}:gather", ws=ws)
    cp.compact_fwd_group(xd, Wd, y2, z2, list(ms), list(rs), seeds, proj=f"sparse-jl:{s}", ws=ws)
    torch.cuda.synchronize()
    assert torch.equal(y.view(torch.int16), y2.view(torch.int16))
    ro = 0
    for j, r in enumerate(rs):
        z_ref, absprod = _gather_ref(x, seeds[j], r, s)
        assert_elementwise(to_np(z)[:, ro:ro + r], z_ref, absprod, K=n, operand_rel=BF16_U, what=f"gather z_{j}")
        ro += r
