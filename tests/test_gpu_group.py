"""GPU checks of compact_fwd_group: projections that share one input (q, k, v of
attention; gate and up of the MLP), each with its own seed and rank.

* The grouped call is bitwise equal to compact_fwd on each column slice (the
  same GEMM with the same K order), with and without the workspace, on shapes
  the persistent kernel takes and on ragged ones it does not.
* Each projection matches the fp64 oracle's forward (Alg. 1) within the bf16
  tolerance.
* The backward of a group through compact_bwd on the concatenated weight and
  the column slices: dx equals the sum over projections of the oracle's
  dL/do_j W_j^T, and each G^_j matches the oracle.
* compact_bwd_group (one dx GEMM, one G^ launch for all projections): the same
  oracle checks on every group shape (including fewer tokens than splits and a
  single projection whose rank spans several row tiles), dx bitwise equal to
  compact_bwd over the concatenated weight, each G^_j within 1e-5 of the
  per-slice call (the token splits differ), dx-only / G^-only calls and zero
  tokens.
"""
import numpy as np
import pytest

from oracle import compact as oc
from synthetic import bwd_inputs, fwd_inputs

from gpu_util import dev, empty, ld_for, to_dev, to_np, workspace

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
cp = pytest.importorskip("paper_2410_15352_amd")

TOL = 2e-2

# (tokens, n, ms, rs): persistent-kernel shapes (n >= 320, even widths) and
# ragged ones that run per projection
GROUPS = [
    (513, 512, (512, 512, 512), (128, 128, 128)),      # q, k, v
    (777, 1024, (1376, 1376), (128, 128)),             # gate, up
    (300, 1024, (256, 512), (64, 96)),                 # mixed widths
    (300, 200, (136, 72), (40, 24)),                   # K < 320: per projection
    (129, 512, (512, 203), (64, 30)),                  # odd last width: per projection
    # eight projections, the most one group takes (persistent GEMM, one G^ layer table)
    (1000, 512, (64, 128, 64, 256, 72, 80, 128, 64), (8, 16, 8, 32, 8, 16, 16, 8)),
]


def _ids(g):
    return "T{}-n{}-m{}-r{}".format(g[0], g[1], "+".join(map(str, g[2])), "+".join(map(str, g[3])))


def _group_inputs(T, n, ms, data_seed):
    x, _ = fwd_inputs(T, n, 8, "bf16", data_seed=data_seed)
    Ws = [fwd_inputs(8, n, m, "bf16", data_seed=data_seed + 1 + j)[1] for j, m in enumerate(ms)]
    return x, Ws


@pytest.mark.parametrize("group", GROUPS, ids=_ids)
@pytest.mark.parametrize("use_ws", [True, False])
def test_group_equals_per_projection(group, use_ws):
    T, n, ms, rs = group
    seeds = [((j + 3) << 32) | 11 for j in range(len(ms))]
    x, Ws = _group_inputs(T, n, ms, data_seed=T + n)
    M, R = sum(ms), sum(rs)
    xd = to_dev(x, "bf16", ld_for(n, "bf16"))
    Wd = to_dev(np.concatenate(Ws, axis=1), "bf16", ld_for(M, "bf16"))
    y = empty(T, M, "bf16", ld_for(M, "bf16"), fill=7.0)
    z = empty(T, R, "bf16", ld_for(R, "bf16"), fill=7.0)
    ws = workspace(cp.fwd_group_workspace_bytes(n, ms, rs)) if use_ws else None
    cp.compact_fwd_group(xd, Wd, y, z, ms, rs, seeds, ws=ws)
    # reference: compact_fwd on each column slice, into separate buffers
    y1 = empty(T, M, "bf16", ld_for(M, "bf16"), fill=-3.0)
    z1 = empty(T, R, "bf16", ld_for(R, "bf16"), fill=-3.0)
    mo = ro = 0
    for j, (m, r) in enumerate(zip(ms, rs)):
        wsj = workspace(cp.fwd_workspace_bytes(n, m, r)) if use_ws else None
        cp.compact_fwd(xd, Wd[:, mo:mo + m], y1[:, mo:mo + m], z1[:, ro:ro + r], seeds[j], ws=wsj)
        mo += m
        ro += r
    torch.cuda.synchronize()
    assert torch.equal(y.view(torch.int16), y1.view(torch.int16))
    assert torch.equal(z.view(torch.int16), z1.view(torch.int16))


@pytest.mark.parametrize("group", GROUPS[:2], ids=_ids)
def test_group_oracle_parity(group):
    T, n, ms, rs = group
    seeds = [((j + 5) << 32) | 1 for j in range(len(ms))]
    x, Ws = _group_inputs(T, n, ms, data_seed=3 * T)
    M, R = sum(ms), sum(rs)
    xd = to_dev(x, "bf16", ld_for(n, "bf16"))
    Wd = to_dev(np.concatenate(Ws, axis=1), "bf16", ld_for(M, "bf16"))
    y = empty(T, M, "bf16", ld_for(M, "bf16"))
    z = empty(T, R, "bf16", ld_for(R, "bf16"))
    cp.compact_fwd_group(xd, Wd, y, z, ms, rs, seeds, ws=workspace(cp.fwd_group_workspace_bytes(n, ms, rs)))
    torch.cuda.synchronize()
    yn, zn = to_np(y), to_np(z)
    mo = ro = 0
    for j, (m, r) in enumerate(zip(ms, rs)):
        y_ref, z_ref = oc.ref_fwd(x, Ws[j], seeds[j], r)
        assert oc.rel_fro(yn[:, mo:mo + m], y_ref) <= TOL
        assert oc.rel_fro(zn[:, ro:ro + r], z_ref) <= TOL
        mo += m
        ro += r


def test_group_backward_through_concatenation():
    # q, k, v share x: dL/dx = sum_j dL/do_j W_j^T, one compact_bwd over [W_0 | W_1 | W_2]
    T, n, ms, rs = 640, 512, (512, 512, 512), (128, 128, 128)
    M, R = sum(ms), sum(rs)
    parts = [bwd_inputs(T, n, m, r, "bf16", data_seed=40 + j) for j, (m, r) in enumerate(zip(ms, rs))]
    dy_all = np.concatenate([p[0] for p in parts], axis=1)
    z_all = np.concatenate([p[1] for p in parts], axis=1)
    W_all = np.concatenate([p[2] for p in parts], axis=1)
    dyd = to_dev(dy_all, "bf16", ld_for(M, "bf16"))
    zd = to_dev(z_all, "bf16", ld_for(R, "bf16"))
    Wd = to_dev(W_all, "bf16", ld_for(M, "bf16"))
    dx = empty(T, n, "bf16", ld_for(n, "bf16"))
    cp.compact_bwd(dyd, Wd, None, dx, None)
    Gs = []
    mo = ro = 0
    for m, r in zip(ms, rs):
        G = torch.empty(r, m, dtype=torch.float32, device=dev())
        cp.compact_bwd(dyd[:, mo:mo + m], None, zd[:, ro:ro + r], None, G,
                       ws=workspace(cp.bwd_workspace_bytes(T, n, m, r)))
        Gs.append(G)
        mo += m
        ro += r
    torch.cuda.synchronize()
    dx_ref = sum(oc.ref_bwd(p[0], p[1], p[2])[0] for p in parts)
    assert oc.rel_fro(to_np(dx), dx_ref) <= TOL
    for G, p in zip(Gs, parts):
        assert oc.rel_fro(G.cpu().numpy(), oc.ref_bwd(p[0], p[1], p[2])[1]) <= TOL


def test_ghat_and_step_on_overhanging_column_slices():
    # G^ and the step on the second column slice of [A | B] where the slice
    # width (1376) is not a multiple of the kernels' column tiles, so the last
    # tile of the slice overhangs the end of the buffer on its last row.  The
    # results must equal those on contiguous copies, bit for bit.
    T, n, r, m = 1000, 1024, 128, 1376
    dy_a, z_a, W_a = bwd_inputs(T, n, m, r, "bf16", data_seed=71)
    dy_b, z_b, W_b = bwd_inputs(T, n, m, r, "bf16", data_seed=72)
    dy_all = to_dev(np.concatenate([dy_a, dy_b], axis=1), "bf16", 2 * m)   # ld = 2m: slice B ends the buffer
    z_all = to_dev(np.concatenate([z_a, z_b], axis=1), "bf16", 2 * r)
    ws = workspace(cp.bwd_workspace_bytes(T, n, m, r))
    G_slice = torch.empty(r, m, dtype=torch.float32, device=dev())
    G_copy = torch.empty(r, m, dtype=torch.float32, device=dev())
    cp.compact_bwd(dy_all[:, m:], None, z_all[:, r:], None, G_slice, ws=ws)
    cp.compact_bwd(to_dev(dy_b, "bf16"), None, to_dev(z_b, "bf16"), None, G_copy, ws=ws)
    torch.cuda.synchronize()
    assert torch.equal(G_slice, G_copy)

    W_all = to_dev(np.concatenate([W_a, W_b], axis=1), "bf16", 2 * m)
    W_copy = to_dev(W_b, "bf16")
    M1, V1 = torch.zeros_like(G_copy), torch.zeros_like(G_copy)
    M2, V2 = torch.zeros_like(G_copy), torch.zeros_like(G_copy)
    wss = workspace(cp.step_workspace_bytes(n, m, r))
    cp.compact_step(W_all[:, m:], G_copy, M1, V1, 9 << 32, 1, 1e-3, alpha=0.25, ws=wss)
    cp.compact_step(W_copy, G_copy, M2, V2, 9 << 32, 1, 1e-3, alpha=0.25, ws=wss)
    torch.cuda.synchronize()
    assert torch.equal(W_all[:, m:].contiguous().view(torch.int16), W_copy.view(torch.int16))
    # the first slice is untouched
    assert torch.equal(W_all[:, :m].contiguous().view(torch.int16), to_dev(W_a, "bf16").view(torch.int16))


def _bwd_group_inputs(T, n, ms, rs, data_seed, dt="bf16"):
    parts = [bwd_inputs(T, n, m, r, dt, data_seed=data_seed + j) for j, (m, r) in enumerate(zip(ms, rs))]
    M, R = sum(ms), sum(rs)
    dy_all = np.concatenate([p[0] for p in parts], axis=1)
    z_all = np.concatenate([p[1] for p in parts], axis=1)
    W_all = np.concatenate([p[2] for p in parts], axis=1)
    dev_t = (to_dev(dy_all, dt, ld_for(M, dt)), to_dev(z_all, dt, ld_for(R, dt)), to_dev(W_all, dt, ld_for(M, dt)))
    return parts, dev_t


BWD_GROUPS = GROUPS + [
    (65, 512, (512, 512, 512), (128, 128, 128)),       # fewer tokens than splits x 32
    (2048, 2736, (1024,), (342,)),                     # one projection (down), r past one row tile
    (777, 1024, (256,) * 8, (256,) * 8),               # eight projections on the 256 x 256 G^ tiles
]


@pytest.mark.parametrize("group", BWD_GROUPS, ids=_ids)
def test_bwd_group_oracle_parity(group):
    # Alg. 2 per projection through one compact_bwd_group call: dx against the
    # sum of the oracle's dL/do_j W_j^T, every G^_j against the oracle's z_j^T dL/do_j
    T, n, ms, rs = group
    parts, (dyd, zd, Wd) = _bwd_group_inputs(T, n, ms, rs, data_seed=90 + T)
    dx = empty(T, n, "bf16", ld_for(n, "bf16"), fill=5.0)
    Gs = [torch.full((r, m), 7.0, dtype=torch.float32, device=dev()) for m, r in zip(ms, rs)]
    ws = workspace(cp.bwd_group_workspace_bytes(T, n, ms, rs))
    cp.compact_bwd_group(dyd, Wd, zd, dx, Gs, ms, rs, ws=ws)
    torch.cuda.synchronize()
    dx_ref = sum(oc.ref_bwd(p[0], p[1], p[2])[0] for p in parts)
    assert oc.rel_fro(to_np(dx), dx_ref) <= TOL
    for G, p in zip(Gs, parts):
        assert oc.rel_fro(G.cpu().numpy(), oc.ref_bwd(p[0], p[1], p[2])[1]) <= TOL


@pytest.mark.parametrize("group", BWD_GROUPS, ids=_ids)
def test_bwd_group_against_per_slice_calls(group):
    # dx is the same GEMM as compact_bwd over the concatenated weight (bitwise);
    # each G^_j sums the same bf16 products over other token splits (fp32)
    T, n, ms, rs = group
    parts, (dyd, zd, Wd) = _bwd_group_inputs(T, n, ms, rs, data_seed=7 * T)
    dx = empty(T, n, "bf16", ld_for(n, "bf16"))
    Gs = [torch.empty(r, m, dtype=torch.float32, device=dev()) for m, r in zip(ms, rs)]
    cp.compact_bwd_group(dyd, Wd, zd, dx, Gs, ms, rs, ws=workspace(cp.bwd_group_workspace_bytes(T, n, ms, rs)))
    dx1 = empty(T, n, "bf16", ld_for(n, "bf16"))
    cp.compact_bwd(dyd, Wd, None, dx1, None)
    G1s = []
    mo = ro = 0
    for m, r in zip(ms, rs):
        G = torch.empty(r, m, dtype=torch.float32, device=dev())
        cp.compact_bwd(dyd[:, mo:mo + m], None, zd[:, ro:ro + r], None, G,
                       ws=workspace(cp.bwd_workspace_bytes(T, n, m, r)))
        G1s.append(G)
        mo += m
        ro += r
    torch.cuda.synchronize()
    assert torch.equal(dx.view(torch.int16), dx1.view(torch.int16))
    for G, G1 in zip(Gs, G1s):
        g, g1 = G.cpu().numpy().astype(np.float64), G1.cpu().numpy().astype(np.float64)
        assert oc.rel_fro(g, g1) <= 1e-5


def test_bwd_group_parts_and_empty():
    # dx only, G^ only, and zero tokens (every G^_j is zero)
    T, n, ms, rs = 513, 512, (512, 512, 512), (128, 128, 128)
    parts, (dyd, zd, Wd) = _bwd_group_inputs(T, n, ms, rs, data_seed=5)
    ws = workspace(cp.bwd_group_workspace_bytes(T, n, ms, rs))
    dx = empty(T, n, "bf16", ld_for(n, "bf16"))
    cp.compact_bwd_group(dyd, Wd, None, dx, None, ms, rs)
    Gs = [torch.empty(r, m, dtype=torch.float32, device=dev()) for m, r in zip(ms, rs)]
    cp.compact_bwd_group(dyd, None, zd, None, Gs, ms, rs, ws=ws)
    G0 = [torch.full((r, m), 3.0, dtype=torch.float32, device=dev()) for m, r in zip(ms, rs)]
    # zero tokens through the raw ABI (an empty torch view has no data pointer)
    import ctypes
    lib = cp.library()
    st = lib.compact_bwd_group(dyd.data_ptr(), dyd.stride(0), None, 0, zd.data_ptr(), zd.stride(0), None, 0,
                               (ctypes.c_void_p * 3)(*[G.data_ptr() for G in G0]), 0, n, 3,
                               (ctypes.c_int64 * 3)(*ms), (ctypes.c_int64 * 3)(*rs), 1, 0, ws.data_ptr(), ws.numel(),
                               torch.cuda.current_stream().cuda_stream)
    assert st == 0
    # zero tokens with accumulate: G^ + (a sum over no tokens) leaves G^ as it is
    G1 = [torch.full((r, m), 3.0, dtype=torch.float32, device=dev()) for m, r in zip(ms, rs)]
    st = lib.compact_bwd_group(dyd.data_ptr(), dyd.stride(0), None, 0, zd.data_ptr(), zd.stride(0), None, 0,
                               (ctypes.c_void_p * 3)(*[G.data_ptr() for G in G1]), 0, n, 3,
                               (ctypes.c_int64 * 3)(*ms), (ctypes.c_int64 * 3)(*rs), 1, 1, ws.data_ptr(), ws.numel(),
                               torch.cuda.current_stream().cuda_stream)
    assert st == 0
    torch.cuda.synchronize()
    assert all(bool((G == 3.0).all()) for G in G1)
    assert oc.rel_fro(to_np(dx), sum(oc.ref_bwd(p[0], p[1], p[2])[0] for p in parts)) <= TOL
    for G, p in zip(Gs, parts):
        assert oc.rel_fro(G.cpu().numpy(), oc.ref_bwd(p[0], p[1], p[2])[1]) <= TOL
    assert all(float(G.abs().max()) == 0.0 for G in G0)


@pytest.mark.parametrize("dt", ["bf16", "f32"])
@pytest.mark.parametrize("T", [513, 16384 + 77])
def test_bwd_group_accumulate(T, dt):
    # gradient accumulation in the library: G^ <- G^ + z^T dL/do is bitwise
    # G^ + (the G^ of a fresh call), one fp32 addition per element, on the
    # bf16 path (one split-K launch; T = 16461 takes several splits) and the
    # fp32 one; against the oracle for two backward passes in a row
    n, ms, rs = 512, (512, 512, 512), (128, 128, 128)
    parts1, (dy1, z1, Wd) = _bwd_group_inputs(T, n, ms, rs, data_seed=11, dt=dt)
    parts2, (dy2, z2, _) = _bwd_group_inputs(T, n, ms, rs, data_seed=12, dt=dt)
    code = cp.BF16 if dt == "bf16" else cp.F32
    ws = workspace(cp.bwd_group_workspace_bytes(T, n, ms, rs, code)) if dt == "bf16" else None
    fresh = [torch.empty(r, m, dtype=torch.float32, device=dev()) for m, r in zip(ms, rs)]
    acc = [torch.empty(r, m, dtype=torch.float32, device=dev()) for m, r in zip(ms, rs)]
    cp.compact_bwd_group(dy1, None, z1, None, acc, ms, rs, ws=ws)                    # first pass
    prev = [g.clone() for g in acc]
    cp.compact_bwd_group(dy2, None, z2, None, acc, ms, rs, ws=ws, accumulate=True)   # second pass, added
    cp.compact_bwd_group(dy2, None, z2, None, fresh, ms, rs, ws=ws)
    torch.cuda.synchronize()
    for a, p, f in zip(acc, prev, fresh):
        assert torch.equal(a, p + f)
    tol = TOL if dt == "bf16" else 1e-5
    for a, q1, q2 in zip(acc, parts1, parts2):
        ref = oc.ref_bwd(q1[0], q1[1], q1[2])[1] + oc.ref_bwd(q2[0], q2[1], q2[2])[1]
        assert oc.rel_fro(a.cpu().numpy(), ref) <= tol
