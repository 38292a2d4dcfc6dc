"""GPU parity of the CompAct layer against the fp64 oracle.

Each ABI call is checked on seeded inputs from ``synthetic`` (the oracle never
sees a value produced on the GPU): relative Frobenius error <= 1e-5 on the fp32
path and <= 2e-2 on the bf16 path, per output.  Shapes span several tiles and
ragged tails in every dimension; a three-step chain checks the whole
fwd -> bwd -> step loop (the first Adam step is sign-like, N = G^/(|G^|+eps),
so the update of step 1 is compared only through the smooth moments).
"""
import numpy as np
import pytest

from oracle import compact as oc
from synthetic import bf16_round, bwd_inputs, fwd_inputs, step_inputs, workload

from gpu_util import dev, empty, ld_for, to_dev, to_np, to_np_f32, workspace

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
cp = pytest.importorskip("paper_2410_15352_amd")

TOL = {"f32": 1e-5, "bf16": 2e-2}
CODE = {"f32": 0, "bf16": 1}

# (tokens, n, m, r, dtype): tile multiples, ragged tails, r not a multiple of 8
SHAPES = [
    (256, 256, 512, 32, "f32"),          # the single fp32 layer workload
    (100, 36, 20, 12, "f32"),
    (300, 200, 136, 40, "bf16"),
    (1000, 1376, 512, 344, "bf16"),
    (513, 512, 1376, 128, "bf16"),
    (2048, 768, 3072, 384, "bf16"),
    (777, 1024, 2736, 128, "bf16"),
    (128, 5461, 64, 682, "bf16"),
    (150, 200, 203, 24, "bf16"),         # odd m: partial column groups in the update
]


def _ids(s):
    return "T{}-n{}-m{}-r{}-{}".format(*s)


# (shape, workspace): the fp32 path has no workspace mode
FWD_CASES = [(s, ws) for s in SHAPES for ws in (True, False) if not (s[4] == "f32" and ws)]


@pytest.mark.parametrize("shape,use_ws", FWD_CASES, ids=[f"{ws}-{_ids(s)}" for s, ws in FWD_CASES])
def test_forward_parity(shape, use_ws):
    T, n, m, r, dt = shape
    seed = (11 << 32) | 3
    x, W = fwd_inputs(T, n, m, dt, data_seed=T + n)
    xd, Wd = to_dev(x, dt, ld_for(n, dt)), to_dev(W, dt, ld_for(m, dt))
    y = empty(T, m, dt, ld_for(m, dt))
    z = empty(T, r, dt, ld_for(r, dt))
    ws = workspace(cp.fwd_workspace_bytes(n, m, r, CODE[dt])) if use_ws else None
    if ws is not None:
        ws.fill_(0xFF)  # stale bytes (NaN patterns) in unwritten padding must not reach y or z
    cp.compact_fwd(xd, Wd, y, z, seed, ws=ws)
    torch.cuda.synchronize()
    y_ref, z_ref = oc.ref_fwd(x, W, seed, r)
    assert oc.rel_fro(to_np(y), y_ref) <= TOL[dt]
    assert oc.rel_fro(to_np(z), z_ref) <= TOL[dt]


@pytest.mark.parametrize("shape", SHAPES, ids=_ids)
def test_backward_parity(shape):
    T, n, m, r, dt = shape
    dy, z, W = bwd_inputs(T, n, m, r, dt, data_seed=T + m)
    dyd = to_dev(dy, dt, ld_for(m, dt))
    zd = to_dev(z, dt, ld_for(r, dt))
    Wd = to_dev(W, dt, ld_for(m, dt))
    dx = empty(T, n, dt, ld_for(n, dt))
    G = torch.empty(r, m, dtype=torch.float32, device=dev())
    ws = workspace(cp.bwd_workspace_bytes(T, n, m, r, CODE[dt]))
    cp.compact_bwd(dyd, Wd, zd, dx, G, ws=ws)
    torch.cuda.synchronize()
    dx_ref, G_ref = oc.ref_bwd(dy, z, W)
    assert oc.rel_fro(to_np(dx), dx_ref) <= TOL[dt]
    assert oc.rel_fro(G.cpu().numpy(), G_ref) <= TOL[dt]


@pytest.mark.parametrize("shape", [s for s in SHAPES if s[4] == "bf16"], ids=_ids)
def test_dx_staged_weight_bitwise(shape):
    # with a workspace the dx GEMM reads a K-tiled copy of W, without one W
    # itself: the same products in the same order, so dx is bitwise equal
    T, n, m, r, dt = shape
    dy, _, W = bwd_inputs(T, n, m, r, dt, data_seed=2 * T + m)
    dyd, Wd = to_dev(dy, dt, ld_for(m, dt)), to_dev(W, dt, ld_for(m, dt))
    dx0 = empty(T, n, dt, ld_for(n, dt), fill=1.0)
    dx1 = empty(T, n, dt, ld_for(n, dt), fill=2.0)
    cp.compact_bwd(dyd, Wd, None, dx0, None)
    ws = workspace(cp.bwd_workspace_bytes(T, n, m, r, CODE[dt]))
    ws.fill_(0xFF)  # stale bytes (NaN patterns) in the padding rows must not reach dx
    cp.compact_bwd(dyd, Wd, None, dx1, None, ws=ws)
    torch.cuda.synchronize()
    assert torch.equal(dx0.view(torch.int16), dx1.view(torch.int16))
    dx_ref, _ = oc.ref_bwd(dy, np.zeros((T, r)), W)
    assert oc.rel_fro(to_np(dx1), dx_ref) <= TOL[dt]


def _dw_on_zero(n, m, r, G, M, V, seed, t, lr, b1, b2, eps, alpha, dt, ws, proj="gaussian"):
    """W' - W of compact_step with fp32 master weights W = 0 (the update
    itself, exact to fp32), on copies of G^, M and V."""
    Wz = torch.zeros(n, ld_for(m, "f32"), dtype=torch.float32, device=dev())[:, :m]
    Gd, Md, Vd = (torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(dev()) for a in (G, M, V))
    cp.compact_step(Wz, Gd, Md, Vd, seed, t, lr, b1, b2, eps, alpha, proj=proj, dtype=dt, ws=ws)
    torch.cuda.synchronize()
    return to_np_f32(Wz).astype(np.float64)


@pytest.mark.parametrize("shape", SHAPES, ids=_ids)
@pytest.mark.parametrize("t", [1, 3])
def test_step_parity(shape, t):
    _, n, m, r, dt = shape
    seed, lr, b1, b2, eps, alpha = (5 << 32) | 1, 1e-3, 0.9, 0.999, 1e-8, 0.25
    W, G, M, V = step_inputs(n, m, r, dt, t=t, data_seed=n + r)
    Wd = to_dev(W, "f32", ld_for(m, "f32"))     # fp32 master copy: dW is exact to fp32
    Gd, Md, Vd = (torch.from_numpy(a.copy()).to(dev()) for a in (G, M, V))
    ws = workspace(cp.step_workspace_bytes(n, m, r, CODE[dt]))
    cp.compact_step(Wd, Gd, Md, Vd, seed, t, lr, b1, b2, eps, alpha, dtype=dt, ws=ws)
    torch.cuda.synchronize()
    W_ref, M_ref, V_ref, dW_ref = oc.ref_step(W, G, M, V, seed, r, t, lr, b1, b2, eps, alpha)
    assert oc.rel_fro(Md.cpu().numpy(), M_ref) <= TOL[dt]
    assert oc.rel_fro(Vd.cpu().numpy(), V_ref) <= TOL[dt]
    assert oc.rel_fro(to_np_f32(Wd), W_ref) <= TOL[dt]
    # the update itself: the same step on W = 0 writes W' = -fp32(coef * acc),
    # dW without the cancellation of W' - W
    assert oc.rel_fro(_dw_on_zero(n, m, r, G, M, V, seed, t, lr, b1, b2, eps, alpha, dt, ws), dW_ref) <= TOL[dt]

    if dt == "bf16":
        # bf16 weights: same kernel, update rounded once to bf16 (RNE(fp32 result))
        Wb = to_dev(W, "bf16", ld_for(m, "bf16"))
        Gd2, Md2, Vd2 = (torch.from_numpy(a.copy()).to(dev()) for a in (G, M, V))
        cp.compact_step(Wb, Gd2, Md2, Vd2, seed, t, lr, b1, b2, eps, alpha, dtype="bf16", ws=ws)
        torch.cuda.synchronize()
        assert np.array_equal(to_np_f32(Wb).view(np.uint32), bf16_round(to_np_f32(Wd)).view(np.uint32))
        assert oc.rel_fro(to_np(Wb), W_ref) <= TOL[dt]


def test_step_dw_fp32_exact_precision():
    # W = 0 in fp32: W' = -fp32(coef * acc) exactly, so dW is compared without
    # the cancellation of W' - W.
    n, m, r = 256, 512, 32
    _, G, M, V = step_inputs(n, m, r, "f32", t=1, data_seed=3)
    Wd = torch.zeros(n, m, dtype=torch.float32, device=dev())
    Gd, Md, Vd = (torch.from_numpy(a.copy()).to(dev()) for a in (G, M, V))
    ws = workspace(cp.step_workspace_bytes(n, m, r, 0))
    cp.compact_step(Wd, Gd, Md, Vd, 1, 1, 1e-3, dtype="f32", ws=ws)
    torch.cuda.synchronize()
    _, _, _, dW_ref = oc.ref_step(np.zeros((n, m)), G, M, V, 1, r, 1, 1e-3, 0.9, 0.999, 1e-8, 1.0)
    assert oc.rel_fro(Wd.cpu().numpy(), dW_ref) <= 1e-5


@pytest.mark.parametrize("dt", ["f32", "bf16"])
def test_identity_projection(dt):
    # P = I, r = n: z equals x bit for bit, and the step equals uncompressed Adam
    T, n, m = 300, 64, 72
    x, W = fwd_inputs(T, n, m, dt, data_seed=1)
    xd, Wd = to_dev(x, dt), to_dev(W, dt)
    y = empty(T, m, dt)
    z = empty(T, n, dt)
    cp.compact_fwd(xd, Wd, y, z, 0, proj="identity")
    torch.cuda.synchronize()
    assert np.array_equal(to_np(z), x.astype(np.float64))
    Wm, G, M, V = step_inputs(n, m, n, dt, t=2, data_seed=2)
    Wmd = to_dev(Wm, "f32")
    Gd, Md, Vd = (torch.from_numpy(a.copy()).to(dev()) for a in (G, M, V))
    ws = workspace(cp.step_workspace_bytes(n, m, n, CODE[dt]))
    cp.compact_step(Wmd, Gd, Md, Vd, 0, 2, 1e-2, alpha=0.5, proj="identity", dtype=dt, ws=ws)
    torch.cuda.synchronize()
    W_ref, M_ref, V_ref, dW_ref = oc.ref_step(Wm, G, M, V, 0, n, 2, 1e-2, 0.9, 0.999, 1e-8, 0.5,
                                              identity=True)
    assert oc.rel_fro(to_np_f32(Wmd), W_ref) <= TOL[dt]
    dW = _dw_on_zero(n, m, n, G, M, V, 0, 2, 1e-2, 0.9, 0.999, 1e-8, 0.5, dt, ws, proj="identity")
    assert oc.rel_fro(dW, dW_ref) <= TOL[dt]
    assert oc.rel_fro(Md.cpu().numpy(), M_ref) <= TOL[dt]


def test_outputs_independent_of_seed_and_deterministic():
    T, n, m, r, dt = 700, 512, 1376, 128, "bf16"
    x, W = fwd_inputs(T, n, m, dt, data_seed=9)
    xd, Wd = to_dev(x, dt), to_dev(W, dt)
    outs = []
    for seed in (1, 2, 1):
        y, z = empty(T, m, dt), empty(T, r, dt)
        cp.compact_fwd(xd, Wd, y, z, seed)
        outs.append((y.clone(), z.clone()))
    torch.cuda.synchronize()
    assert torch.equal(outs[0][0].view(torch.int16), outs[1][0].view(torch.int16))
    assert not torch.equal(outs[0][1].view(torch.int16), outs[1][1].view(torch.int16))
    assert torch.equal(outs[0][1].view(torch.int16), outs[2][1].view(torch.int16))
    dy, _, _ = bwd_inputs(T, n, m, r, dt, data_seed=9)
    dyd = to_dev(dy, dt)
    ws = workspace(cp.bwd_workspace_bytes(T, n, m, r))
    res = []
    for z_ in (outs[0][1], outs[1][1], outs[0][1]):
        dx = empty(T, n, dt)
        G = torch.empty(r, m, dtype=torch.float32, device=dev())
        cp.compact_bwd(dyd, Wd, z_, dx, G, ws=ws)
        res.append((dx.clone(), G.clone()))
    torch.cuda.synchronize()
    assert torch.equal(res[0][0].view(torch.int16), res[1][0].view(torch.int16))  # dx ignores P
    assert torch.equal(res[0][1], res[2][1])                                      # G^ deterministic


@pytest.mark.parametrize("name", ["single-f32", "llama-60m"])
def test_three_step_chain(name):
    wl = workload(name)
    L = wl.layers[0] if name == "single-f32" else wl.layers[6]  # the down projection
    T = min(wl.tokens, 1024)
    dt = wl.dtype
    n, m, r, seed = L.n, L.m, L.r, L.seed
    x0, W0 = fwd_inputs(T, n, m, dt, data_seed=100)
    W_gpu = to_dev(W0, "f32", ld_for(m, "f32"))     # fp32 master weights
    M = torch.zeros(r, m, dtype=torch.float32, device=dev())
    V = torch.zeros_like(M)
    W_ref = W0.astype(np.float64)
    M_ref = np.zeros((r, m))
    V_ref = np.zeros((r, m))
    ws_b = workspace(cp.bwd_workspace_bytes(T, n, m, r, CODE[dt]))
    ws_s = workspace(cp.step_workspace_bytes(n, m, r, CODE[dt]))
    for t in (1, 2, 3):
        x, _ = fwd_inputs(T, n, m, dt, data_seed=100 + t)
        dy, _, _ = bwd_inputs(T, n, m, r, dt, data_seed=200 + t)
        W_cmp = W_gpu if dt == "f32" else W_gpu.to(torch.bfloat16)
        xd, dyd = to_dev(x, dt), to_dev(dy, dt)
        y, z = empty(T, m, dt), empty(T, r, dt)
        cp.compact_fwd(xd, W_cmp, y, z, seed)
        dx = empty(T, n, dt)
        G = torch.empty(r, m, dtype=torch.float32, device=dev())
        cp.compact_bwd(dyd, W_cmp, z, dx, G, ws=ws_b)
        W_before = W_gpu.clone()
        G_in, M_in, V_in = G.cpu().numpy(), M.cpu().numpy(), V.cpu().numpy()
        cp.compact_step(W_gpu, G, M, V, seed, t, wl.lr, wl.beta1, wl.beta2, wl.eps, wl.alpha,
                        dtype=dt, ws=ws_s)
        torch.cuda.synchronize()
        _, z_ref = oc.ref_fwd(x, W_ref, seed, r)
        dx_ref, G_ref = oc.ref_bwd(dy, z_ref, W_ref)
        W_new, M_ref, V_ref, dW_ref = oc.ref_step(W_ref, G_ref, M_ref, V_ref, seed, r, t, wl.lr,
                                                  wl.beta1, wl.beta2, wl.eps, wl.alpha)
        tol = TOL[dt]
        if t == 1:  # later steps use weights that already differ by rounding
            assert oc.rel_fro(to_np(dx), dx_ref) <= tol
        assert oc.rel_fro(to_np(z), z_ref) <= tol
        assert oc.rel_fro(G.cpu().numpy(), G_ref) <= tol
        assert oc.rel_fro(M.cpu().numpy(), M_ref) <= tol
        assert oc.rel_fro(V.cpu().numpy(), V_ref) <= tol
        if t >= 2:
            # the update on W = 0 from this step's G^, M, V (no cancellation)
            dW = _dw_on_zero(n, m, r, G_in, M_in, V_in, seed, t, wl.lr, wl.beta1, wl.beta2, wl.eps, wl.alpha,
                             dt, ws_s)
            assert oc.rel_fro(dW, dW_ref) <= tol
            # and W' - W of the chained step agrees with it up to the rounding of W'
            assert oc.rel_fro((W_gpu - W_before).cpu().numpy().astype(np.float64), dW_ref) <= max(tol, 2e-4)
        W_ref = W_new
        new_seed = oc.next_seed(seed, t, 2)  # Alg. 3: re-sample every T = 2 steps
        assert cp.compact_next_seed(seed, t, 2) == new_seed
        seed = new_seed


def test_step_batched_equals_per_layer():
    # the batched launches compute exactly what compact_step computes per layer;
    # 45 layers make two launch groups, so the two-stream schedule runs
    shapes = [(512, 512, 128), (512, 1376, 128), (1376, 512, 344), (300, 200, 40), (5461, 64, 1365)] * 9
    layers_a, layers_b, states = [], [], []
    for i, (n, m, r) in enumerate(shapes):
        W, G, M, V = step_inputs(n, m, r, "bf16", t=2, data_seed=50 + i)
        wa = to_dev(W, "bf16", ld_for(m, "bf16"))
        wb = to_dev(W, "bf16", ld_for(m, "bf16"))
        ga, ma, va = (torch.from_numpy(a.copy()).to(dev()) for a in (G, M, V))
        gb, mb, vb = (torch.from_numpy(a.copy()).to(dev()) for a in (G, M, V))
        seed = ((i + 1) << 32) | 7
        layers_a.append(dict(W=wa, G=ga, M=ma, V=va, seed=seed, alpha=0.25 + 0.01 * i))
        layers_b.append(dict(W=wb, G=gb, M=mb, V=vb, seed=seed, alpha=0.25 + 0.01 * i))
    ws = workspace(cp.step_batched_workspace_bytes(layers_a))
    cp.compact_step_batched(layers_a, 2, 1e-3, ws=ws)
    for L in layers_b:
        n, m = L["W"].shape
        r = L["G"].shape[0]
        ws1 = workspace(cp.step_workspace_bytes(n, m, r))
        cp.compact_step(L["W"], L["G"], L["M"], L["V"], L["seed"], 2, 1e-3, alpha=L["alpha"], ws=ws1)
    torch.cuda.synchronize()
    for La, Lb in zip(layers_a, layers_b):
        assert torch.equal(La["M"], Lb["M"]) and torch.equal(La["V"], Lb["V"])
        assert torch.equal(La["W"].view(torch.int16), Lb["W"].view(torch.int16))


def test_step_batched_stream_order():
    # on a caller's stream: work enqueued before the call (G, M, V, W set) is
    # seen by every launch group, and work enqueued after it (clones) sees the
    # finished step, with no host synchronisation in between
    shapes = [(512, 512, 128), (512, 1376, 128), (1376, 512, 344)] * 30  # three launch groups
    rng = np.random.default_rng(77)
    s = torch.cuda.Stream()
    layers, ref = [], []
    for i, (n, m, r) in enumerate(shapes):
        W, G, M, V = step_inputs(n, m, r, "bf16", t=3, data_seed=300 + i)
        host = [torch.from_numpy(a.copy()).pin_memory() for a in (G, M, V)]
        wh = to_dev(W, "bf16", ld_for(m, "bf16")).cpu().pin_memory()
        layers.append(dict(W=torch.zeros(n, ld_for(m, "bf16"), dtype=torch.bfloat16, device=dev())[:, :m],
                           G=torch.zeros(r, m, device=dev()), M=torch.zeros(r, m, device=dev()),
                           V=torch.zeros(r, m, device=dev()), seed=((i + 3) << 32) | 1, alpha=0.5, host=host, wh=wh))
        wr = to_dev(W, "bf16", ld_for(m, "bf16"))
        gr, mr, vr = (torch.from_numpy(a.copy()).to(dev()) for a in (G, M, V))
        ref.append(dict(W=wr, G=gr, M=mr, V=vr, seed=layers[-1]["seed"], alpha=0.5))
    for L in ref:
        n, m = L["W"].shape
        ws1 = workspace(cp.step_workspace_bytes(n, m, L["G"].shape[0]))
        cp.compact_step(L["W"], L["G"], L["M"], L["V"], L["seed"], 3, 1e-3, alpha=L["alpha"], ws=ws1)
    torch.cuda.synchronize()
    batch = [dict(W=L["W"], G=L["G"], M=L["M"], V=L["V"], seed=L["seed"], alpha=L["alpha"]) for L in layers]
    ws = workspace(cp.step_batched_workspace_bytes(batch))
    torch.cuda.synchronize()
    with torch.cuda.stream(s):
        # a slow kernel first, so that a launch group not ordered after it would
        # run before the copies below land
        big = torch.empty(1 << 28, dtype=torch.uint8, device=dev())
        for _ in range(4):
            big.fill_(int(rng.integers(1, 255)))
        for L in layers:
            for d, h in zip((L["G"], L["M"], L["V"]), L["host"]):
                d.copy_(h, non_blocking=True)
            L["W"].copy_(L["wh"][:, :L["W"].shape[1]], non_blocking=True)
        cp.compact_step_batched(batch, 3, 1e-3, ws=ws, stream=s.cuda_stream)
        outs = [(L["W"].clone(), L["M"].clone(), L["V"].clone()) for L in layers]
        for L in layers:  # overwritten right after the clones were taken
            L["M"].fill_(0.0)
    torch.cuda.synchronize()
    for (w, m_, v), R in zip(outs, ref):
        assert torch.equal(m_, R["M"]) and torch.equal(v, R["V"])
        assert torch.equal(w.view(torch.int16), R["W"].view(torch.int16))


# degenerate sizes: rank 1, a single column, a single token, r = n, a wide n
# with a narrow m; every path (forward, backward, step) on both dtypes
TINY = [(1, 1, 1, 1), (3, 5, 2, 1), (7, 16, 1, 16), (40, 8, 3, 8), (2, 2048, 2, 1), (65, 33, 9, 7)]
TINY_CASES = [(s + (dt,)) for s in TINY for dt in ("f32", "bf16")]


@pytest.mark.parametrize("shape", TINY_CASES, ids=_ids)
def test_degenerate_shapes(shape):
    T, n, m, r, dt = shape
    seed = (21 << 32) | 9
    x, W = fwd_inputs(T, n, m, dt, data_seed=7 * T + n)
    xd, Wd = to_dev(x, dt, ld_for(n, dt)), to_dev(W, dt, ld_for(m, dt))
    y, z = empty(T, m, dt, ld_for(m, dt)), empty(T, r, dt, ld_for(r, dt))
    fws = cp.fwd_workspace_bytes(n, m, r, CODE[dt])
    cp.compact_fwd(xd, Wd, y, z, seed, ws=workspace(fws) if fws else None)
    dy, _, _ = bwd_inputs(T, n, m, r, dt, data_seed=7 * T + m)
    dyd = to_dev(dy, dt, ld_for(m, dt))
    dx = empty(T, n, dt, ld_for(n, dt))
    G = torch.empty(r, m, dtype=torch.float32, device=dev())
    cp.compact_bwd(dyd, Wd, z, dx, G, ws=workspace(cp.bwd_workspace_bytes(T, n, m, r, CODE[dt])))
    torch.cuda.synchronize()
    y_ref, z_ref = oc.ref_fwd(x, W, seed, r)
    assert oc.rel_fro(to_np(y), y_ref) <= TOL[dt]
    assert oc.rel_fro(to_np(z), z_ref) <= TOL[dt]
    dx_ref, G_ref = oc.ref_bwd(dy, to_np(z), W)
    assert oc.rel_fro(to_np(dx), dx_ref) <= TOL[dt]
    assert oc.rel_fro(G.cpu().numpy(), G_ref) <= TOL[dt]
    # step (t = 3: smooth moments), fp32 master weights
    t, lr, b1, b2, eps, alpha = 3, 1e-3, 0.9, 0.999, 1e-8, 0.5
    W0, Gs, M, V = step_inputs(n, m, r, dt, t=t, data_seed=n + 3 * r)
    Wm = to_dev(W0, "f32", ld_for(m, "f32"))
    Gd, Md, Vd = (torch.from_numpy(a.copy()).to(dev()) for a in (Gs, M, V))
    cp.compact_step(Wm, Gd, Md, Vd, seed, t, lr, b1, b2, eps, alpha, dtype=dt,
                    ws=workspace(cp.step_workspace_bytes(n, m, r, CODE[dt])))
    torch.cuda.synchronize()
    _, M_ref, V_ref, dW_ref = oc.ref_step(W0, Gs, M, V, seed, r, t, lr, b1, b2, eps, alpha)
    assert oc.rel_fro(Md.cpu().numpy(), M_ref) <= TOL[dt]
    assert oc.rel_fro(Vd.cpu().numpy(), V_ref) <= TOL[dt]
    dW = _dw_on_zero(n, m, r, Gs, M, V, seed, t, lr, b1, b2, eps, alpha, dt,
                     workspace(cp.step_workspace_bytes(n, m, r, CODE[dt])))
    assert oc.rel_fro(dW, dW_ref) <= TOL[dt]


@pytest.mark.parametrize("dt", ["f32", "bf16"])
def test_zero_tokens(dt):
    # an empty batch through the raw ABI (an empty torch view has no data
    # pointer): the forward writes nothing, G^ (a sum over no tokens) is zero
    n, m, r = 64, 48, 16
    lib = cp.library()
    stream = torch.cuda.current_stream().cuda_stream
    x = empty(4, n, dt, ld_for(n, dt), fill=1.0)
    _, W = fwd_inputs(4, n, m, dt, data_seed=3)
    Wd = to_dev(W, dt, ld_for(m, dt))
    y = empty(4, m, dt, ld_for(m, dt), fill=5.0)
    z = empty(4, r, dt, ld_for(r, dt), fill=6.0)
    fws = cp.fwd_workspace_bytes(n, m, r, CODE[dt])
    wsf = workspace(fws)
    st = lib.compact_fwd(x.data_ptr(), x.stride(0), Wd.data_ptr(), Wd.stride(0), y.data_ptr(), y.stride(0),
                         z.data_ptr(), z.stride(0), 0, n, m, r, 7, 0, CODE[dt], wsf.data_ptr() if fws else None,
                         fws, stream)
    assert st == 0
    G = torch.full((r, m), 3.0, dtype=torch.float32, device=dev())
    dx = empty(4, n, dt, ld_for(n, dt), fill=8.0)
    bws = cp.bwd_workspace_bytes(0, n, m, r, CODE[dt])
    wsb = workspace(bws)
    st = lib.compact_bwd(y.data_ptr(), y.stride(0), Wd.data_ptr(), Wd.stride(0), z.data_ptr(), z.stride(0),
                         dx.data_ptr(), dx.stride(0), G.data_ptr(), 0, n, m, r, CODE[dt],
                         wsb.data_ptr() if bws else None, bws, stream)
    assert st == 0
    torch.cuda.synchronize()
    assert float(G.abs().max()) == 0.0
    assert bool((y.float() == 5.0).all()) and bool((z.float() == 6.0).all()) and bool((dx.float() == 8.0).all())
