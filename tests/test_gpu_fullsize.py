"""Parity at the benchmark's full sizes (LLaMA-350M shapes and 65536 tokens, and
the other workloads' shapes at their token counts), in the launch configuration
the benchmark times.  q|k|v and gate|up run as input
groups (compact_fwd_group with its workspace: one staged operand, one
persistent GEMM); o and down run alone; the backward of each group is one
compact_bwd_group call (dL/dx over the concatenated weight, every G^_j of the
group in one split-K launch); Alg. 3 runs for all 168 layers in one
compact_step_batched call on column slices of the group weights.

Every distinct input group of every bf16 workload is covered the same way
(LLaMA-60M, RoBERTa-Base, LLaMA-1B at r = n/4 and n/8 too, each at its full
token count; LLaMA-1B's gate and up run apart, their width 5461 not being a
multiple of 8).  The oracle computes sampled outputs directly from the same
seeded inputs (it never sees a GPU value): rows of y, z and dL/dx for sampled tokens (the last
token always among them), columns of G^ as sums over all 65536 tokens, and
columns of the updated W, M and V (the last column always among them).
"""
import numpy as np
import pytest

from oracle import compact as oc
from oracle.pstream import projection
from synthetic import normal_bf16_blocked, workload

from gpu_util import dev, empty, ld_for, to_dev, to_np, workspace

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
cp = pytest.importorskip("paper_2410_15352_amd")

TOL = 2e-2


def _distinct_groups():
    """(workload, tokens, n, widths, ranks, seeds) of every distinct input group
    of the bf16 workloads, as the benchmark forms them (synthetic.input_groups)."""
    from synthetic import input_groups
    cases = []
    for name in ("llama-60m", "roberta-base", "llama-350m", "llama-1b-r4", "llama-1b-r8"):
        wl = workload(name)
        seen = set()
        for g in input_groups(wl):
            Ls = [wl.layers[i] for i in g]
            key = (Ls[0].n, tuple(L.m for L in Ls), tuple(L.r for L in Ls))
            if key in seen:
                continue
            seen.add(key)
            cases.append((name, wl.tokens, key[0], key[1], key[2], tuple(L.seed for L in Ls)))
    return cases


CASES = _distinct_groups()


def _case_id(c):
    return "{}-n{}-m{}-r{}".format(c[0], c[2], "+".join(map(str, c[3])), "+".join(map(str, c[4])))


def _rows(t, idx):
    return to_np(t[torch.as_tensor(idx, device=dev())])


def _sample(rng, size, k):
    s = np.sort(rng.choice(size, k, replace=False))
    s[-1] = size - 1
    return s


@pytest.mark.parametrize("case", CASES, ids=_case_id)
def test_full_size_forward_backward(case):
    _, T, n, ms, rs, seeds = case
    M, R = sum(ms), sum(rs)
    x = normal_bf16_blocked(T, n, seed=1000 + n)
    Ws = [normal_bf16_blocked(n, m, seed=2000 + 10 * k + n, scale=0.02) for k, m in enumerate(ms)]
    dy = normal_bf16_blocked(T, M, seed=3000 + M, scale=0.01)
    xd = to_dev(x, "bf16", ld_for(n, "bf16"))
    Wd = to_dev(np.concatenate(Ws, axis=1), "bf16", ld_for(M, "bf16"))
    dyd = to_dev(dy, "bf16", ld_for(M, "bf16"))
    y = empty(T, M, "bf16", ld_for(M, "bf16"))
    z = empty(T, R, "bf16", ld_for(R, "bf16"))
    ws_f = workspace(cp.fwd_group_workspace_bytes(n, ms, rs))
    if len(ms) > 1:
        cp.compact_fwd_group(xd, Wd, y, z, ms, rs, seeds, ws=ws_f)
    else:
        cp.compact_fwd(xd, Wd, y, z, seeds[0], ws=ws_f)
    dx = empty(T, n, "bf16", ld_for(n, "bf16"))
    Gs = [torch.empty(r, m, dtype=torch.float32, device=dev()) for m, r in zip(ms, rs)]
    ws_b = workspace(cp.bwd_group_workspace_bytes(T, n, ms, rs))
    cp.compact_bwd_group(dyd, Wd, z, dx, Gs, ms, rs, ws=ws_b)
    torch.cuda.synchronize()

    rng = np.random.default_rng(7)
    ts = _sample(rng, T, 48)
    y_s, z_s, dx_s = _rows(y, ts), _rows(z, ts), _rows(dx, ts)
    x64 = x.astype(np.float64)
    dx_ref = np.zeros((len(ts), n))
    mo = ro = 0
    for k, (m, r) in enumerate(zip(ms, rs)):
        y_ref, z_ref = oc.ref_fwd(x[ts], Ws[k], seeds[k], r)
        assert oc.rel_fro(y_s[:, mo:mo + m], y_ref) <= TOL
        assert oc.rel_fro(z_s[:, ro:ro + r], z_ref) <= TOL
        dx_ref += oc.ref_bwd(dy[ts, mo:mo + m], z_ref, Ws[k])[0]
        # G^ columns: sums over all tokens of the oracle's own z
        cs = _sample(rng, m, 16)
        z_full = x64 @ projection(seeds[k], n, r)
        G_ref = z_full.T @ dy[:, mo + cs].astype(np.float64)
        assert oc.rel_fro(Gs[k][:, torch.as_tensor(cs, device=dev())].cpu().numpy(), G_ref) <= TOL
        mo += m
        ro += r
    assert oc.rel_fro(dx_s, dx_ref) <= TOL


def test_full_size_step_batched():
    wl = workload("llama-350m")
    t = 3
    layers, host = [], []
    per_block = ((0, 1, 2), (3,), (4, 5), (6,))
    for b in range(len(wl.layers) // 7):
        for grp in per_block:
            Ls = [wl.layers[7 * b + k] for k in grp]
            n, M = Ls[0].n, sum(L.m for L in Ls)
            W_all = normal_bf16_blocked(n, M, seed=5000 + 7 * b + grp[0], scale=0.02)
            Wd = to_dev(W_all, "bf16", ld_for(M, "bf16"))
            mo = 0
            for L in Ls:
                s0 = 9000 + 4 * L.layer_id
                G = normal_bf16_blocked(L.r, L.m, seed=s0, bf16=False)
                Mo = normal_bf16_blocked(L.r, L.m, seed=s0 + 1, scale=0.1, bf16=False)
                V = (Mo * Mo + 1e-3 * np.abs(normal_bf16_blocked(L.r, L.m, seed=s0 + 2, bf16=False))).astype(np.float32)
                d = dict(W=Wd[:, mo:mo + L.m], G=torch.from_numpy(G).to(dev()), M=torch.from_numpy(Mo).to(dev()),
                         V=torch.from_numpy(V).to(dev()), seed=L.seed, alpha=wl.alpha)
                layers.append(d)
                host.append((L, W_all[:, mo:mo + L.m], G, Mo, V))
                mo += L.m
    W_before = [d["W"].clone() for d in layers]
    ws = workspace(cp.step_batched_workspace_bytes(layers))
    cp.compact_step_batched(layers, t, wl.lr, wl.beta1, wl.beta2, wl.eps, ws=ws)
    torch.cuda.synchronize()
    rng = np.random.default_rng(11)
    for i in range(0, len(layers), 13):
        L, W0, G, Mo, V = host[i]
        cs = _sample(rng, L.m, 8)
        ci = torch.as_tensor(cs, device=dev())
        _, M_ref, V_ref, dW_ref = oc.ref_step(W0[:, cs], G[:, cs], Mo[:, cs], V[:, cs], L.seed, L.r, t, wl.lr,
                                              wl.beta1, wl.beta2, wl.eps, wl.alpha)
        d = layers[i]
        assert np.array_equal(to_np(W_before[i][:, ci]), W0[:, cs].astype(np.float64))
        assert oc.rel_fro(d["M"][:, ci].cpu().numpy(), M_ref) <= 1e-5
        assert oc.rel_fro(d["V"][:, ci].cpu().numpy(), V_ref) <= 1e-5
        # W is bf16 and the update is rounded once (RNE): every updated element
        # lies within one bf16 unit of the exact W + dW, plus the error the bf16
        # operands P and N put into dW (bounded by 2% of the column's largest
        # update; it matters where W + dW is near zero and the unit is small)
        exact = W0[:, cs].astype(np.float64) + dW_ref
        ulp = 2.0 ** (np.floor(np.log2(np.maximum(np.abs(exact), 1e-30))) - 7)
        op_err = 0.02 * np.abs(dW_ref).max(axis=0, keepdims=True)
        assert np.all(np.abs(to_np(d["W"][:, ci]) - exact) <= ulp + op_err)
        # and the update is not lost in the rounding: most elements moved
        assert np.mean(to_np(d["W"][:, ci]) != W0[:, cs]) > 0.5


# One input group per workload at its full token count, every element:
# the group with the most output tiles that the benchmark forms.
EVERY = [
    ("llama-60m", 512, (512, 512, 512), (128, 128, 128)),
    ("roberta-base", 768, (768, 768, 768), (384, 384, 384)),
    ("llama-350m", 1024, (2736, 2736), (128, 128)),
    ("llama-1b-r4", 2048, (2048, 2048, 2048), (512, 512, 512)),
    ("llama-1b-r8", 2048, (2048, 2048, 2048), (256, 256, 256)),
    # the widths of 5461: down (K = 5461, z of 1365 columns) and gate (5461 outputs)
    ("llama-1b-r4", 5461, (2048,), (1365,)),
    ("llama-1b-r8", 2048, (5461,), (256,)),
]
CHUNK = 8192


@pytest.mark.parametrize("case", EVERY, ids=lambda c: "{}-n{}-m{}".format(c[0], c[1], "+".join(map(str, c[2]))))
def test_full_size_every_element(case):
    from gpu_util import BF16_U, assert_elementwise
    name, n, ms, rs = case
    wl = workload(name)
    T = wl.tokens
    M, R = sum(ms), sum(rs)
    seeds = tuple(((3 + k) << 32) | 1 for k in range(len(ms)))
    x = normal_bf16_blocked(T, n, seed=4000 + n)
    W = normal_bf16_blocked(n, M, seed=4100 + M, scale=0.02)
    dy = normal_bf16_blocked(T, M, seed=4200 + M, scale=0.01)
    zs = normal_bf16_blocked(T, R, seed=4300 + R, scale=float(np.sqrt(n / rs[0])))
    xd = to_dev(x, "bf16", ld_for(n, "bf16"))
    Wd = to_dev(W, "bf16", ld_for(M, "bf16"))
    dyd = to_dev(dy, "bf16", ld_for(M, "bf16"))
    zsd = to_dev(zs, "bf16", ld_for(R, "bf16"))
    y = empty(T, M, "bf16", ld_for(M, "bf16"), fill=float("nan"))
    z = empty(T, R, "bf16", ld_for(R, "bf16"), fill=float("nan"))
    dx = empty(T, n, "bf16", ld_for(n, "bf16"), fill=float("nan"))
    ws_f = workspace(cp.fwd_group_workspace_bytes(n, ms, rs))
    ws_b = workspace(cp.bwd_group_workspace_bytes(T, n, ms, rs))
    if len(ms) > 1:
        cp.compact_fwd_group(xd, Wd, y, z, ms, rs, seeds, ws=ws_f)
    else:
        cp.compact_fwd(xd, Wd, y, z, seeds[0], ws=ws_f)
    Gs = [torch.full((r, m), float("nan"), dtype=torch.float32, device=dev()) for m, r in zip(ms, rs)]
    cp.compact_bwd_group(dyd, Wd, z, dx, Gs, ms, rs, ws=ws_b)      # as the benchmark chains them
    Gz = [torch.full((r, m), float("nan"), dtype=torch.float32, device=dev()) for m, r in zip(ms, rs)]
    cp.compact_bwd_group(dyd, None, zsd, None, Gz, ms, rs, ws=ws_b)  # on a synthetic z
    torch.cuda.synchronize()
    Ps = [projection(s, n, r) for s, r in zip(seeds, rs)]
    W64 = W.astype(np.float64)
    aW = np.abs(W64)
    G_ref = [np.zeros((r, m)) for m, r in zip(ms, rs)]
    Gz_ref = [np.zeros((r, m)) for m, r in zip(ms, rs)]
    Gz_abs = [np.zeros((r, m)) for m, r in zip(ms, rs)]
    for r0 in range(0, T, CHUNK):
        r1 = min(T, r0 + CHUNK)
        xc, dyc, zsc = x[r0:r1].astype(np.float64), dy[r0:r1].astype(np.float64), zs[r0:r1].astype(np.float64)
        ax = np.abs(xc)
        yc, zc, dxc = to_np(y[r0:r1]), to_np(z[r0:r1]), to_np(dx[r0:r1])
        assert_elementwise(yc, xc @ W64, ax @ aW, n, what=f"y rows {r0}..{r1}")
        assert_elementwise(dxc, dyc @ W64.T, np.abs(dyc) @ aW.T, M, what=f"dx rows {r0}..{r1}")
        mo = ro = 0
        for k, (m, r) in enumerate(zip(ms, rs)):
            z_ref = xc @ Ps[k]
            assert_elementwise(zc[:, ro:ro + r], z_ref, ax @ np.abs(Ps[k]), n, operand_rel=BF16_U * 1.001,
                               what=f"z[{k}] rows {r0}..{r1}")
            G_ref[k] += z_ref.T @ dyc[:, mo:mo + m]
            Gz_ref[k] += zsc[:, ro:ro + r].T @ dyc[:, mo:mo + m]
            Gz_abs[k] += np.abs(zsc[:, ro:ro + r]).T @ np.abs(dyc[:, mo:mo + m])
            mo += m
            ro += r
    for k in range(len(ms)):
        # chained: the GPU's G^ sums its own (bf16) z, the oracle its exact z
        assert oc.rel_fro(Gs[k].cpu().numpy(), G_ref[k]) <= TOL
        got = Gz[k].cpu().numpy().astype(np.float64)
        assert_elementwise(got, Gz_ref[k], Gz_abs[k], T + 256, bf16_out=False, what=f"G^[{k}] (synthetic z)")
        assert oc.rel_fro(got, Gz_ref[k]) <= TOL
