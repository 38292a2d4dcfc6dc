"""Non-finite values propagate through the path and are never masked.

IEEE arithmetic carries a NaN (or an infinity) in an input to exactly the
outputs that depend on it (Alg. 1-3): a NaN in token t of x reaches row t of
y and z; a NaN in dL/do at (t, c) reaches row t of dL/dx, column c of G^, of M
and V, and column c of W (every row of P N's column c sums over N[:, c]).
Every other element stays finite and equal to the result without the NaN.
An infinity in dL/do gives +-inf in that column of G^ and M, inf in V and then
NaN in N (inf / inf), so column c of W is NaN too.
"""
import numpy as np
import pytest

from synthetic import bwd_inputs, fwd_inputs, step_inputs

from gpu_util import dev, empty, ld_for, to_dev, workspace

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
cp = pytest.importorskip("paper_2410_15352_amd")

T, N, M_, R = 600, 512, 1376, 128
T0, C0, I0 = 333, 700, 41


def _nonfinite(t):
    return ~torch.isfinite(t.float())


def _bits_equal(a, b, mask):
    """a and b agree bit for bit outside `mask`."""
    ai = a.contiguous().view(torch.int16 if a.dtype == torch.bfloat16 else torch.int32)
    bi = b.contiguous().view(torch.int16 if b.dtype == torch.bfloat16 else torch.int32)
    return bool(((ai == bi) | mask).all())


@pytest.mark.parametrize("dt", ["bf16", "f32"])
def test_nan_in_x_reaches_its_rows(dt):
    x, W = fwd_inputs(T, N, M_, dt, data_seed=31)
    xd, Wd = to_dev(x, dt, ld_for(N, dt)), to_dev(W, dt, ld_for(M_, dt))
    outs = []
    for poison in (False, True):
        if poison:
            xd[T0, I0] = float("nan")
        y, z = empty(T, M_, dt, ld_for(M_, dt)), empty(T, R, dt, ld_for(R, dt))
        fws = cp.fwd_workspace_bytes(N, M_, R, cp.BF16 if dt == "bf16" else cp.F32)
        cp.compact_fwd(xd, Wd, y, z, 5 << 32, ws=workspace(fws) if fws else None)
        outs.append((y, z))
    torch.cuda.synchronize()
    (y0, z0), (y1, z1) = outs
    rows = torch.zeros(T, 1, dtype=torch.bool, device=dev())
    rows[T0] = True
    for clean, got in ((y0, y1), (z0, z1)):
        assert bool(_nonfinite(got)[T0].all())
        assert not bool(_nonfinite(got)[~rows[:, 0]].any())
        assert _bits_equal(clean, got, rows.expand_as(got))


@pytest.mark.parametrize("value", [float("nan"), float("inf")], ids=["nan", "inf"])
@pytest.mark.parametrize("dt", ["bf16", "f32"])
def test_nonfinite_dy_reaches_dx_ghat_moments_and_w(dt, value):
    code = cp.BF16 if dt == "bf16" else cp.F32
    dy, z, W = bwd_inputs(T, N, M_, R, dt, data_seed=32)
    dyd, zd = to_dev(dy, dt, ld_for(M_, dt)), to_dev(z, dt, ld_for(R, dt))
    Wd = to_dev(W, dt, ld_for(M_, dt))
    _, _, M0, V0 = step_inputs(N, M_, R, dt, t=3, data_seed=33)
    res = []
    for poison in (False, True):
        if poison:
            dyd[T0, C0] = value
        dx = empty(T, N, dt, ld_for(N, dt))
        G = torch.empty(R, M_, dtype=torch.float32, device=dev())
        cp.compact_bwd(dyd, Wd, zd, dx, G, ws=workspace(cp.bwd_workspace_bytes(T, N, M_, R, code)))
        Wn = Wd.clone()
        Md, Vd = torch.from_numpy(M0.copy()).to(dev()), torch.from_numpy(V0.copy()).to(dev())
        cp.compact_step(Wn, G, Md, Vd, 7 << 32, 3, 1e-3, alpha=0.25, dtype=dt,
                        ws=workspace(cp.step_workspace_bytes(N, M_, R, code)))
        res.append((dx, G, Md, Vd, Wn))
    torch.cuda.synchronize()
    clean, bad = res
    row = torch.zeros(T, N, dtype=torch.bool, device=dev())
    row[T0] = True
    col_g = torch.zeros(R, M_, dtype=torch.bool, device=dev())
    col_g[:, C0] = True
    col_w = torch.zeros(N, M_, dtype=torch.bool, device=dev())
    col_w[:, C0] = True
    for (name, mask), c, b in zip((("dx", row), ("G^", col_g), ("M", col_g), ("V", col_g), ("W", col_w)), clean, bad):
        nf = _nonfinite(b)
        assert bool(nf[mask].all()), f"{name}: a dependent element stayed finite"
        assert not bool(nf[~mask].any()), f"{name}: the non-finite value leaked"
        assert _bits_equal(c, b, mask), f"{name}: an independent element changed"
    if value == float("inf"):
        # N = M^ / (sqrt(V^) + eps) = inf / inf: the column of W becomes NaN
        assert bool(torch.isnan(bad[4].float())[:, C0].all())
        assert bool(torch.isinf(bad[1][:, C0]).all())
