"""Pins for the oracle's fp32 Box-Muller transform and the P stream layout.

The fp32 log / sin / cos series are checked exhaustively over every input the
stream can feed them, against numpy's float64 functions: a wrong or dropped
series coefficient, a wrong reduction constant or a wrong quadrant fails here.
The normals are then checked against the standard normal law (moments and a
Kolmogorov-Smirnov test), and the (i, j) -> counter layout against
element-by-element generation.
"""
import numpy as np
import pytest

from oracle import pstream as ps

F32 = np.float32


def ulp_err(approx_f32, exact_f64):
    """Error in units of the last place of the fp32 value nearest the exact one."""
    exact32 = exact_f64.astype(F32)
    ulp = np.spacing(np.abs(exact32)).astype(np.float64)
    return np.abs(approx_f32.astype(np.float64) - exact_f64) / ulp


def test_log_exhaustive_over_radius_codes():
    ka = np.arange(1 << 23, dtype=np.uint32)
    u = (2 * ka + 1).astype(F32) * F32(2.0 ** -24)
    assert np.all(u.astype(np.float64) == (2 * ka.astype(np.float64) + 1) * 2.0 ** -24)
    got = ps.log_f32(u)
    exact = np.log(u.astype(np.float64))
    err = ulp_err(got, exact)
    assert err.max() <= 4.0, err.max()


def test_sin_cos_exhaustive_over_reduced_angles():
    c = np.arange(1 << 21, dtype=np.uint32)
    x = (2 * c + 1).astype(F32) * F32(2.0 ** -23) * ps.HALF_PI_F32
    assert x.max() <= np.pi / 4
    xs = x.astype(np.float64)
    assert ulp_err(ps.sin_f32(x), np.sin(xs)).max() <= 2.0
    assert ulp_err(ps.cos_f32(x), np.cos(xs)).max() <= 2.0


def test_radius_exhaustive():
    a = np.arange(1 << 23, dtype=np.uint32) << np.uint32(9)
    rho = ps.radius_f32(a)
    u = ((a >> 9).astype(np.float64) * 2 + 1) * 2.0 ** -24
    exact = np.sqrt(-2.0 * np.log(u))
    assert ulp_err(rho, exact).max() <= 3.0
    # truncation of the radius: u >= 2^-24 bounds |g| by sqrt(48 ln 2)
    assert rho.max() <= np.sqrt(48 * np.log(2.0)) * (1 + 1e-6)
    assert rho.min() > 0


def test_angle_exhaustive_against_exact_angle():
    b = np.arange(1 << 24, dtype=np.uint32) << np.uint32(8)
    ct, st = ps.angle_cs_f32(b)
    theta = 2 * np.pi * ((b >> 8).astype(np.float64) + 0.5) / 2.0 ** 24
    # absolute error: fp32 reduction constant + series, both ~1e-7
    assert np.abs(ct - np.cos(theta)).max() < 3e-7
    assert np.abs(st - np.sin(theta)).max() < 3e-7
    assert np.abs(ct.astype(np.float64) ** 2 + st.astype(np.float64) ** 2 - 1).max() < 5e-7


def test_normals_are_standard_normal():
    from scipy import stats
    g = ps.gaussian_raw(0x5EED, 1 << 12, 1 << 10).ravel().astype(np.float64)  # 4M samples
    n = g.size
    assert abs(g.mean()) < 5 / np.sqrt(n)
    assert abs(g.var() - 1) < 5 * np.sqrt(2.0 / n)
    # kurtosis of N(0,1) is 3 (sd of the estimate ~ sqrt(24/n))
    kurt = np.mean(g ** 4) / g.var() ** 2
    assert abs(kurt - 3) < 5 * np.sqrt(24.0 / n)
    ks = stats.kstest(g[: 1 << 20], "norm")
    assert ks.pvalue > 1e-4
    assert np.abs(g).max() <= np.sqrt(48 * np.log(2.0)) * (1 + 1e-6)


def test_stream_layout_elementwise():
    seed = (3 << 32) | 17
    n, r = 11, 5  # n not a multiple of 4: last quad partly discarded
    G = ps.gaussian_raw(seed, n, r)
    assert G.shape == (n, r) and G.dtype == F32
    for i in range(n):
        for j in range(r):
            assert G[i, j] == ps.gaussian_element(seed, i, j)
    # a taller matrix shares its leading rows (counter depends on (i, j) only)
    G2 = ps.gaussian_raw(seed, 37, r)
    assert np.array_equal(G2[:n], G)
    G3 = ps.gaussian_raw(seed, n, 9)
    assert np.array_equal(G3[:, :r], G)


def test_stream_pairs_follow_definition():
    seed = 42
    k0, k1 = ps.seed_key(seed)
    G = ps.gaussian_raw(seed, 8, 3)
    for p in range(2):
        for j in range(3):
            w = [int(v) for v in ps.philox4x32_10(p, j, 0, 0, k0, k1)]
            for half, (a, b) in enumerate(((w[0], w[1]), (w[2], w[3]))):
                rho = float(ps.radius_f32(np.array([a], np.uint32))[0])
                ct, st = ps.angle_cs_f32(np.array([b], np.uint32))
                assert G[4 * p + 2 * half, j] == F32(rho) * ct[0]
                assert G[4 * p + 2 * half + 1, j] == F32(rho) * st[0]


def test_distinct_seeds_are_uncorrelated():
    a = ps.gaussian_raw(1 << 32, 256, 64).ravel().astype(np.float64)
    b = ps.gaussian_raw(2 << 32, 256, 64).ravel().astype(np.float64)
    c = ps.gaussian_raw((1 << 32) + 1, 256, 64).ravel().astype(np.float64)
    lim = 5 / np.sqrt(a.size)
    assert abs(np.corrcoef(a, b)[0, 1]) < lim
    assert abs(np.corrcoef(a, c)[0, 1]) < lim


def test_projection_scale_and_identity():
    P = ps.projection(9, 16, 4)
    assert np.array_equal(P, ps.gaussian_raw(9, 16, 4).astype(np.float64) / 2.0)
    assert np.array_equal(ps.projection(0, 6, 6, identity=True), np.eye(6))
    with pytest.raises(ValueError):
        ps.projection(0, 6, 5, identity=True)
