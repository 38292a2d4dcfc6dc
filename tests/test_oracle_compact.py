"""Pins for the fp64 oracle of Alg. 1-3 (forward, backward, Adam step).

What fixes each result independently of the oracle's own code:

* brute force in exact rational arithmetic (fractions.Fraction) on tiny
  non-square shapes, for o, z, dx and G^ (a transposed operand or a wrong
  index changes the shapes or the values);
* P = I with r = n: the whole step must equal an uncompressed linear layer
  trained by ``torch.optim.Adam`` (a library Adam), for several steps, and
  z must equal x;
* o and dx do not depend on the projection seed (Alg. 1 and Alg. 2 use W only);
* G^ = P^T (x^T dy): the GaLore-with-Q=I identity of §3.2;
* E[P P^T] = I over many seeds (variance 1/r, §3.3), and with an identity
  optimizer the decompressed update P P^T G is an unbiased estimate of G;
* closed forms of Adam at t = 1 and t = 2;
* the seed schedule of Alg. 3 and the memory scaling of Table 1.
"""
import os
import re
from fractions import Fraction

import numpy as np
import pytest

from oracle import compact as oc
from oracle import pstream as ps

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def _frac_matmul(A, B):
    n, k = len(A), len(A[0])
    k2, m = len(B), len(B[0])
    assert k == k2
    return [[sum((A[i][t] * B[t][j] for t in range(k)), Fraction(0)) for j in range(m)]
            for i in range(n)]


def _to_frac(a):
    return [[Fraction(float(v)) for v in row] for row in np.asarray(a, dtype=np.float64)]


def _frac_T(A):
    return [list(col) for col in zip(*A)]


def test_bruteforce_fraction_forward_backward():
    rng = np.random.Generator(np.random.PCG64(5))
    T, n, m, r = 4, 3, 2, 2
    x = rng.standard_normal((T, n))
    W = rng.standard_normal((n, m))
    dy = rng.standard_normal((T, m))
    seed = 77
    o, z = oc.ref_fwd(x, W, seed, r)
    P = ps.projection(seed, n, r)
    fo = _frac_matmul(_to_frac(x), _to_frac(W))
    fz = _frac_matmul(_to_frac(x), _to_frac(P))
    assert o.shape == (T, m) and z.shape == (T, r)
    for i in range(T):
        for j in range(m):
            assert abs(Fraction(float(o[i, j])) - fo[i][j]) <= abs(fo[i][j]) * Fraction(1, 2**50) + Fraction(1, 2**1000)
        for j in range(r):
            assert abs(Fraction(float(z[i, j])) - fz[i][j]) <= abs(fz[i][j]) * Fraction(1, 2**50) + Fraction(1, 2**1000)
    dx, G = oc.ref_bwd(dy, z, W)
    fG = _frac_matmul(_frac_T(_to_frac(z)), _to_frac(dy))
    fdx = _frac_matmul(_to_frac(dy), _frac_T(_to_frac(W)))
    assert G.shape == (r, m) and dx.shape == (T, n)
    for i in range(r):
        for j in range(m):
            assert abs(Fraction(float(G[i, j])) - fG[i][j]) <= abs(fG[i][j]) * Fraction(1, 2**50) + Fraction(1, 2**1000)
    for i in range(T):
        for j in range(n):
            assert abs(Fraction(float(dx[i, j])) - fdx[i][j]) <= abs(fdx[i][j]) * Fraction(1, 2**50) + Fraction(1, 2**1000)


@pytest.mark.parametrize("alpha", [1.0, 0.5])
def test_identity_projection_reduces_to_uncompressed_adam(alpha):
    torch = pytest.importorskip("torch")
    rng = np.random.Generator(np.random.PCG64(11))
    T, n, m = 16, 6, 5
    lr, b1, b2, eps = 1e-2, 0.9, 0.999, 1e-8
    W0 = rng.standard_normal((n, m))
    Wt = torch.nn.Parameter(torch.tensor(W0, dtype=torch.float64))
    opt = torch.optim.Adam([Wt], lr=lr * alpha, betas=(b1, b2), eps=eps, foreach=False)
    W = W0.copy()
    M = np.zeros((n, m))
    V = np.zeros((n, m))
    for t in range(1, 4):
        x = rng.standard_normal((T, n))
        dy = rng.standard_normal((T, m))
        o, z = oc.ref_fwd(x, W, seed=123, r=n, identity=True)
        assert np.array_equal(z, x)
        dx, G = oc.ref_bwd(dy, z, W)
        W, M, V, dW = oc.ref_step(W, G, M, V, 123, n, t, lr, b1, b2, eps, alpha, identity=True)
        # library Adam on the uncompressed gradient dL/dW = x^T dy
        opt.zero_grad()
        Wt.grad = torch.tensor(x.T @ dy, dtype=torch.float64)
        opt.step()
        ref = Wt.detach().numpy()
        assert np.abs(W - ref).max() <= 1e-12 * max(1.0, np.abs(ref).max())
        st = opt.state[Wt]
        assert np.allclose(M, st["exp_avg"].numpy(), rtol=1e-13, atol=0)
        assert np.allclose(V, st["exp_avg_sq"].numpy(), rtol=1e-13, atol=0)


def test_outputs_independent_of_projection_seed():
    rng = np.random.Generator(np.random.PCG64(3))
    x = rng.standard_normal((9, 8))
    W = rng.standard_normal((8, 5))
    dy = rng.standard_normal((9, 5))
    o1, z1 = oc.ref_fwd(x, W, 1, 3)
    o2, z2 = oc.ref_fwd(x, W, 2, 3)
    assert np.array_equal(o1, o2)
    assert not np.allclose(z1, z2)
    dx1, _ = oc.ref_bwd(dy, z1, W)
    dx2, _ = oc.ref_bwd(dy, z2, W)
    assert np.array_equal(dx1, dx2)
    assert np.array_equal(dx1, dy @ W.T)


def test_galore_identity_q_eq_i():
    rng = np.random.Generator(np.random.PCG64(8))
    T, n, m, r = 40, 12, 7, 3
    x = rng.standard_normal((T, n))
    W = rng.standard_normal((n, m))
    dy = rng.standard_normal((T, m))
    seed = (5 << 32) | 2
    _, z = oc.ref_fwd(x, W, seed, r)
    _, G = oc.ref_bwd(dy, z, W)
    P = ps.projection(seed, n, r)
    full = x.T @ dy  # the uncompressed weight gradient
    assert oc.rel_fro(G, P.T @ full) < 1e-12


def test_expected_projection_outer_product_is_identity():
    n, r, S = 8, 4, 20000
    acc = np.zeros((n, n))
    for s in range(S):
        P = ps.projection((s + 1) << 32, n, r)
        acc += P @ P.T
    mean = acc / S
    # per-entry sd of the mean: diag sqrt(2/(r S)), off-diag sqrt(1/(r S))
    sd = np.where(np.eye(n, dtype=bool), np.sqrt(2.0 / (r * S)), np.sqrt(1.0 / (r * S)))
    assert np.all(np.abs(mean - np.eye(n)) < 5 * sd)
    # a mis-scaled projection (variance 1/r^2 or 1) is far outside this band
    assert np.abs(np.diag(mean) - 1).max() < 0.05


def test_decompressed_sgd_update_is_unbiased():
    rng = np.random.Generator(np.random.PCG64(21))
    T, n, m, r, S = 32, 6, 4, 2, 6000
    x = rng.standard_normal((T, n))
    dy = rng.standard_normal((T, m))
    W = np.zeros((n, m))
    G_full = x.T @ dy
    acc = np.zeros((n, m))
    for s in range(S):
        seed = (s + 1) << 32
        _, z = oc.ref_fwd(x, W, seed, r)
        _, G = oc.ref_bwd(dy, z, W)
        _, _, _, dW = oc.ref_step(W, G, np.zeros_like(G), np.zeros_like(G), seed, r, 1,
                                  lr=1.0, beta1=0.9, beta2=0.999, eps=1e-8, alpha=1.0, rho="sgd")
        acc += -dW  # = P P^T G_full
    mean = acc / S
    # each entry of P P^T G has sd about |G| sqrt(1/r) / sqrt(S) per sample
    tol = 6 * np.linalg.norm(G_full) / np.sqrt(r * S)
    assert np.abs(mean - G_full).max() < tol
    assert oc.rel_fro(mean, G_full) < 0.1


def test_adam_closed_forms():
    G1 = np.array([[3.0, -2.0, 0.0], [1e-9, -5e-9, 4.0]])
    b1, b2, eps = 0.9, 0.999, 1e-8
    M1, V1, N1 = oc.ref_adam(G1, 0 * G1, 0 * G1, 1, b1, b2, eps)
    assert np.allclose(M1, 0.1 * G1, rtol=1e-15, atol=0)
    assert np.allclose(V1, 0.001 * G1 ** 2, rtol=1e-15, atol=0)
    assert np.allclose(N1, G1 / (np.abs(G1) + eps), rtol=1e-12, atol=0)
    # the §3.2 display (no bias correction, eps under the root) is a different map
    other = (0.1 * G1) / np.sqrt(0.001 * G1 ** 2 + eps)
    assert np.abs(N1[0, 0] - other[0, 0]) > 1.0
    G2 = np.array([[1.0, 4.0, -1.0], [2.0, 0.5, -3.0]])
    M2, V2, N2 = oc.ref_adam(G2, M1, V1, 2, b1, b2, eps)
    M2x = b1 * 0.1 * G1 + 0.1 * G2
    V2x = b2 * 0.001 * G1 ** 2 + 0.001 * G2 ** 2
    N2x = (M2x / (1 - b1 ** 2)) / (np.sqrt(V2x / (1 - b2 ** 2)) + eps)
    assert np.allclose(M2, M2x, rtol=1e-14, atol=0)
    assert np.allclose(V2, V2x, rtol=1e-14, atol=0)
    assert np.allclose(N2, N2x, rtol=1e-12, atol=0)
    with pytest.raises(ValueError):
        oc.ref_adam(G1, M1, V1, 0, b1, b2, eps)


def test_step_update_closed_form_and_sign():
    rng = np.random.Generator(np.random.PCG64(4))
    n, m, r = 10, 6, 4
    W = rng.standard_normal((n, m))
    G = rng.standard_normal((r, m))
    seed, lr, alpha = 99, 1e-3, 0.25
    W1, M1, V1, dW = oc.ref_step(W, G, 0 * G, 0 * G, seed, r, 1, lr, 0.9, 0.999, 1e-8, alpha)
    P = ps.gaussian_raw(seed, n, r).astype(np.float64) / np.sqrt(r)
    N = G / (np.abs(G) + 1e-8)
    assert np.allclose(dW, -lr * alpha * (P @ N), rtol=1e-12, atol=1e-18)
    assert np.array_equal(W1, W + dW)
    # descent: for a 1-column problem the update opposes P P^T G
    assert np.sum(dW * (P @ G)) < 0


def test_seed_schedule():
    s0 = 7 << 32
    seeds, s = [], s0
    for t in range(1, 11):
        seeds.append(s)  # seed used at step t
        s = oc.next_seed(s, t, 3)
    # steps 1-3 use s0, 4-6 s0+1, 7-9 s0+2, 10 s0+3
    assert seeds == [s0] * 3 + [s0 + 1] * 3 + [s0 + 2] * 3 + [s0 + 3]
    assert oc.next_seed(s0, 5, 1) == s0 + 1
    assert oc.next_seed(s0, 5, 0) == s0  # never re-seed
    assert oc.next_seed(2**64 - 1, 2, 2) == 0


def test_memory_model_matches_table1():
    rows = {}
    with open(os.path.join(GOLDEN, "table1_memory_scaling.txt")) as f:
        for line in f:
            if line.startswith("#") or not line.strip():
                continue
            comp, orig, cpt = line.split()
            rows[comp] = (orig, cpt)

    def evaluate(expr, b, l, n, m, r):
        mult = re.match(r"^(\d*)([a-z]+)$", expr)
        k = int(mult.group(1)) if mult.group(1) else 1
        val = {"b": b, "l": l, "n": n, "m": m, "r": r}
        out = k
        for ch in mult.group(2):
            out *= val[ch]
        return out

    for (b, l, n, m, r) in [(256, 256, 1024, 2736, 128), (32, 512, 768, 3072, 384), (2, 3, 5, 7, 1)]:
        got = oc.memory_elements(b, l, n, m, r)
        for comp, (orig, cpt) in rows.items():
            assert got["original"][comp] == evaluate(orig, b, l, n, m, r)
            assert got["compact"][comp] == evaluate(cpt, b, l, n, m, r)
    # activation bytes stored per layer at LLaMA-350M shapes, bf16: 16 MiB vs 128 MiB
    me = oc.memory_elements(256, 256, 1024, 1024, 128)
    assert me["compact"]["activations"] * 2 == 16 << 20
    assert me["original"]["activations"] * 2 == 128 << 20
