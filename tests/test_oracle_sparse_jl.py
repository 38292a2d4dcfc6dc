"""Pins for the oracle's sparse Johnson-Lindenstrauss projection (the sparse JL
matrices of the ablation, §5; after Dasgupta, Kumar and Sarlos, 2010).

* Brute force: S rebuilt draw by draw from the scalar Philox code
  (philox4_generic, itself pinned against numpy's Philox) equals the
  vectorised construction, entry for entry.
* Structure: integer entries, at most s nonzeros per row, sum of |S| over a row
  at most s and of the parity of s; s = 1 gives exactly one +-1 per row
  (a count sketch).
* E[P P^T] = I over seeds (Monte Carlo band), as for the Gaussian: the property
  that keeps Alg. 3's decompression unbiased; the decompressed SGD update
  P P^T G averages to G.
* Uniform columns (chi-square) and balanced signs; the JL norm property:
  |x P|^2 / |x|^2 has mean 1 and a spread near sqrt(2 / r).
"""
import numpy as np
import pytest
from scipy import stats

from oracle import compact as oc
from oracle.pstream import (SJLT_TAG, U32, U64, philox4_generic, philox4x32_10, projection, seed_key,
                            sparse_jl_raw)


def _brute(seed, n, r, s):
    k0, k1 = (int(v) for v in seed_key(seed))
    S = np.zeros((n, r))
    for i in range(n):
        for q in range(s):
            w = philox4_generic((i, q >> 1, SJLT_TAG, 0), (k0, k1), wordbits=32)
            a, b = (w[0], w[1]) if q % 2 == 0 else (w[2], w[3])
            S[i, (a * r) >> 32] += -1.0 if b >> 31 else 1.0
    return S


@pytest.mark.parametrize("seed,n,r,s", [(1, 7, 5, 3), ((9 << 32) | 77, 13, 8, 8), (2**64 - 1, 6, 1, 4),
                                        (12345, 9, 16, 1), (3 << 40, 5, 3, 64)])
def test_matches_draw_by_draw_construction(seed, n, r, s):
    assert np.array_equal(sparse_jl_raw(seed, n, r, s), _brute(seed, n, r, s))


@pytest.mark.parametrize("s", [1, 2, 3, 8, 16])
def test_row_structure(s):
    n, r = 512, 64
    S = sparse_jl_raw(7 << 32, n, r, s)
    assert np.array_equal(S, np.round(S))
    assert np.all((S != 0).sum(1) <= s)
    assert np.all(np.abs(S).sum(1) <= s)
    assert np.all((S.sum(1) - s) % 2 == 0)          # every draw adds +-1
    if s == 1:
        assert np.all((S != 0).sum(1) == 1) and np.all(np.abs(S).sum(1) == 1)
    P = projection(7 << 32, n, r, sparse_s=s)
    assert np.allclose(P, S / np.sqrt(s))


def test_expected_outer_product_is_identity():
    n, r, s, N = 12, 6, 4, 4000
    acc = np.zeros((n, n))
    for k in range(N):
        P = projection((k + 1) << 32, n, r, sparse_s=s)
        acc += P @ P.T
    mean = acc / N
    # per sample: diagonal = 1 + (collision terms), off-diagonal entries have
    # variance <= s * s / (r s^2) = 1 / r; a 5 sigma band over N samples
    assert np.abs(np.diag(mean) - 1).max() < 5 * np.sqrt(2.0 / (r * N)) + 1e-12
    off = mean - np.diag(np.diag(mean))
    assert np.abs(off).max() < 5 * np.sqrt(1.0 / (r * N))
    # a mis-scaled projection (1/s instead of 1/sqrt(s)) fails the diagonal
    assert np.abs(np.diag(mean) - 1).max() < 0.05


def test_decompressed_sgd_update_is_unbiased():
    rng = np.random.Generator(np.random.PCG64(31))
    T, n, m, r, s, N = 32, 6, 4, 3, 2, 6000
    x = rng.standard_normal((T, n))
    dy = rng.standard_normal((T, m))
    W = np.zeros((n, m))
    G_full = x.T @ dy
    acc = np.zeros((n, m))
    for k in range(N):
        seed = (k + 1) << 32
        _, z = oc.ref_fwd(x, W, seed, r, sparse_s=s)
        _, G = oc.ref_bwd(dy, z, W)
        _, _, _, dW = oc.ref_step(W, G, np.zeros_like(G), np.zeros_like(G), seed, r, 1, lr=1.0, beta1=0.9,
                                  beta2=0.999, eps=1e-8, alpha=1.0, rho="sgd", sparse_s=s)
        acc += -dW
    mean = acc / N
    tol = 6 * np.linalg.norm(G_full) / np.sqrt(r * N)
    assert np.abs(mean - G_full).max() < tol
    assert oc.rel_fro(mean, G_full) < 0.1


def test_columns_uniform_and_signs_balanced():
    n, r, s = 4096, 64, 8
    S = sparse_jl_raw(99, n, r, s)
    # draws per column, counted from the words (two draws of opposite sign on
    # one column cancel in S)
    cols = np.zeros(r)
    k0, k1 = seed_key(99)
    i = np.arange(n, dtype=U32)[:, None]
    p = np.arange(s // 2, dtype=U32)[None, :]
    w0, w1, w2, w3 = philox4x32_10(i, p, U32(SJLT_TAG), U32(0), k0, k1)
    a = np.concatenate([w0.ravel(), w2.ravel()])
    b = np.concatenate([w1.ravel(), w3.ravel()])
    col = ((a.astype(U64) * U64(r)) >> U64(32)).astype(np.int64)
    np.add.at(cols, col, 1)
    assert stats.chisquare(cols).pvalue > 1e-4
    plus = np.count_nonzero((b >> U32(31)) == 0)
    assert abs(plus - a.size / 2) < 5 * np.sqrt(a.size / 4)
    # S holds these draws: |S| sums to at most their number, with equality
    # less the cancelled pairs
    assert np.abs(S).sum() <= a.size and (a.size - np.abs(S).sum()) % 2 == 0


def test_norm_preservation():
    rng = np.random.Generator(np.random.PCG64(5))
    n, r, s = 1024, 128, 8
    P = projection(3 << 32, n, r, sparse_s=s)
    X = rng.standard_normal((400, n))
    ratio = np.square(X @ P).sum(1) / np.square(X).sum(1)
    assert abs(ratio.mean() - 1) < 0.03
    assert 0.6 * np.sqrt(2 / r) < ratio.std() < 1.5 * np.sqrt(2 / r)
