"""Oracle for the CompAct linear layer in fp64 — test infrastructure only.

Each function follows one passage of the paper (CompAct, §3.2 and §3.3):

* ``ref_fwd``   Alg. 1: o = x W and the saved activation z = x P.
* ``ref_bwd``   Alg. 2: G^ = z^T dL/do (r x m) and dL/dx = dL/do W^T.
* ``ref_adam``  Alg. 3, first block: Adam moments on the r x m compressed
                gradient, bias correction, N = M^ / (sqrt(V^) + eps).
* ``ref_step``  Alg. 3: ref_adam, then W <- W - lr * alpha * P N with P
                re-sampled from the layer seed.
* ``next_seed`` Alg. 3, end: t <- t + 1 and the seed advances every T steps.
* ``memory_elements`` Table 1, CompAct column.

Readings where the paper is silent or inconsistent:

* The Adam of Alg. 3 (bias-corrected, eps added to sqrt(V^)) is used, not the
  §3.2 display (no bias correction, eps inside the root).
* Alg. 3 overwrites M_t, V_t with their bias-corrected values; here the
  corrected values are temporaries and the stored moments stay uncorrected
  (otherwise the correction would compound from step to step).
* The step index used in the bias correction is 1-based (t = 1 on the first
  step), which is the only reading that avoids 1 - beta^0 = 0.
* Descent sign: W_{t+1} = W_t - lr * G~ (§3.2, Alg. 3).
* No bias term and no weight decay (§3.1 drops the bias).

Everything here is numpy float64; inputs given in a narrower type are taken as
the exact values they hold.
"""
from __future__ import annotations

import numpy as np

from .pstream import projection

F64 = np.float64


def _f64(a):
    return np.asarray(a, dtype=F64)


def ref_fwd(x, W, seed: int, r: int, identity: bool = False, sparse_s: int = 0):
    """Alg. 1.  x: (T, n), W: (n, m) -> (o (T, m), z (T, r)).  sparse_s > 0
    takes the sparse JL projection with that many draws per row (§5)."""
    x, W = _f64(x), _f64(W)
    n = x.shape[1]
    P = projection(seed, n, r, identity, sparse_s)
    o = x @ W
    z = x @ P
    return o, z


def ref_bwd(dy, z, W):
    """Alg. 2.  dy: (T, m), z: (T, r), W: (n, m) -> (dx (T, n), Ghat (r, m))."""
    dy, z, W = _f64(dy), _f64(z), _f64(W)
    Ghat = z.T @ dy
    dx = dy @ W.T
    return dx, Ghat


def ref_adam(Ghat, M, V, t: int, beta1: float, beta2: float, eps: float):
    """Alg. 3 moments.  Returns (M_t, V_t, N_t) with M_t, V_t uncorrected."""
    if t < 1:
        raise ValueError("step index t is 1-based")
    G, M, V = _f64(Ghat), _f64(M), _f64(V)
    b1, b2 = F64(beta1), F64(beta2)
    M_t = b1 * M + (F64(1) - b1) * G
    V_t = b2 * V + (F64(1) - b2) * G * G
    M_hat = M_t / (F64(1) - b1 ** t)
    V_hat = V_t / (F64(1) - b2 ** t)
    N_t = M_hat / (np.sqrt(V_hat) + F64(eps))
    return M_t, V_t, N_t


def ref_step(W, Ghat, M, V, seed: int, r: int, t: int, lr: float, beta1: float,
             beta2: float, eps: float, alpha: float, identity: bool = False,
             rho: str = "adam", sparse_s: int = 0):
    """Alg. 3.  Returns (W_{t+1}, M_t, V_t, dW) with dW = W_{t+1} - W_t.

    ``rho="sgd"`` replaces the Adam normalisation by the identity (N = G^);
    it exists only to test the unbiasedness of the decompression."""
    W = _f64(W)
    n = W.shape[0]
    if rho == "adam":
        M_t, V_t, N_t = ref_adam(Ghat, M, V, t, beta1, beta2, eps)
    elif rho == "sgd":
        M_t, V_t, N_t = _f64(M), _f64(V), _f64(Ghat)
    else:
        raise ValueError(rho)
    P = projection(seed, n, r, identity, sparse_s)
    G_tilde = F64(alpha) * (P @ N_t)
    dW = -F64(lr) * G_tilde
    return W + dW, M_t, V_t, dW


def next_seed(seed: int, t: int, T: int):
    """Alg. 3 schedule.  ``t`` is the 1-based index of the step just taken with
    ``seed``; returns the seed for step t + 1.  T <= 0 means never re-seed."""
    if t < 1:
        raise ValueError("step index t is 1-based")
    seed = int(seed)
    if T > 0 and t % T == 0:
        seed = (seed + 1) & ((1 << 64) - 1)
    return seed


def memory_elements(b: int, l: int, n: int, m: int, r: int):
    """Table 1 (CompAct column): element counts per linear layer, against the
    uncompressed layer (Original column)."""
    return {
        "compact": {"weights": m * n, "gradients": m * r,
                    "optim_states": 2 * m * r, "activations": b * l * r},
        "original": {"weights": m * n, "gradients": m * n,
                     "optim_states": 2 * m * n, "activations": b * l * n},
    }


def rel_fro(a, b):
    """Relative Frobenius error |a - b|_F / |b|_F (b is the reference)."""
    a, b = _f64(a), _f64(b)
    den = np.linalg.norm(b)
    num = np.linalg.norm(a - b)
    return float(num / den) if den > 0 else float(num)
