"""Oracle for the CompAct linear layer in fp64 — test infrastructure only.

Each function states one part of the method (CompAct, §3.2 and §3.3):

* ``ref_fwd``   forward (Alg. 1): the output x W and the kept activation x P.
* ``ref_bwd``   backward (Alg. 2): the input gradient and the compressed
                weight gradient z^T dL/do (r x m).
* ``ref_adam``  Adam on the compressed gradient (Alg. 3): moments and the
                bias-corrected, normalised direction.
* ``ref_step``  the update (Alg. 3): the direction mapped back through the
                re-drawn P, scaled by alpha and the learning rate.
* ``next_seed`` the re-sampling schedule (end of Alg. 3).
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
    """Forward of the compressed layer (§3.2, Alg. 1): the layer output x W and
    the activation kept for the backward pass, x P, with P drawn from the layer
    seed (§3.3).  x: (T, n), W: (n, m) -> ((T, m), (T, r)).  sparse_s > 0 takes
    the sparse JL projection with that many draws per row (§5)."""
    x, W = _f64(x), _f64(W)
    proj = projection(seed, x.shape[1], r, identity, sparse_s)
    return x @ W, x @ proj


def ref_bwd(dy, z, W):
    """Backward of the compressed layer (§3.2, Alg. 2): the input gradient
    dL/do W^T (exact, P does not enter it) and the weight gradient in the
    projected space, z^T dL/do.  dy: (T, m), z: (T, r), W: (n, m) ->
    ((T, n), (r, m))."""
    dy, z, W = _f64(dy), _f64(z), _f64(W)
    return dy @ W.T, z.T @ dy


def ref_adam(Ghat, M, V, t: int, beta1: float, beta2: float, eps: float):
    """Adam on the r x m compressed gradient (§3.2; the bias-corrected form of
    Alg. 3): exponential averages of the gradient and of its square, and the
    normalised step direction built from their bias-corrected values.
    Returns (first moment, second moment, direction); the stored moments are
    the uncorrected averages.  t is the 1-based step index."""
    if t < 1:
        raise ValueError("step index t is 1-based")
    g, mean, sq = _f64(Ghat), _f64(M), _f64(V)
    b1, b2 = F64(beta1), F64(beta2)
    mean = b1 * mean + (F64(1) - b1) * g
    sq = b2 * sq + (F64(1) - b2) * g * g
    mean_unbiased = mean / (F64(1) - b1 ** t)
    sq_unbiased = sq / (F64(1) - b2 ** t)
    return mean, sq, mean_unbiased / (np.sqrt(sq_unbiased) + F64(eps))


def ref_step(W, Ghat, M, V, seed: int, r: int, t: int, lr: float, beta1: float,
             beta2: float, eps: float, alpha: float, identity: bool = False,
             rho: str = "adam", sparse_s: int = 0):
    """One optimizer step of the compressed layer (§3.2, Alg. 3): the Adam
    direction in the projected space is mapped back to the weight space by
    the same P as the forward (re-drawn from the seed, §3.3), scaled by alpha
    and the learning rate, and subtracted from W.
    Returns (new W, first moment, second moment, the change of W).

    ``rho="sgd"`` uses the compressed gradient itself as the direction; it
    exists only to test that the decompressed update is unbiased."""
    W = _f64(W)
    if rho == "adam":
        mean, sq, direction = ref_adam(Ghat, M, V, t, beta1, beta2, eps)
    elif rho == "sgd":
        mean, sq, direction = _f64(M), _f64(V), _f64(Ghat)
    else:
        raise ValueError(rho)
    proj = projection(seed, W.shape[0], r, identity, sparse_s)
    change = -F64(lr) * (F64(alpha) * (proj @ direction))
    return W + change, mean, sq, change


def next_seed(seed: int, t: int, T: int):
    """The re-sampling schedule (§3.3, end of Alg. 3): after the step with
    1-based index ``t``, the layer moves to the next seed (a new P) when t is
    a multiple of the period T; T <= 0 keeps one P for the whole run."""
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
