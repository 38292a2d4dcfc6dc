"""The oracle trains a small least-squares problem (the gradient form of
Theorem 1) with Alg. 1-3 and re-sampling every 20 steps: the loss falls by a
large factor, the identity projection (P = I, r = n: plain Adam) does at least
as well, and a larger rank does at least as well as a smaller one.  A property
of the method that a wrong sign, a dropped term or a transposed operand in the
oracle's forward, backward or step would break."""
import numpy as np

from oracle import compact as oc

T, N_IN, M_OUT = 256, 32, 16
STEPS, LR = 400, 5e-3


def _train(X, Y, r, identity=False, period=20):
    W = np.zeros((N_IN, M_OUT))
    M = np.zeros((r, M_OUT))
    V = np.zeros((r, M_OUT))
    seed = 3 << 32
    losses = []
    for t in range(1, STEPS + 1):
        y, z = oc.ref_fwd(X, W, seed, r, identity=identity)
        err = y - Y
        losses.append(float((err * err).mean()) / 2)
        _, G = oc.ref_bwd(err / (T * M_OUT), z, W)
        W, M, V, _ = oc.ref_step(W, G, M, V, seed, r, t, LR, 0.9, 0.999, 1e-8, 1.0, identity=identity)
        seed = oc.next_seed(seed, t, period)
    return np.array(losses)


def test_oracle_training_converges():
    g = np.random.Generator(np.random.PCG64(5))
    X = g.standard_normal((T, N_IN))
    W_star = 0.1 * g.standard_normal((N_IN, M_OUT))
    Y = X @ W_star
    full = _train(X, Y, N_IN, identity=True)
    r4 = _train(X, Y, N_IN // 4)
    r2 = _train(X, Y, N_IN // 2)
    for L in (full, r4, r2):
        assert L[-1] < 0.05 * L[0]
    assert full[-1] <= r2[-1] <= r4[-1]
