"""Multi-step training on a synthetic least-squares problem, through the C ABI.

Linear regression Y = X W* (+ noise) with loss |X W - Y|^2 / (2 T m): its weight
gradient X^T (X W - Y) / T = B W - A has the form of Theorem 1 (A = X^T Y / T,
B = X^T X / T, C = I).  CompAct (Alg. 1-3: forward with z = X P, G^ = z^T dL/do,
Adam on r x m moments, W -= lr alpha P N, P re-sampled every `period` steps)
is compared with uncompressed Adam, which is the same library with the
identity projection (P = I, r = n).  Both policies for the moments at a
re-sample are run: kept (the literal Alg. 3) and reset to zero.

Checked: every CompAct run makes steady progress (the loss at steps 100, 200
and 300 keeps falling), uncompressed Adam falls by 1000x (to the noise floor), CompAct at r = n/2 by 20x and
at r = n/8 (each re-sample explores a new r-dimensional subspace of the n = 512
rows) by at least a third in 300 steps, and the order is Adam <= r = n/2 <=
r = n/8.  On MI355X: 1.1e-6, 1.8e-3 and 4.4e-2 from 1.0e-1.
"""
import numpy as np
import pytest

from synthetic import normal_bf16_blocked

from gpu_util import dev, ld_for, to_dev, workspace

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
cp = pytest.importorskip("paper_2410_15352_amd")

T, N_IN, M_OUT = 4096, 512, 256
STEPS, LR, ALPHA = 300, 2e-3, 1.0


def _problem():
    X = normal_bf16_blocked(T, N_IN, seed=61)
    W_star = normal_bf16_blocked(N_IN, M_OUT, seed=62, scale=0.02)
    noise = normal_bf16_blocked(T, M_OUT, seed=63, scale=1e-3, bf16=False)
    Y = (X.astype(np.float64) @ W_star.astype(np.float64) + noise).astype(np.float32)
    return X, Y


def _train(X, Y, r, proj="gaussian", period=50, reset_moments=False, steps=STEPS):
    Xd = to_dev(X, "bf16", ld_for(N_IN, "bf16"))
    Yd = torch.from_numpy(Y).to(dev())
    W = torch.zeros(N_IN, M_OUT, dtype=torch.float32, device=dev())   # fp32 master weights
    M = torch.zeros(r, M_OUT, dtype=torch.float32, device=dev())
    V = torch.zeros_like(M)
    G = torch.empty_like(M)
    y = torch.empty(T, M_OUT, dtype=torch.bfloat16, device=dev())
    z = torch.empty(T, r, dtype=torch.bfloat16, device=dev())
    ws_f = workspace(cp.fwd_workspace_bytes(N_IN, M_OUT, r))
    ws_b = workspace(cp.bwd_workspace_bytes(T, N_IN, M_OUT, r))
    ws_s = workspace(cp.step_workspace_bytes(N_IN, M_OUT, r, 0))
    seed = 17 << 32
    losses = []
    for t in range(1, steps + 1):
        Wb = W.to(torch.bfloat16)
        cp.compact_fwd(Xd, Wb, y, z, seed, proj=proj, ws=ws_f)
        err = y.float() - Yd
        losses.append(float((err * err).mean()) / 2)
        dy = (err / (T * M_OUT)).to(torch.bfloat16)
        cp.compact_bwd(dy, None, z, None, G, ws=ws_b)
        cp.compact_step(W, G, M, V, seed, t, LR, alpha=ALPHA, proj=proj, dtype="f32", ws=ws_s)
        new_seed = cp.compact_next_seed(seed, t, period)
        if reset_moments and new_seed != seed:
            M.zero_()
            V.zero_()
        seed = new_seed
    torch.cuda.synchronize()
    return np.array(losses)


def test_compact_converges_like_adam():
    X, Y = _problem()
    full = _train(X, Y, N_IN, proj="identity")
    kept = _train(X, Y, N_IN // 8)
    reset = _train(X, Y, N_IN // 8, reset_moments=True)
    half = _train(X, Y, N_IN // 2)
    print("\nloss at steps 1, 50, 100, 200, 300:")
    for name, L in (("adam (P = I)", full), ("compact r=n/8, moments kept", kept),
                    ("compact r=n/8, moments reset", reset), ("compact r=n/2, moments kept", half)):
        print(f"  {name:30s} " + "  ".join(f"{L[i]:.3e}" for i in (0, 49, 99, 199, STEPS - 1)))
    for L in (full, kept, reset, half):
        assert np.all(np.isfinite(L))
    for L in (kept, reset, half):  # Adam reaches the noise floor (~1e-6) by step 200
        assert L[299] < L[199] < L[99] < L[0]
    assert full[-1] < 1e-3 * full[0]
    assert half[-1] < 0.05 * half[0]
    assert kept[-1] < 0.67 * kept[0] and reset[-1] < 0.67 * reset[0]
    assert full[-1] <= half[-1] <= kept[-1]


def test_sparse_jl_converges_like_gaussian():
    # §5: the sparse JL projection performs comparably to the Gaussian
    X, Y = _problem()
    gauss = _train(X, Y, N_IN // 8)
    sparse = _train(X, Y, N_IN // 8, proj="sparse-jl")
    sparse1 = _train(X, Y, N_IN // 8, proj="sparse-jl:1")
    print(f"\nloss at step 300, r = n/8: gaussian {gauss[-1]:.3e}, sparse JL s=8 {sparse[-1]:.3e}, "
          f"s=1 {sparse1[-1]:.3e} (from {gauss[0]:.3e})")
    for L in (sparse, sparse1):
        assert np.all(np.isfinite(L))
        assert L[299] < L[199] < L[99] < L[0]
        assert 0.5 * gauss[-1] < L[-1] < 2.0 * gauss[-1]

