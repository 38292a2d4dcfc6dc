"""PyTorch modules over the CompAct ABI: linear layers whose backward keeps only
the compressed activation z = x P (Alg. 1) and whose weight gradient is the
r x m compressed gradient G^ = z^T dL/do (Alg. 2), and an optimizer that runs
Alg. 3 (Adam on the r x m moments, W -= lr alpha P N, the seed schedule) for
all of them in a few batched launches.

    lin = CompActLinear(n, m, r)                  # one projection
    qkv = CompActGroup(n, [d, d, d], [r, r, r])   # projections sharing x
    opt = CompActAdam([lin, qkv], lr=1e-3, reseed_period=200)
    loss(lin(x), qkv(x)).backward(); opt.step(); opt.zero_grad()

The weights are bf16 tensors outside autograd (no dense weight gradient is
ever formed); inputs are bf16 of shape (..., n).  Every arithmetic step runs in
the library's HIP kernels; these classes only hold buffers and call the ABI.
"""
from __future__ import annotations

import torch

from . import (bwd_group_workspace_bytes, compact_bwd_group, compact_fwd, compact_fwd_group, compact_next_seed,
               compact_step_batched, fwd_group_workspace_bytes, fwd_workspace_bytes, prepare_layers,
               step_batched_workspace_bytes)

__all__ = ["CompActLinear", "CompActGroup", "CompActAdam", "WorkspacePool"]


class WorkspacePool:
    """One growing scratch buffer per (device, purpose), shared by all modules:
    calls on one stream run in order, so consecutive calls may reuse it."""

    _bufs = {}

    @classmethod
    def get(cls, device, purpose, nbytes):
        key = (str(device), purpose)
        buf = cls._bufs.get(key)
        if buf is None or buf.numel() < nbytes:
            buf = torch.empty(max(int(nbytes), 256), dtype=torch.uint8, device=device)
            cls._bufs[key] = buf
        return buf


def _empty2d(rows, cols, dtype, device):
    """(rows, cols) view of a buffer whose rows are padded to a multiple of 8."""
    buf = torch.empty(rows, (cols + 7) // 8 * 8, dtype=dtype, device=device)
    return buf[:, :cols]


def _as_abi(t):
    """A 2-D view the ABI accepts (unit column stride, leading dimension a
    multiple of 8, 16-byte aligned), copying only when t is not one."""
    if t.stride(1) == 1 and t.stride(0) % 8 == 0 and t.data_ptr() % 16 == 0:
        return t
    out = _empty2d(t.shape[0], t.shape[1], t.dtype, t.device)
    out.copy_(t)
    return out


def _flat(x, n):
    if x.dtype != torch.bfloat16:
        raise TypeError("CompAct modules take bf16 inputs")
    if x.shape[-1] != n:
        raise ValueError(f"last dimension {x.shape[-1]} != {n}")
    return _as_abi(x.reshape(-1, n))


class _GroupFn(torch.autograd.Function):
    """y = x [W_0 | W_1 | ...] with z_j = x P_j saved for the backward."""

    @staticmethod
    def forward(ctx, x2, anchor, mod):
        T = x2.shape[0]
        y = _empty2d(T, mod.msum, torch.bfloat16, x2.device)
        z = _empty2d(T, mod.rsum, torch.bfloat16, x2.device)
        if len(mod.ms) == 1:
            ws = WorkspacePool.get(x2.device, "fwd", fwd_workspace_bytes(mod.n, mod.ms[0], mod.rs[0]))
            compact_fwd(x2, mod.weight, y, z, mod.seeds[0], proj=mod.proj, ws=ws)
        else:
            ws = WorkspacePool.get(x2.device, "fwd", fwd_group_workspace_bytes(mod.n, mod.ms, mod.rs))
            compact_fwd_group(x2, mod.weight, y, z, mod.ms, mod.rs, mod.seeds, proj=mod.proj, ws=ws)
        ctx.mod = mod
        ctx.save_for_backward(z)  # T x sum(r): the activation CompAct keeps instead of x
        return y

    @staticmethod
    def backward(ctx, dy):
        (z,) = ctx.saved_tensors
        mod = ctx.mod
        dy = _as_abi(dy.to(torch.bfloat16))
        T = dy.shape[0]
        dx = None
        if ctx.needs_input_grad[0]:
            dx = _empty2d(T, mod.n, torch.bfloat16, dy.device)
        # Alg. 2 for the whole group in one call: dL/dx summed over the
        # projections (one GEMM over the concatenated weight) and every G^_j,
        # added to the G^ of earlier backward passes until zero_grad (the
        # library's accumulate mode)
        ws = WorkspacePool.get(dy.device, "bwd", bwd_group_workspace_bytes(T, mod.n, mod.ms, mod.rs))
        compact_bwd_group(dy, mod.weight if dx is not None else None, z, dx, mod.ghat, mod.ms, mod.rs, ws=ws,
                          accumulate=mod.grad_ready)
        mod.grad_ready = True
        return dx, None, None


class CompActGroup(torch.nn.Module):
    """Projections j = 0 .. k-1 of one input x: y = [x W_0 | x W_1 | ...]
    (n -> sum(ms)), each with its own rank rs[j] and seed.  Every width and rank
    but the last must be a multiple of 8 (the ABI's column slices).  proj:
    "gaussian" (§3.3) or "sparse-jl[:s]" (the sparse JL projection of §5)."""

    def __init__(self, n, ms, rs, seeds=None, alpha=1.0, device="cuda", weight=None, proj="gaussian"):
        super().__init__()
        self.proj = proj
        self.n, self.ms, self.rs = int(n), [int(m) for m in ms], [int(r) for r in rs]
        self.msum, self.rsum = sum(self.ms), sum(self.rs)
        self.alpha = float(alpha)
        self.seeds = [int(s) for s in (seeds or [(j + 1) << 32 for j in range(len(self.ms))])]
        if weight is None:
            weight = (0.02 * torch.randn(self.n, self.msum, device=device)).to(torch.bfloat16)
        if tuple(weight.shape) != (self.n, self.msum) or weight.dtype != torch.bfloat16:
            raise ValueError("weight must be a bf16 (n, sum(ms)) tensor")
        if weight.stride(1) != 1 or weight.stride(0) % 8 != 0:
            weight = _as_abi(weight)
        self.register_buffer("weight", weight)
        # An empty tensor that requires grad, so that the backward (and G^) runs
        # even where x itself needs no gradient (the first layer of a network).
        self._anchor = torch.nn.Parameter(torch.empty(0, device=weight.device))
        self.ghat = [torch.zeros(r, m, dtype=torch.float32, device=weight.device) for m, r in zip(self.ms, self.rs)]
        self.exp_avg = [torch.zeros_like(g) for g in self.ghat]
        self.exp_avg_sq = [torch.zeros_like(g) for g in self.ghat]
        self.grad_ready = False

    def weight_slice(self, j):
        mo = sum(self.ms[:j])
        return self.weight[:, mo:mo + self.ms[j]]

    def forward(self, x):
        y = _GroupFn.apply(_flat(x, self.n), self._anchor, self)
        return y.reshape(*x.shape[:-1], self.msum)


class CompActLinear(CompActGroup):
    """One CompAct projection n -> m of rank r (Alg. 1-3)."""

    def __init__(self, n, m, r, seed=None, alpha=1.0, device="cuda", weight=None, proj="gaussian"):
        super().__init__(n, [m], [r], None if seed is None else [seed], alpha, device, weight, proj)


class CompActAdam:
    """Alg. 3 for every projection of the given CompAct modules: Adam on the
    compressed gradients (moments r x m, bias-corrected with the 1-based step
    count) and W -= lr alpha P N, in batched launches; then the seed schedule
    (a new P every `reseed_period` steps).  With reset_on_reseed the moments
    are zeroed when a projection's seed changes."""

    def __init__(self, modules, lr=1e-3, betas=(0.9, 0.999), eps=1e-8, reseed_period=200,
                 reset_on_reseed=False):
        self.modules = list(modules)
        projs = {mod.proj for mod in self.modules}
        if len(projs) != 1:
            raise ValueError("CompActAdam steps modules of one projection kind")
        self.proj = projs.pop()
        self.lr, self.betas, self.eps = float(lr), betas, float(eps)
        self.reseed_period = int(reseed_period)
        self.reset_on_reseed = bool(reset_on_reseed)
        self.t = 0
        self._layers = []
        for mod in self.modules:
            for j in range(len(mod.ms)):
                self._layers.append((mod, j))
        self._batch = prepare_layers([dict(W=mod.weight_slice(j), G=mod.ghat[j], M=mod.exp_avg[j],
                                           V=mod.exp_avg_sq[j], seed=mod.seeds[j], alpha=mod.alpha)
                                      for mod, j in self._layers])
        dev = self.modules[0].weight.device
        self._ws = torch.empty(step_batched_workspace_bytes(self._batch), dtype=torch.uint8, device=dev)

    def zero_grad(self):
        for mod in self.modules:
            mod.grad_ready = False

    @torch.no_grad()
    def step(self):
        if not all(mod.grad_ready for mod in self.modules):
            raise RuntimeError("step() before every module's backward")
        self.t += 1
        self._batch.set_seeds([mod.seeds[j] for mod, j in self._layers])
        compact_step_batched(self._batch, self.t, self.lr, self.betas[0], self.betas[1], self.eps, proj=self.proj,
                             ws=self._ws)
        for mod in self.modules:
            for j in range(len(mod.seeds)):
                new = compact_next_seed(mod.seeds[j], self.t, self.reseed_period)
                if new != mod.seeds[j] and self.reset_on_reseed:
                    mod.exp_avg[j].zero_()
                    mod.exp_avg_sq[j].zero_()
                mod.seeds[j] = new
