"""A LLaMA decoder block and model whose linear layers are CompAct layers, in the
setup of the paper's pretraining experiments (App. B, App. E):

* q, k, v (one input group) and gate, up (one input group) and down are CompAct
  layers (Alg. 1-3); the attention output projection stays uncompressed,
  because its input is the attention output that flash attention keeps anyway
  (App. B.2, "CompAct and FlashAttention").
* Everything runs in bf16; RMSNorm saves its input and the b x l inverse RMS
  only (Table 7 counts no type conversion); attention is flash attention.
* With rank=None every linear layer is an ordinary bf16 layer (the baseline).

The saved activations of one block are then exactly Table 7's list:
    x1, rstd1 | x2 (baseline) or z_q, z_k, z_v | q, k, v, two b x h x l
    buffers, x3 (shared by o) | x5, rstd2 | x6 or z_gate, z_up | x_gate, x_up
    (one storage), x_act | x7 or z_down
and block_saved_bytes() gives that sum.  Rotary embeddings are left out: they
save no activations and do not touch the linear layers.
"""
from __future__ import annotations

import torch
from torch.nn.attention import SDPBackend, sdpa_kernel

from .nn import CompActAdam, CompActGroup, CompActLinear

__all__ = ["RMSNorm", "DenseLinear", "LlamaBlock", "LlamaModel", "block_saved_bytes", "make_optimizers"]


def _pad8(c):
    return (c + 7) // 8 * 8


class _RMSNormFn(torch.autograd.Function):
    """y = x / rms(x) * g over the last dimension, saving x and 1/rms only."""

    @staticmethod
    def forward(ctx, x, g, eps):
        xf = x.float()
        rstd = torch.rsqrt(xf.square().mean(-1) + eps)
        ctx.save_for_backward(x, rstd, g)
        return (xf * rstd.unsqueeze(-1) * g.float()).to(x.dtype)

    @staticmethod
    def backward(ctx, dy):
        x, rstd, g = ctx.saved_tensors
        xhat = x.float() * rstd.unsqueeze(-1)
        dyf = dy.float()
        gdy = dyf * g.float()
        dx = rstd.unsqueeze(-1) * (gdy - xhat * (gdy * xhat).mean(-1, keepdim=True))
        dg = (dyf * xhat).reshape(-1, x.shape[-1]).sum(0)
        return dx.to(x.dtype), dg.to(g.dtype), None


class RMSNorm(torch.nn.Module):
    def __init__(self, d, eps=1e-6, device="cuda"):
        super().__init__()
        self.weight = torch.nn.Parameter(torch.ones(d, dtype=torch.bfloat16, device=device))
        self.eps = eps

    def forward(self, x):
        return _RMSNormFn.apply(x, self.weight, self.eps)


class DenseLinear(torch.nn.Module):
    """y = x W with W (n, m) a bf16 parameter: the uncompressed layer."""

    def __init__(self, n, m, device="cuda", weight=None):
        super().__init__()
        if weight is None:
            weight = (0.02 * torch.randn(n, m, device=device)).to(torch.bfloat16)
        self.weight = torch.nn.Parameter(weight)

    def forward(self, x):
        return (x.reshape(-1, x.shape[-1]) @ self.weight).reshape(*x.shape[:-1], self.weight.shape[1])


class LlamaBlock(torch.nn.Module):
    """Pre-norm LLaMA block on (b, l, d) bf16 input.  rank: the CompAct rank of
    the d-input layers (q, k, v, gate, up) and rank_down that of down
    (default ffn * rank / d); None for the uncompressed baseline.  compress_o
    also makes the attention output projection a CompAct layer (which saves
    memory only where attention does not keep its output)."""

    def __init__(self, d, heads, ffn, rank=None, rank_down=None, seeds=None, alpha=1.0,
                 compress_o=False, device="cuda", weights=None, proj="gaussian"):
        super().__init__()
        self.d, self.heads, self.ffn = d, heads, ffn
        self.rank = rank
        self.rank_down = (rank_down or max(1, ffn * rank // d)) if rank else None
        self.compress_o = bool(compress_o and rank)
        Wqkv, Wo, Wgu, Wdown = weights if weights is not None else (None,) * 4
        seeds = list(seeds) if seeds is not None else [(j + 1) << 32 for j in range(7)]
        self.norm1 = RMSNorm(d, device=device)
        self.norm2 = RMSNorm(d, device=device)
        if rank:
            self.qkv = CompActGroup(d, [d] * 3, [rank] * 3, seeds=seeds[0:3], alpha=alpha, device=device,
                                    weight=Wqkv, proj=proj)
            self.gu = CompActGroup(d, [ffn] * 2, [rank] * 2, seeds=seeds[4:6], alpha=alpha, device=device,
                                   weight=Wgu, proj=proj)
            self.down = CompActLinear(ffn, d, self.rank_down, seed=seeds[6], alpha=alpha, device=device,
                                      weight=Wdown, proj=proj)
        else:
            self.qkv = DenseLinear(d, 3 * d, device, Wqkv)
            self.gu = DenseLinear(d, 2 * ffn, device, Wgu)
            self.down = DenseLinear(ffn, d, device, Wdown)
        if self.compress_o:
            self.o = CompActLinear(d, d, rank, seed=seeds[3], alpha=alpha, device=device, weight=Wo, proj=proj)
        else:
            self.o = DenseLinear(d, d, device, Wo)

    def forward(self, x):
        b, l, d = x.shape
        h = self.norm1(x)
        qkv = self.qkv(h.reshape(b * l, d)).reshape(b, l, 3, self.heads, d // self.heads)
        q, k, v = (qkv[:, :, i].transpose(1, 2) for i in range(3))
        with sdpa_kernel([SDPBackend.FLASH_ATTENTION]):
            a = torch.nn.functional.scaled_dot_product_attention(q, k, v, is_causal=True)
        x5 = x + self.o(a.transpose(1, 2).reshape(b * l, d)).reshape(b, l, d)
        h2 = self.norm2(x5)
        gu = self.gu(h2.reshape(b * l, d))
        act = torch.nn.functional.silu(gu[:, :self.ffn]) * gu[:, self.ffn:]
        return x5 + self.down(act).reshape(b, l, d)

    def compact_modules(self):
        return [m for m in (self.qkv, self.o, self.gu, self.down) if isinstance(m, CompActGroup)]


def block_saved_bytes(b, l, d, heads, ffn, rank=None, rank_down=None, compress_o=False):
    """Table 7 for this block: bytes of the activations one block keeps for
    its backward (bf16 tensors, fp32 inverse RMS and attention log-sum-exp,
    two int64 scalars of the attention's dropout state).  A CompAct z of r
    columns is stored with its rows padded to a multiple of 8 elements."""
    T = b * l
    common = (2 * T * d          # x1
              + 4 * T            # 1 / rms(x1)
              + 2 * T * 3 * d    # q, k, v (one storage)
              + 4 * b * heads * l + 16
              + 2 * T * d        # x3, also the input of o
              + 2 * T * d + 4 * T  # x5, 1 / rms(x5)
              + 2 * T * 2 * ffn  # x_gate, x_up (one storage)
              + 2 * T * ffn)     # x_act
    if not rank:
        return common + 2 * T * d + 2 * T * d + 2 * T * ffn   # x2, x6, x7
    rd = rank_down or max(1, ffn * rank // d)
    z = 2 * T * (_pad8(3 * rank) + _pad8(2 * rank) + _pad8(rd))
    if compress_o:
        z += 2 * T * _pad8(rank)
    return common + z


class LlamaModel(torch.nn.Module):
    """Token embedding, n_layers blocks, final RMSNorm and the output layer
    (uncompressed), with the mean cross-entropy of next-token prediction."""

    def __init__(self, vocab, d, heads, ffn, n_layers, rank=None, alpha=1.0, device="cuda", proj="gaussian"):
        super().__init__()
        self.embed = torch.nn.Parameter((0.02 * torch.randn(vocab, d, device=device)).to(torch.bfloat16))
        self.blocks = torch.nn.ModuleList(
            LlamaBlock(d, heads, ffn, rank=rank, alpha=alpha, device=device, proj=proj,
                       seeds=[((7 * i + j + 1) << 32) for j in range(7)])
            for i in range(n_layers))
        self.norm = RMSNorm(d, device=device)
        self.head = DenseLinear(d, vocab, device)

    def forward(self, tokens, targets):
        x = self.embed[tokens]
        for blk in self.blocks:
            x = blk(x)
        logits = self.head(self.norm(x))
        return torch.nn.functional.cross_entropy(logits.reshape(-1, logits.shape[-1]).float(), targets.reshape(-1))

    def compact_modules(self):
        return [m for blk in self.blocks for m in blk.compact_modules()]


def make_optimizers(model, lr=1e-3, betas=(0.9, 0.999), eps=1e-8, reseed_period=200):
    """Adam for the model: CompActAdam (Alg. 3) over the CompAct layers, and
    torch's Adam over every other parameter (embedding, norms, uncompressed
    layers).  Returns the list of optimizers, each with step() and zero_grad()."""
    opts = []
    cms = model.compact_modules()
    if cms:
        opts.append(CompActAdam(cms, lr=lr, betas=betas, eps=eps, reseed_period=reseed_period))
    params = [p for name, p in model.named_parameters() if p.numel() > 0]
    if params:
        opts.append(torch.optim.Adam(params, lr=lr, betas=betas, eps=eps, foreach=True))
    return opts
