"""Seeded synthetic inputs for the CompAct layer workloads.

This module holds no part of the method's arithmetic: it only defines the
layer shapes of the workloads and draws seeded random tensors for them.  Both
the GPU tests / benchmark and the CPU oracle tests take their inputs from here.

Value recipe (the same for every workload): x ~ N(0, 1), W ~ N(0, 0.02^2),
dL/do ~ N(0, 1e-4).  Tensors are drawn with numpy's PCG64 from a data seed
(1234 + layer id by default), in float64, then rounded once to the storage
type: float32, or bfloat16 with round-to-nearest-even.

Layer seeds for the projection: linear k (0..6 = q, k, v, o, gate, up, down)
of block b uses seed ((8 b + k + 1) << 32), so the high word names the layer
and the low word is free for the re-seed counter.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import List

import numpy as np

LINEAR_NAMES = ("q", "k", "v", "o", "gate", "up", "down")


def bf16_round(a) -> np.ndarray:
    """Round float values to the nearest bfloat16 (ties to even); float32 out."""
    f = np.ascontiguousarray(np.asarray(a, dtype=np.float32))
    bits = f.view(np.uint32).astype(np.uint64)
    rounding = np.uint64(0x7FFF) + ((bits >> np.uint64(16)) & np.uint64(1))
    out = ((bits + rounding) >> np.uint64(16)) << np.uint64(16)
    return out.astype(np.uint32).view(np.float32).reshape(f.shape)


def bf16_bits(a) -> np.ndarray:
    """uint16 bit patterns of values that are already bfloat16-exact."""
    f = np.ascontiguousarray(np.asarray(a, dtype=np.float32))
    return (f.view(np.uint32) >> np.uint32(16)).astype(np.uint16)


def from_bf16_bits(b) -> np.ndarray:
    b = np.ascontiguousarray(np.asarray(b, dtype=np.uint16))
    return (b.astype(np.uint32) << np.uint32(16)).view(np.float32)


@dataclass(frozen=True)
class Linear:
    name: str
    block: int
    k: int            # index within the block (0..6)
    n: int            # input features
    m: int            # output features
    r: int            # projection rank

    @property
    def layer_id(self) -> int:
        return 8 * self.block + self.k

    @property
    def seed(self) -> int:
        return (self.layer_id + 1) << 32


@dataclass
class Workload:
    name: str
    tokens: int                  # b * l
    dtype: str                   # "f32" or "bf16"
    layers: List[Linear] = field(default_factory=list)
    lr: float = 1e-3
    beta1: float = 0.9
    beta2: float = 0.999
    eps: float = 1e-8
    alpha: float = 1.0
    description: str = ""

    def distinct_shapes(self):
        seen, out = set(), []
        for L in self.layers:
            key = (L.n, L.m, L.r)
            if key not in seen:
                seen.add(key)
                out.append(L)
        return out


def _llama_block_layers(blocks, hidden, inter, ratio):
    layers = []
    shapes = [(hidden, hidden)] * 4 + [(hidden, inter)] * 2 + [(inter, hidden)]
    for b in range(blocks):
        for k, (n, m) in enumerate(shapes):
            layers.append(Linear(LINEAR_NAMES[k], b, k, n, m, int(n * ratio)))
    return layers


def _roberta_block_layers(blocks, hidden, inter, ratio):
    names = ("q", "k", "v", "o", "ffn_in", "ffn_out")
    shapes = [(hidden, hidden)] * 4 + [(hidden, inter), (inter, hidden)]
    layers = []
    for b in range(blocks):
        for k, (n, m) in enumerate(shapes):
            layers.append(Linear(names[k], b, k, n, m, int(n * ratio)))
    return layers


def workload(name: str) -> Workload:
    """The five synthetic workloads (shapes of the paper's model families)."""
    if name == "single-f32":
        w = Workload(name, 256, "f32", [Linear("single", 0, 0, 256, 512, 32)],
                     description="single fp32 linear layer, 256 tokens, n=256, m=512, r=32, seed 1")
        # this workload uses projection seed 1 explicitly
        w.layers = [_SeedOverride("single", 0, 0, 256, 512, 32, seed_value=1)]
        return w
    if name == "llama-60m":
        return Workload(name, 128 * 256, "bf16", _llama_block_layers(8, 512, 1376, 0.25),
                        alpha=0.25,
                        description="LLaMA-60M-shaped: 8 blocks x 7 linears, 128x256 tokens, r=n/4")
    if name == "roberta-base":
        return Workload(name, 32 * 512, "bf16", _roberta_block_layers(12, 768, 3072, 0.5),
                        alpha=2.0,
                        description="RoBERTa-Base-shaped: 12 blocks x 6 linears, 32x512 tokens, r=n/2")
    if name == "llama-350m":
        return Workload(name, 256 * 256, "bf16", _llama_block_layers(24, 1024, 2736, 0.125),
                        alpha=0.25,
                        description="LLaMA-350M-shaped: 24 blocks x 7 linears, 256x256 tokens, r=n/8")
    if name in ("llama-1b-r4", "llama-1b-r8"):
        ratio = 0.25 if name.endswith("r4") else 0.125
        return Workload(name, 64 * 1024, "bf16", _llama_block_layers(24, 2048, 5461, ratio),
                        alpha=0.25,
                        description=f"LLaMA-1B-shaped: 24 blocks x 7 linears, 64x1024 tokens, r=n*{ratio}")
    raise KeyError(name)


@dataclass(frozen=True)
class _SeedOverride(Linear):
    seed_value: int = 1

    @property
    def seed(self) -> int:
        return self.seed_value


# Projections that read the same input in the model (Table 7: q, k, v read
# the normed block input, gate and up the normed attention output).
GROUPABLE = (("q", "k", "v"), ("gate", "up"))


def input_groups(wl, grouped=True):
    """Lists of layer indices that read the same input and run as one group:
    q, k, v and gate, up of one block (when grouped and the group's column
    slices start on 16-byte boundaries: every width and rank but the last a
    multiple of 8), every other layer on its own."""
    out, i, L = [], 0, wl.layers
    while i < len(L):
        g = [i]
        if grouped:
            for names in GROUPABLE:
                k = len(names)
                cand = L[i:i + k]
                if (tuple(x.name for x in cand) == names and
                        all(x.block == L[i].block and x.n == L[i].n for x in cand) and
                        all(x.m % 8 == 0 and x.r % 8 == 0 for x in cand[:-1])):
                    g = list(range(i, i + k))
                    break
        out.append(g)
        i += len(g)
    return out


WORKLOAD_NAMES = ("single-f32", "llama-60m", "roberta-base", "llama-350m",
                  "llama-1b-r4", "llama-1b-r8")


def _rng(seed):
    return np.random.Generator(np.random.PCG64(seed))


def _cast(a, dtype):
    if dtype == "bf16":
        return bf16_round(a)
    if dtype == "f32":
        return np.asarray(a, dtype=np.float32)
    raise ValueError(dtype)


def normal_bf16_blocked(rows, cols, seed, scale=1.0, block_rows=4096, threads=None, bf16=True):
    """A (rows, cols) float32 matrix of scale * N(0, 1) values, rounded to bf16
    (ties to even) unless bf16=False, for the full-size parity tests: row block
    b (block_rows rows) is drawn by PCG64(seed).jumped(b + 1) in float32, the
    blocks filled in parallel threads.  Same (rows, cols, seed, scale,
    block_rows, bf16) -> same values, whatever the thread count."""
    import concurrent.futures
    import os as _os
    out = np.empty((rows, cols), np.float32)
    nblk = (rows + block_rows - 1) // block_rows
    base = np.random.PCG64(seed)

    def fill(b):
        g = np.random.Generator(base.jumped(b + 1))
        r0, r1 = b * block_rows, min(rows, (b + 1) * block_rows)
        blk = out[r0:r1]
        g.standard_normal(out=blk, dtype=np.float32)
        if scale != 1.0:
            blk *= np.float32(scale)
        if not bf16:
            return
        bits = blk.view(np.uint32)
        lsb = (bits >> np.uint32(16)) & np.uint32(1)
        bits += np.uint32(0x7FFF)
        bits += lsb
        bits &= np.uint32(0xFFFF0000)

    workers = threads or min(16, _os.cpu_count() or 1)
    with concurrent.futures.ThreadPoolExecutor(max_workers=workers) as ex:
        list(ex.map(fill, range(nblk)))
    return out


def fwd_inputs(T, n, m, dtype, data_seed=1234):
    """x (T, n) ~ N(0,1) and W (n, m) ~ N(0, 0.02^2), rounded to dtype."""
    g = _rng(data_seed)
    x = _cast(g.standard_normal((T, n)), dtype)
    W = _cast(0.02 * g.standard_normal((n, m)), dtype)
    return x, W


def bwd_inputs(T, n, m, r, dtype, data_seed=1234):
    """dy (T, m) ~ N(0, 1e-4), a saved activation z (T, r) ~ N(0, n/r) and W."""
    g = _rng(data_seed + 7919)
    dy = _cast(0.01 * g.standard_normal((T, m)), dtype)
    z = _cast(np.sqrt(n / r) * g.standard_normal((T, r)), dtype)
    W = _cast(0.02 * g.standard_normal((n, m)), dtype)
    return dy, z, W


def step_inputs(n, m, r, w_dtype, t=1, data_seed=1234):
    """W (n, m), a compressed gradient G^ (r, m) fp32 and Adam moments.

    For t == 1 the moments are zero (Alg. 3 initialisation); for t > 1 they are
    drawn as a plausible history: M ~ N(0, 0.1^2) * |G^| scale, V = M^2 + c."""
    g = _rng(data_seed + 104729)
    W = _cast(0.02 * g.standard_normal((n, m)), w_dtype)
    G = g.standard_normal((r, m)).astype(np.float32)
    if t == 1:
        M = np.zeros((r, m), np.float32)
        V = np.zeros((r, m), np.float32)
    else:
        M = (0.1 * g.standard_normal((r, m))).astype(np.float32)
        V = (M.astype(np.float64) ** 2 + 1e-3 * g.random((r, m))).astype(np.float32)
    return W, G, M, V


def identity_matrix(n):
    return np.eye(n, dtype=np.float32)
