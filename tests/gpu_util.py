"""Helpers for the GPU tests: host <-> device transfers of bf16 / fp32 data."""
from __future__ import annotations

import numpy as np

from synthetic import bf16_bits, from_bf16_bits


def dev():
    import torch
    return torch.device("cuda:0")


def to_dev(a, dtype, ld=None):
    """numpy (rows, cols) -> device tensor of `dtype` ("bf16"|"f32"), optionally
    as a view into a wider buffer with leading dimension ld."""
    import torch
    a = np.asarray(a, dtype=np.float32)
    rows, cols = a.shape
    ld = cols if ld is None else ld
    if dtype == "bf16":
        buf = np.zeros((rows, ld), dtype=np.uint16)
        buf[:, :cols] = bf16_bits(a)
        t = torch.from_numpy(buf.view(np.int16)).view(torch.bfloat16).to(dev())
    else:
        buf = np.zeros((rows, ld), dtype=np.float32)
        buf[:, :cols] = a
        t = torch.from_numpy(buf).to(dev())
    return t[:, :cols]


def empty(rows, cols, dtype, ld=None, fill=None):
    import torch
    ld = cols if ld is None else ld
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    t = torch.empty(rows, ld, dtype=tdt, device=dev())
    if fill is not None:
        t.fill_(fill)
    return t[:, :cols]


def to_np(t):
    """Device tensor (bf16 or fp32) -> numpy float64 (exact values)."""
    import torch
    if t.dtype == torch.bfloat16:
        u = t.contiguous().view(torch.int16).cpu().numpy().view(np.uint16)
        return from_bf16_bits(u).astype(np.float64)
    return t.detach().cpu().numpy().astype(np.float64)


def to_np_f32(t):
    import torch
    if t.dtype == torch.bfloat16:
        u = t.contiguous().view(torch.int16).cpu().numpy().view(np.uint16)
        return from_bf16_bits(u)
    return t.detach().cpu().numpy().astype(np.float32)


def workspace(nbytes):
    import torch
    return torch.zeros(max(int(nbytes), 1), dtype=torch.uint8, device=dev())


def ld_for(cols, dtype):
    q = 8 if dtype == "bf16" else 4
    return (cols + q - 1) // q * q


# Elementwise bounds for the bf16 GEMM outputs.  A dot product of K terms
# accumulated in fp32 is off by at most lam sqrt(K) u sum|terms| (u = 2^-24)
# with probability >= 1 - 2 exp(-lam^2 / 2) per element (the probabilistic
# rounding-error bound of Higham and Mary, 2019); lam = 8 makes a false alarm
# over 10^9 elements about 10^-5 likely.  A bf16 output adds one rounding to
# nearest even, at most 2^-8 of the value; an operand rounded to bf16 (P in
# the forward) adds 2^-8 of its share of sum|terms|.
U32 = 2.0 ** -24
BF16_U = 2.0 ** -8
LAM = 8.0


def acc_bound(K):
    return LAM * np.sqrt(float(K)) * U32


def assert_elementwise(gpu, ref, absprod, K, bf16_out=True, operand_rel=0.0, what=""):
    """|gpu - ref| <= out_round * |ref| + (operand_rel + acc(K)) * (1 + out_round) * absprod
    + a floor below the smallest normal bf16, for every element; absprod is
    the exact sum of |terms| of each element (|x| |W| etc.)."""
    gpu = np.asarray(gpu, np.float64)
    ref = np.asarray(ref, np.float64)
    out_r = BF16_U if bf16_out else 0.0
    bound = out_r * np.abs(ref) + (operand_rel + acc_bound(K)) * (1.0 + out_r) * absprod + 2.0 ** -120
    err = np.abs(gpu - ref)
    bad = ~(err <= bound)  # NaN counts as a failure
    if bad.any():
        idx = np.argwhere(bad)
        i = tuple(idx[0])
        raise AssertionError(f"{what}: {int(bad.sum())} of {bad.size} elements outside the bound; first at {i}: "
                             f"gpu {gpu[i]!r} ref {ref[i]!r} bound {bound[i]!r}")
