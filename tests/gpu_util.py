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
