"""GPU parity of the projection stream (bit-exact against the oracle).

* compact_pstream (the standalone generator) against oracle.pstream.gaussian_raw;
* the Box-Muller step over every radius code and every angle code;
* the stream as it enters the fused forward GEMM (x = I gives a single product
  per output, so z is the stream itself after the fp32 scale and the output
  rounding) and the decompression kernel (W = 0, N = I), in both forward modes
  (panel in workspace, tiles regenerated in LDS).
"""
import numpy as np
import pytest

from oracle import pstream as ps
from synthetic import bf16_round

from gpu_util import dev, empty, ld_for, to_dev, to_np_f32, workspace

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
cp = pytest.importorskip("paper_2410_15352_amd")


@pytest.mark.parametrize("seed,n,r", [
    (1, 256, 32), ((5 << 32) | 3, 1024, 128), ((7 << 32), 1379, 345), (2**64 - 1, 5, 3),
    ((9 << 32) | 2, 5461, 1365),
])
def test_pstream_bitwise(seed, n, r):
    out = empty(n, r, "f32", ld=ld_for(r, "f32") + 4)
    cp.compact_pstream(seed, out)
    torch.cuda.synchronize()
    got = to_np_f32(out)
    exp = ps.gaussian_raw(seed, n, r)
    assert got.shape == exp.shape
    mism = np.count_nonzero(got.view(np.uint32) != exp.view(np.uint32))
    assert mism == 0, f"{mism} of {got.size} elements differ"


def _bm(a, b):
    at = torch.from_numpy(a.view(np.int32)).to(dev())
    bt = torch.from_numpy(b.view(np.int32)).to(dev())
    ge = torch.empty(a.size, dtype=torch.float32, device=dev())
    go = torch.empty_like(ge)
    cp.compact_pstream_boxmuller(at, bt, ge, go)
    torch.cuda.synchronize()
    return ge.cpu().numpy(), go.cpu().numpy()


def test_boxmuller_every_radius_code():
    ka = np.arange(1 << 23, dtype=np.uint32)
    a = (ka << np.uint32(9)) | (ka & np.uint32(0x1FF))          # low bits are ignored
    b = (np.uint32(0x9E3779B9) * ka).astype(np.uint32)          # assorted angles
    ge, go = _bm(a, b)
    ee, eo = ps.box_muller_f32(a, b)
    assert np.array_equal(ge.view(np.uint32), ee.view(np.uint32))
    assert np.array_equal(go.view(np.uint32), eo.view(np.uint32))


def test_boxmuller_every_angle_code():
    kb = np.arange(1 << 24, dtype=np.uint32)
    b = (kb << np.uint32(8)) | (kb & np.uint32(0xFF))
    a = (np.uint32(0x85EBCA6B) * kb).astype(np.uint32)
    ge, go = _bm(a, b)
    ee, eo = ps.box_muller_f32(a, b)
    assert np.array_equal(ge.view(np.uint32), ee.view(np.uint32))
    assert np.array_equal(go.view(np.uint32), eo.view(np.uint32))


@pytest.mark.parametrize("dtype,use_ws", [("bf16", True), ("bf16", False), ("f32", False)])  # no fp32 workspace mode
@pytest.mark.parametrize("n,r,seed", [(256, 32, 1), (200, 44, (3 << 32) | 1), (1024, 128, 77)])
def test_in_gemm_stream_x_identity(dtype, use_ws, n, r, seed):
    m = 8
    x = to_dev(np.eye(n, dtype=np.float32), dtype, ld=ld_for(n, dtype))
    W = to_dev(np.zeros((n, m), np.float32), dtype, ld=ld_for(m, dtype))
    y = empty(n, m, dtype, ld=ld_for(m, dtype))
    z = empty(n, r, dtype, ld=ld_for(r, dtype), fill=7.0)
    ws = workspace(cp.fwd_workspace_bytes(n, m, r, cp.BF16 if dtype == "bf16" else cp.F32)) if use_ws else None
    cp.compact_fwd(x, W, y, z, seed, ws=ws)
    torch.cuda.synchronize()
    got = to_np_f32(z)
    G = ps.gaussian_raw(seed, n, r)
    s = np.float32(1.0 / np.sqrt(np.float64(r)))
    # fp32: z = (x G) s;  bf16: P = G s is formed in fp32 and rounded to bf16
    # once, and x = I passes it through the MFMA unchanged
    exp = G * s if dtype == "f32" else bf16_round(G * s)
    assert np.array_equal(got.view(np.uint32), exp.astype(np.float32).view(np.uint32))


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("n,r,seed", [(256, 32, 1), (300, 64, (4 << 32) | 9), (2736, 342, 5)])
def test_decompression_stream_w_zero(dtype, n, r, seed):
    # G = I (m = r) makes Adam's N exactly I at t = 1, so with lr = alpha = 1
    # the update is -fp32(1/sqrt r) * P-stream, rounded once in fp32.
    m = r
    W = to_dev(np.zeros((n, m), np.float32), "f32", ld=ld_for(m, "f32"))
    G = torch.eye(r, dtype=torch.float32, device=dev())
    M = torch.zeros_like(G)
    V = torch.zeros_like(G)
    ws = workspace(cp.step_workspace_bytes(n, m, r, cp.BF16 if dtype == "bf16" else cp.F32))
    cp.compact_step(W, G, M, V, seed, 1, lr=1.0, alpha=1.0, dtype=dtype, ws=ws)
    torch.cuda.synchronize()
    got = -to_np_f32(W)
    Gs = ps.gaussian_raw(seed, n, r)
    s = np.float32(1.0 / np.sqrt(np.float64(r)))
    src = bf16_round(Gs) if dtype == "bf16" else Gs
    exp = (src * s).astype(np.float32)
    assert np.array_equal(got.view(np.uint32), exp.view(np.uint32))
