"""compact_bwd_noalloc (the backward for callers that cannot allocate) against
compact_bwd with a caller workspace, through the C ABI: dL/dx and G^ bitwise
equal, on two calls in a row, the second with a smaller input (the scratch
keeps the first call's partial sums, which must not reach the second's
result); then the second call's results against the oracle."""
import numpy as np
import pytest

from oracle import compact as oc
from synthetic import bwd_inputs

from gpu_util import dev, empty, ld_for, to_dev, to_np, workspace

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
cp = pytest.importorskip("paper_2410_15352_amd")


def _call(lib, fn, dy, W, z, dx, G, T, n, m, r, ws=None):
    stream = torch.cuda.current_stream().cuda_stream
    args = [dy.data_ptr(), dy.stride(0), W.data_ptr(), W.stride(0), z.data_ptr(), z.stride(0), dx.data_ptr(),
            dx.stride(0), G.data_ptr(), T, n, m, r, cp.BF16]
    if ws is not None:
        args += [ws.data_ptr(), ws.numel()]
    st = getattr(lib, fn)(*args, stream)
    assert st == 0, (fn, st, lib.compact_last_error().decode())


def test_noalloc_matches_workspace_path_twice():
    lib = cp.library()
    # the LLaMA-350M gate projection, then a smaller ragged one
    for T, n, m, r in ((8192, 1024, 2736, 128), (1000, 512, 1376, 40)):
        dy, z, W = bwd_inputs(T, n, m, r, "bf16", data_seed=T + m)
        dyd, zd, Wd = to_dev(dy, "bf16", ld_for(m, "bf16")), to_dev(z, "bf16", ld_for(r, "bf16")), \
            to_dev(W, "bf16", ld_for(m, "bf16"))
        outs = []
        for fn in ("compact_bwd", "compact_bwd_noalloc"):
            dx = empty(T, n, "bf16", ld_for(n, "bf16"), fill=float("nan"))
            G = torch.full((r, m), float("nan"), dtype=torch.float32, device=dev())
            ws = workspace(cp.NOALLOC_SCRATCH_BYTES) if fn == "compact_bwd" else None
            _call(lib, fn, dyd, Wd, zd, dx, G, T, n, m, r, ws)
            outs.append((dx, G))
        torch.cuda.synchronize()
        (dx0, G0), (dx1, G1) = outs
        assert torch.equal(dx0.view(torch.int16), dx1.view(torch.int16))
        assert torch.equal(G0.view(torch.int32), G1.view(torch.int32))
    dx_ref, G_ref = oc.ref_bwd(dy, z, W)
    assert oc.rel_fro(to_np(dx1), dx_ref) <= 2e-2
    assert oc.rel_fro(G1.cpu().numpy(), G_ref) <= 2e-2


def test_noalloc_largest_workload_layer():
    # a LLaMA-1B q/k/v/o projection at r = n/4: the largest need of the bf16
    # workloads, every byte of the scratch (G^ partial sums up to its end)
    lib = cp.library()
    T, n, m, r = 1000, 2048, 2048, 512
    assert cp.bwd_workspace_bytes(T, n, m, r) == cp.NOALLOC_SCRATCH_BYTES
    dy, z, W = bwd_inputs(T, n, m, r, "bf16", data_seed=17)
    dyd, zd, Wd = to_dev(dy, "bf16", m), to_dev(z, "bf16", r), to_dev(W, "bf16", m)
    outs = []
    for fn in ("compact_bwd", "compact_bwd_noalloc"):
        dx = empty(T, n, "bf16", n, fill=float("nan"))
        G = torch.full((r, m), float("nan"), dtype=torch.float32, device=dev())
        ws = workspace(cp.NOALLOC_SCRATCH_BYTES) if fn == "compact_bwd" else None
        _call(lib, fn, dyd, Wd, zd, dx, G, T, n, m, r, ws)
        outs.append((dx, G))
    torch.cuda.synchronize()
    (dx0, G0), (dx1, G1) = outs
    assert torch.equal(dx0.view(torch.int16), dx1.view(torch.int16))
    assert torch.equal(G0.view(torch.int32), G1.view(torch.int32))
    dx_ref, G_ref = oc.ref_bwd(dy, z, W)
    assert oc.rel_fro(to_np(dx1), dx_ref) <= 2e-2
    assert oc.rel_fro(G1.cpu().numpy(), G_ref) <= 2e-2


def test_noalloc_rejects_oversized_requests():
    # G^ of r = 2048, m = 16384 needs more partial sums than the scratch holds:
    # a clear error and nothing launched (the pointers are never touched)
    lib = cp.library()
    T, n, m, r = 4096, 2048, 16384, 2048
    need = cp.bwd_workspace_bytes(T, n, m, r)
    assert need > cp.NOALLOC_SCRATCH_BYTES
    dy = torch.empty(8, dtype=torch.bfloat16, device=dev())
    st = lib.compact_bwd_noalloc(dy.data_ptr(), m, dy.data_ptr(), m, dy.data_ptr(), r, dy.data_ptr(), n,
                                 dy.data_ptr(), T, n, m, r, cp.BF16, None)
    assert st == -3  # COMPACT_EUNSUPPORTED
    assert "scratch" in lib.compact_last_error().decode()
    torch.cuda.synchronize()
