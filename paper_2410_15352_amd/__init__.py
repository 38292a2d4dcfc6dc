"""CompAct compressed linear layer on AMD MI355X (gfx950).

A thin Python binding over the C ABI of ``libcompact.so`` (include/compact.h):
the functions below only translate torch tensors into device pointers, leading
dimensions and the current HIP stream, call the library, and raise on a
non-zero status.  All arithmetic runs in the library's HIP kernels; there is
no fallback path.

    compact_fwd   Alg. 1: y = x W, z = x P          (CompAct, §3.2)
    compact_bwd   Alg. 2: G^ = z^T dy, dx = dy W^T
    compact_step  Alg. 3: Adam on r x m moments, W -= lr alpha P N
    compact_pstream      the seeded projection stream (unscaled normals)
    compact_next_seed    the Alg. 3 seed schedule
"""
from __future__ import annotations

import ctypes

from . import _lib

F32, BF16 = 0, 1
PROJ = {"gaussian": 0, "identity": 1, "sparse-jl": 2}
SPARSE_JL_DEFAULT_S = 8
PROJ_GATHER = 1 << 16  # COMPACT_PROJ_GATHER: the forward's z of a sparse projection by gather-add


def proj_code(proj):
    """The ABI's compact_proj code of a projection: "gaussian", "identity",
    "sparse-jl" (s = 8 draws per row), "sparse-jl:<s>", either sparse form
    with the suffix ":gather" (COMPACT_PROJ_GATHER), or an int code."""
    if isinstance(proj, int):
        return proj
    flags = 0
    if proj.startswith("sparse-jl") and proj.endswith(":gather"):
        proj, flags = proj[: -len(":gather")], PROJ_GATHER
    if proj.startswith("sparse-jl:"):
        s_ = int(proj.split(":", 1)[1])
        if not 1 <= s_ <= 64:
            raise ValueError("sparse-jl draws per row must be in [1, 64]")
        return PROJ["sparse-jl"] | (s_ << 8) | flags
    return PROJ[proj] | flags


__all__ = ["compact_fwd", "compact_fwd_group", "compact_projection", "proj_code", "fwd_group_workspace_bytes", "compact_bwd", "compact_bwd_noalloc", "compact_step", "compact_pstream", "compact_next_seed",
           "compact_pstream_boxmuller", "compact_step_batched", "step_batched_workspace_bytes",
           "LayerBatch", "prepare_layers",
           "fwd_workspace_bytes", "bwd_workspace_bytes", "step_workspace_bytes",
           "saved_activation_elems", "CompactError", "library", "F32", "BF16"]


class CompactError(RuntimeError):
    def __init__(self, fn, status):
        lib = _lib.load()
        msg = lib.compact_status_string(status).decode()
        detail = lib.compact_last_error().decode()
        super().__init__(f"{fn}: {msg} ({status}): {detail}")
        self.status = status


def library():
    return _lib.load()


def _dtype_code(t):
    import torch
    if t.dtype == torch.bfloat16:
        return BF16
    if t.dtype == torch.float32:
        return F32
    raise TypeError(f"unsupported dtype {t.dtype}")


def _ptr(t):
    return None if t is None else t.data_ptr()


def _ld(t):
    if t is None:
        return 0
    if t.dim() != 2 or t.stride(1) != 1:
        raise ValueError("expected a 2-D tensor with unit column stride")
    return t.stride(0)


def _stream(stream, ref):
    import torch
    if stream is not None:
        return stream
    return torch.cuda.current_stream(ref.device).cuda_stream


def _ws(ws):
    if ws is None:
        return None, 0
    return ws.data_ptr(), ws.numel() * ws.element_size()


def _check(fn, status):
    if status != 0:
        raise CompactError(fn, status)


def fwd_workspace_bytes(n, m, r, dtype=BF16):
    return int(_lib.load().compact_fwd_workspace_bytes(n, m, r, dtype))


def bwd_workspace_bytes(tokens, n, m, r, dtype=BF16):
    return int(_lib.load().compact_bwd_workspace_bytes(tokens, n, m, r, dtype))


def step_workspace_bytes(n, m, r, dtype=BF16):
    return int(_lib.load().compact_step_workspace_bytes(n, m, r, dtype))


def saved_activation_elems(tokens, n, r):
    return int(_lib.load().compact_saved_activation_elems(tokens, n, r))


def compact_fwd(x, W, y, z, seed, proj="gaussian", ws=None, stream=None):
    """y = x W and z = x P (Alg. 1).  x (T, n), W (n, m), y (T, m), z (T, r)."""
    lib = _lib.load()
    T, n = x.shape
    m = W.shape[1]
    r = z.shape[1]
    wp, wb = _ws(ws)
    st = lib.compact_fwd(_ptr(x), _ld(x), _ptr(W), _ld(W), _ptr(y), _ld(y), _ptr(z), _ld(z),
                         T, n, m, r, int(seed) & (2**64 - 1), proj_code(proj), _dtype_code(x),
                         wp, wb, _stream(stream, x))
    _check("compact_fwd", st)


def _group_arrays(ms, rs, seeds=None):
    count = len(ms)
    if len(rs) != count or (seeds is not None and len(seeds) != count):
        raise ValueError("one m, r (and seed) per projection")
    m_arr = (ctypes.c_int64 * count)(*[int(v) for v in ms])
    r_arr = (ctypes.c_int64 * count)(*[int(v) for v in rs])
    s_arr = None if seeds is None else (ctypes.c_uint64 * count)(*[int(v) & (2**64 - 1) for v in seeds])
    return count, m_arr, r_arr, s_arr


def fwd_group_workspace_bytes(n, ms, rs, dtype=BF16):
    count, m_arr, r_arr, _ = _group_arrays(ms, rs)
    return int(_lib.load().compact_fwd_group_workspace_bytes(int(n), count, m_arr, r_arr, dtype))


def compact_fwd_group(x, W, y, z, ms, rs, seeds, proj="gaussian", ws=None, stream=None):
    """Alg. 1 for projections that share the input x: W = [W_0 | W_1 | ...]
    (n, sum m), y (T, sum m), z (T, sum r); projection j uses columns
    sum(ms[:j]) .. of W and y, columns sum(rs[:j]) .. of z and seed seeds[j].
    Bitwise equal to compact_fwd on each column slice."""
    lib = _lib.load()
    T, n = x.shape
    count, m_arr, r_arr, s_arr = _group_arrays(ms, rs, seeds)
    wp, wb = _ws(ws)
    st = lib.compact_fwd_group(_ptr(x), _ld(x), _ptr(W), _ld(W), _ptr(y), _ld(y), _ptr(z), _ld(z), T, n, count,
                               m_arr, r_arr, s_arr, proj_code(proj), _dtype_code(x), wp, wb, _stream(stream, x))
    _check("compact_fwd_group", st)


def compact_bwd(dy, W, z, dx, G, ws=None, stream=None):
    """G^ = z^T dy (fp32, r x m) and dx = dy W^T (Alg. 2).  dx or G may be None."""
    lib = _lib.load()
    T, m = dy.shape
    r = z.shape[1] if z is not None else (G.shape[0] if G is not None else 1)
    n = W.shape[0] if W is not None else (dx.shape[1] if dx is not None else r)
    if G is not None and (not G.is_contiguous() or tuple(G.shape) != (r, m)):
        raise ValueError("G must be a contiguous (r, m) fp32 tensor")
    wp, wb = _ws(ws)
    st = lib.compact_bwd(_ptr(dy), _ld(dy), _ptr(W), _ld(W), _ptr(z), _ld(z), _ptr(dx), _ld(dx),
                         _ptr(G), T, n, m, r, _dtype_code(dy), wp, wb, _stream(stream, dy))
    _check("compact_bwd", st)


NOALLOC_SCRATCH_BYTES = (64 << 20) + 256


def compact_bwd_noalloc(dy, W, z, dx, G, stream=None):
    """compact_bwd without a workspace: the library's own per-GPU scratch
    (calls that overlap on one GPU race)."""
    lib = _lib.load()
    T, m = dy.shape
    r = z.shape[1] if z is not None else (G.shape[0] if G is not None else 1)
    n = W.shape[0] if W is not None else (dx.shape[1] if dx is not None else r)
    if G is not None and (not G.is_contiguous() or tuple(G.shape) != (r, m)):
        raise ValueError("G must be a contiguous (r, m) fp32 tensor")
    st = lib.compact_bwd_noalloc(_ptr(dy), _ld(dy), _ptr(W), _ld(W), _ptr(z), _ld(z), _ptr(dx), _ld(dx),
                                 _ptr(G), T, n, m, r, _dtype_code(dy), _stream(stream, dy))
    _check("compact_bwd_noalloc", st)


def bwd_group_workspace_bytes(tokens, n, ms, rs, dtype=BF16):
    count, m_arr, r_arr, _ = _group_arrays(ms, rs)
    return int(_lib.load().compact_bwd_group_workspace_bytes(int(tokens), int(n), count, m_arr, r_arr, dtype))


def compact_bwd_group(dy, W, z, dx, Gs, ms, rs, ws=None, stream=None, accumulate=False):
    """Alg. 2 for the projections of an input group: dx = dy W^T over the
    concatenated weight W = [W_0 | W_1 | ...] (the sum over the projections)
    and G^_j = z_j^T dy_j for column slices dy_j (sum(ms[:j]) ..) and z_j
    (sum(rs[:j]) ..), one split-K launch for all of them.  dx or Gs may be
    None; Gs is a list of contiguous (r_j, m_j) fp32 tensors, overwritten, or
    with accumulate=True increased by G^_j (gradient accumulation)."""
    import ctypes
    lib = _lib.load()
    T = dy.shape[0]
    count, m_arr, r_arr, _ = _group_arrays(ms, rs)
    n = W.shape[0] if W is not None else (dx.shape[1] if dx is not None else max(int(v) for v in rs))
    g_arr = None
    if Gs is not None:
        if len(Gs) != count:
            raise ValueError("one G per projection")
        for G, m, r in zip(Gs, ms, rs):
            if not G.is_contiguous() or tuple(G.shape) != (r, m):
                raise ValueError("every G must be a contiguous (r, m) fp32 tensor")
        g_arr = (ctypes.c_void_p * count)(*[G.data_ptr() for G in Gs])
    wp, wb = _ws(ws)
    st = lib.compact_bwd_group(_ptr(dy), _ld(dy), _ptr(W), _ld(W), _ptr(z), _ld(z), _ptr(dx), _ld(dx), g_arr, T,
                               n, count, m_arr, r_arr, _dtype_code(dy), 1 if accumulate else 0, wp, wb,
                               _stream(stream, dy))
    _check("compact_bwd_group", st)


def compact_step(W, G, M, V, seed, t, lr, beta1=0.9, beta2=0.999, eps=1e-8, alpha=1.0,
                 proj="gaussian", dtype=None, ws=None, stream=None):
    """Adam on the compressed gradient and W -= lr alpha P N (Alg. 3), in place."""
    lib = _lib.load()
    n, m = W.shape
    r = G.shape[0]
    for name, t_ in (("G", G), ("M", M), ("V", V)):
        if not t_.is_contiguous() or tuple(t_.shape) != (r, m):
            raise ValueError(f"{name} must be a contiguous (r, m) fp32 tensor")
    w_code = _dtype_code(W)
    d_code = w_code if dtype is None else {"bf16": BF16, "f32": F32}[dtype]
    wp, wb = _ws(ws)
    st = lib.compact_step(_ptr(W), _ld(W), _ptr(G), _ptr(M), _ptr(V), n, m, r,
                          int(seed) & (2**64 - 1), int(t), float(lr), float(beta1), float(beta2),
                          float(eps), float(alpha), proj_code(proj), d_code, w_code, wp, wb,
                          _stream(stream, W))
    _check("compact_step", st)


def _layer_array(layers):
    arr = (_lib.CompactLayer * len(layers))()
    for i, L in enumerate(layers):
        W, G, M, V = L["W"], L["G"], L["M"], L["V"]
        r, m = G.shape
        for name, t_ in (("G", G), ("M", M), ("V", V)):
            if not t_.is_contiguous() or tuple(t_.shape) != (r, m):
                raise ValueError(f"layer {i}: {name} must be a contiguous (r, m) fp32 tensor")
        arr[i] = _lib.CompactLayer(W.data_ptr(), _ld(W), G.data_ptr(), M.data_ptr(), V.data_ptr(),
                                   W.shape[0], m, r, int(L["seed"]) & (2**64 - 1),
                                   float(L.get("alpha", 1.0)))
    return arr


class LayerBatch:
    """The compact_layer array of compact_step_batched, marshalled once.  The
    tensors must stay alive and in place; seeds change with set_seeds (the
    seed schedule of Alg. 3) without rebuilding the array."""

    def __init__(self, layers):
        if not layers:
            raise ValueError("empty layer list")
        self.arr = _layer_array(layers)
        self.count = len(layers)
        self.w0 = layers[0]["W"]
        self._keep = [dict(L) for L in layers]

    def set_seeds(self, seeds):
        if len(seeds) != self.count:
            raise ValueError("one seed per layer")
        for i, s_ in enumerate(seeds):
            self.arr[i].seed = int(s_) & (2**64 - 1)


def prepare_layers(layers):
    return LayerBatch(layers)


def _as_batch(layers):
    return layers if isinstance(layers, LayerBatch) else LayerBatch(layers)


def step_batched_workspace_bytes(layers, dtype=BF16):
    b = _as_batch(layers)
    return int(_lib.load().compact_step_batched_workspace_bytes(b.arr, b.count, dtype))


def compact_step_batched(layers, t, lr, beta1=0.9, beta2=0.999, eps=1e-8, proj="gaussian",
                         ws=None, stream=None):
    """Alg. 3 for many layers in a few launches.  layers: a LayerBatch, or a
    list of dicts with keys W, G, M, V, seed and optional alpha (bf16
    compute; W bf16 or fp32)."""
    lib = _lib.load()
    if not isinstance(layers, LayerBatch) and not layers:
        return
    b = _as_batch(layers)
    w_code = _dtype_code(b.w0)
    wp, wb = _ws(ws)
    st = lib.compact_step_batched(b.arr, b.count, int(t), float(lr), float(beta1), float(beta2),
                                  float(eps), proj_code(proj), BF16, w_code, wp, wb, _stream(stream, b.w0))
    _check("compact_step_batched", st)


def compact_pstream(seed, out, stream=None):
    """Fill out (n, r) fp32 with the unscaled stream G(seed, i, j)."""
    lib = _lib.load()
    n, r = out.shape
    st = lib.compact_pstream(int(seed) & (2**64 - 1), n, r, _ptr(out), _ld(out),
                             _stream(stream, out))
    _check("compact_pstream", st)


def compact_projection(seed, out, proj="gaussian", stream=None):
    """Fill out (n, r) fp32 with the unscaled stream of a projection: G, the
    identity, or the sparse JL integers S."""
    lib = _lib.load()
    n, r = out.shape
    st = lib.compact_projection(int(seed) & (2**64 - 1), n, r, proj_code(proj), _ptr(out), _ld(out),
                                _stream(stream, out))
    _check("compact_projection", st)


def compact_pstream_boxmuller(a, b, g_even, g_odd, stream=None):
    """Box-Muller step of the stream on word pairs (int32 tensors viewed as uint32)."""
    lib = _lib.load()
    st = lib.compact_pstream_boxmuller(_ptr(a), _ptr(b), _ptr(g_even), _ptr(g_odd), a.numel(),
                                       _stream(stream, a))
    _check("compact_pstream_boxmuller", st)


def compact_next_seed(seed, t, T):
    return int(_lib.load().compact_next_seed(int(seed) & (2**64 - 1), int(t), int(T)))
