"""CPU checks of the C ABI: the library loads, exports every function declared
in include/compact.h, and its host-only logic (argument validation, workspace
sizing, seed schedule, status strings) behaves as documented.  No call here
reaches a kernel launch: every invalid call returns before any HIP call."""
import ctypes
import os
import re

import pytest

from oracle import compact as oc

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "compact.h")


def _declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    names = re.findall(r"\b(compact_[a-z0-9_]+)\s*\(", text)
    return sorted(set(names))


@pytest.fixture(scope="module")
def lib():
    from paper_2410_15352_amd import _lib
    if not os.path.exists(_lib.LIB_PATH):
        pytest.skip("libcompact.so not built (run __graft_entry__.build())")
    return _lib.load()


def test_header_declares_the_boundary():
    names = _declared_functions()
    for required in ("compact_fwd", "compact_bwd", "compact_step", "compact_pstream",
                     "compact_next_seed", "compact_fwd_workspace_bytes",
                     "compact_bwd_workspace_bytes", "compact_step_workspace_bytes"):
        assert required in names


def test_library_exports_every_declared_symbol(lib):
    from paper_2410_15352_amd import _lib
    for name in _declared_functions():
        assert hasattr(lib, name), name
        assert name in _lib.SIGNATURES, f"binding lacks a signature for {name}"


def test_missing_library_fails_loudly(tmp_path):
    from paper_2410_15352_amd import _lib
    saved = _lib._lib
    _lib._lib = None
    try:
        with pytest.raises(_lib.CompactLibraryMissing):
            _lib.load(str(tmp_path / "absent.so"))
    finally:
        _lib._lib = saved


def test_seed_schedule_matches_oracle(lib):
    for seed in (0, 7 << 32, 2**64 - 1):
        for T in (0, 1, 3, 50):
            for t in range(1, 12):
                assert lib.compact_next_seed(seed, t, T) == oc.next_seed(seed, t, T)


def test_saved_activation_elems(lib):
    me = oc.memory_elements(256, 256, 1024, 1024, 128)
    assert lib.compact_saved_activation_elems(65536, 1024, 128) == me["compact"]["activations"]


def test_status_strings(lib):
    for code in (0, -1, -2, -3, -4, -5):
        assert lib.compact_status_string(code)
    assert lib.compact_status_string(0) == b"ok"
    assert lib.compact_version() >= 100


def test_workspace_sizes(lib):
    # [W^T; P^T]: round_up(m, 256) + r rows of round_up(n, 64) bf16 values
    assert lib.compact_fwd_workspace_bytes(1024, 1000, 128, 1) >= (1024 + 128) * 1024 * 2
    assert lib.compact_fwd_workspace_bytes(1000, 2736, 128, 1) >= (2816 + 128) * 1024 * 2
    assert lib.compact_fwd_workspace_bytes(1024, 1024, 128, 0) == 0
    assert lib.compact_bwd_workspace_bytes(65536, 1024, 1024, 128, 1) > 128 * 1024 * 4
    assert lib.compact_step_workspace_bytes(1024, 1024, 128, 1) >= 128 * 1024 * 2
    assert lib.compact_step_workspace_bytes(256, 512, 32, 0) >= 32 * 512 * 4



def _header_define(name):
    m = re.search(r"#define\s+" + name + r"\s+(.+)", open(HEADER).read())
    return eval(re.sub(r"(\d+)u\b", r"\1", m.group(1)), {})


@pytest.mark.parametrize("tokens", [1, 1000, 4096, 8192, 32768, 65536, 1 << 20])
def test_noalloc_scratch_covers_every_workload_layer(lib, tokens):
    # compact_bwd_noalloc's scratch holds the backward of every layer of the
    # bf16 workloads (LLaMA-60M/350M/1B, RoBERTa-Base) at any token count
    import paper_2410_15352_amd as cp
    from synthetic import WORKLOAD_NAMES, workload
    size = _header_define("COMPACT_NOALLOC_SCRATCH_BYTES")
    assert size == cp.NOALLOC_SCRATCH_BYTES and size % 256 == 0
    most = 0
    for name in WORKLOAD_NAMES:
        wl = workload(name)
        if wl.dtype != "bf16":
            continue
        for L in wl.layers:
            most = max(most, lib.compact_bwd_workspace_bytes(tokens, L.n, L.m, L.r, 1))
    assert 0 < most <= size

FAKE = 0x100000  # an aligned non-NULL address; never dereferenced (validation fails first)


@pytest.mark.parametrize("kw,status", [
    (dict(r=0), -1), (dict(r=2000), -1), (dict(n=0), -1), (dict(tokens=-1), -1),
    (dict(proj=1), -1),             # identity needs r == n
    (dict(proj=7), -1), (dict(dtype=5), -1),
    (dict(proj=2 | (65 << 8)), -1),  # sparse JL: at most 64 draws per row
    (dict(proj=4 << 8), -1),         # draws given to the Gaussian
    (dict(proj=-1), -1),
    (dict(proj=2 | (64 << 8), ws=FAKE, ws_bytes=16), -4),  # a valid sparse code reaches the workspace check
    (dict(proj=0 | (1 << 16)), -1),          # the gather flag on the Gaussian
    (dict(proj=2 | (1 << 17)), -1),          # an unknown flag bit
    (dict(proj=2 | (17 << 8) | (1 << 16)), -3),  # gather-add: at most 16 draws per row
    (dict(proj=2 | (16 << 8) | (1 << 16), ws=FAKE, ws_bytes=16), -4),  # a valid gather code
    (dict(proj=2 | (1 << 16), n=70000, r=65535), -3),  # gather-add: r below 65535
    (dict(ldx=1000), -1),           # ld < n
    (dict(ldx=1028), -2),           # bf16 ld not a multiple of 8
    (dict(x=FAKE + 2), -2),         # misaligned pointer
    (dict(x=None), -1),
    (dict(ws=FAKE, ws_bytes=16), -4),
])
def test_fwd_validation(lib, kw, status):
    a = dict(x=FAKE, ldx=1024, W=FAKE, ldw=1024, y=FAKE, ldy=1024, z=FAKE, ldz=128, tokens=64,
             n=1024, m=1024, r=128, seed=1, proj=0, dtype=1, ws=None, ws_bytes=0, stream=None)
    a.update(kw)
    st = lib.compact_fwd(a["x"], a["ldx"], a["W"], a["ldw"], a["y"], a["ldy"], a["z"], a["ldz"],
                         a["tokens"], a["n"], a["m"], a["r"], a["seed"], a["proj"], a["dtype"],
                         a["ws"], a["ws_bytes"], a["stream"])
    assert st == status
    assert lib.compact_last_error()


def _i64s(*v):
    return (ctypes.c_int64 * len(v))(*v)


def test_fwd_group_workspace_size(lib):
    # [W_0^T; W_1^T; W_2^T; pad to 256; P_0^T; P_1^T; P_2^T]: one stacked operand
    ms, rs = _i64s(1024, 1024, 1024), _i64s(128, 128, 128)
    assert lib.compact_fwd_group_workspace_bytes(1024, 3, ms, rs, 1) == \
        lib.compact_fwd_workspace_bytes(1024, 3072, 384, 1)
    ms2, rs2 = _i64s(2736, 2736), _i64s(128, 128)
    assert lib.compact_fwd_group_workspace_bytes(1024, 2, ms2, rs2, 1) == \
        lib.compact_fwd_workspace_bytes(1024, 5472, 256, 1)
    assert lib.compact_fwd_group_workspace_bytes(1024, 3, ms, rs, 0) == 0
    assert lib.compact_fwd_group_workspace_bytes(1024, 0, ms, rs, 1) == 0
    assert lib.compact_fwd_group_workspace_bytes(1024, 9, ms, rs, 1) == 0


@pytest.mark.parametrize("kw,status", [
    (dict(count=0), -1), (dict(count=9), -1),
    (dict(m=None), -1), (dict(r=None), -1), (dict(seeds=None), -1),
    (dict(m=(1020, 1024, 1024)), -2),   # a slice that is not 16-byte aligned
    (dict(r=(128, 124, 128)), -2),
    (dict(r=(128, 128, 2000)), -1),     # r > n
    (dict(m=(1024, 0, 1024)), -1),
    (dict(ldw=3000), -1),               # ld < sum of m
    (dict(ldz=376), -1),                # ld < sum of r
    (dict(proj=1), -1),                 # identity needs r == n
    (dict(ws=FAKE, ws_bytes=16), -4),
])
def test_fwd_group_validation(lib, kw, status):
    a = dict(x=FAKE, ldx=1024, W=FAKE, ldw=3072, y=FAKE, ldy=3072, z=FAKE, ldz=384, tokens=64, n=1024,
             count=3, m=(1024, 1024, 1024), r=(128, 128, 128), seeds=(1, 2, 3), proj=0, dtype=1, ws=None,
             ws_bytes=0, stream=None)
    a.update(kw)
    arr = lambda v, t: None if v is None else (t * len(v))(*v)
    st = lib.compact_fwd_group(a["x"], a["ldx"], a["W"], a["ldw"], a["y"], a["ldy"], a["z"], a["ldz"],
                               a["tokens"], a["n"], a["count"], arr(a["m"], ctypes.c_int64),
                               arr(a["r"], ctypes.c_int64), arr(a["seeds"], ctypes.c_uint64), a["proj"],
                               a["dtype"], a["ws"], a["ws_bytes"], a["stream"])
    assert st == status
    assert lib.compact_last_error()


@pytest.mark.parametrize("kw,status", [
    (dict(dx=None, G=None), -1), (dict(ws=None), -4), (dict(ws_bytes=8), -4),
    (dict(lddy=1020), -1), (dict(G=FAKE + 4), -2), (dict(r=1025), -1),
])
def test_bwd_validation(lib, kw, status):
    a = dict(dy=FAKE, lddy=1024, W=FAKE, ldw=1024, z=FAKE, ldz=128, dx=FAKE, lddx=1024, G=FAKE,
             tokens=4096, n=1024, m=1024, r=128, dtype=1, ws=FAKE, ws_bytes=1 << 40, stream=None)
    a.update(kw)
    st = lib.compact_bwd(a["dy"], a["lddy"], a["W"], a["ldw"], a["z"], a["ldz"], a["dx"], a["lddx"],
                         a["G"], a["tokens"], a["n"], a["m"], a["r"], a["dtype"], a["ws"],
                         a["ws_bytes"], a["stream"])
    assert st == status


def test_bwd_group_workspace_size(lib):
    # one split-K plan for all projections; at least what each slice needs alone
    ms, rs = _i64s(1024, 1024, 1024), _i64s(128, 128, 128)
    need = lib.compact_bwd_group_workspace_bytes(65536, 1024, 3, ms, rs, 1)
    assert need >= lib.compact_bwd_workspace_bytes(65536, 1024, 1024, 128, 1)
    # 12 tiles of 128 x 256, 21 splits: 3 x 21 x 128 x 1024 fp32 partial sums (+ alignment)
    assert need >= 3 * 21 * 128 * 1024 * 4
    assert lib.compact_bwd_group_workspace_bytes(65536, 1024, 3, ms, rs, 0) == 0
    assert lib.compact_bwd_group_workspace_bytes(65536, 1024, 0, ms, rs, 1) == 0
    assert lib.compact_bwd_group_workspace_bytes(65536, 1024, 9, ms, rs, 1) == 0


@pytest.mark.parametrize("kw,status", [
    (dict(count=0), -1), (dict(count=9), -1), (dict(m=None), -1), (dict(r=None), -1),
    (dict(dx=None, G=None), -1),
    (dict(m=(1020, 1024, 1024)), -2),   # a slice that is not 16-byte aligned
    (dict(r=(128, 124, 128)), -2),
    (dict(r=(128, 128, 2000)), -1),     # r > n
    (dict(lddy=3000), -1),              # ld < sum of m
    (dict(ldz=376), -1),                # ld < sum of r
    (dict(G=(FAKE, None, FAKE)), -1),
    (dict(G=(FAKE, FAKE + 4, FAKE)), -2),
    (dict(ws=None), -4), (dict(ws_bytes=64), -4),
    (dict(accumulate=2), -1),
])
def test_bwd_group_validation(lib, kw, status):
    a = dict(dy=FAKE, lddy=3072, W=FAKE, ldw=3072, z=FAKE, ldz=384, dx=FAKE, lddx=1024, G=(FAKE, FAKE, FAKE),
             tokens=4096, n=1024, count=3, m=(1024, 1024, 1024), r=(128, 128, 128), dtype=1, accumulate=0, ws=FAKE,
             ws_bytes=1 << 40, stream=None)
    a.update(kw)
    arr = lambda v, t: None if v is None else (t * len(v))(*v)
    st = lib.compact_bwd_group(a["dy"], a["lddy"], a["W"], a["ldw"], a["z"], a["ldz"], a["dx"], a["lddx"],
                               arr(a["G"], ctypes.c_void_p), a["tokens"], a["n"], a["count"],
                               arr(a["m"], ctypes.c_int64), arr(a["r"], ctypes.c_int64), a["dtype"],
                               a["accumulate"], a["ws"], a["ws_bytes"], a["stream"])
    assert st == status
    assert lib.compact_last_error()


@pytest.mark.parametrize("kw,status", [
    (dict(t=0), -1), (dict(beta1=1.0), -1), (dict(beta2=-0.1), -1), (dict(eps=0.0), -1),
    (dict(lr=-1.0), -1), (dict(lr=float("nan")), -1), (dict(ws=None), -4),
    (dict(dtype=0, w_dtype=1), -3),  # fp32 decompression into bf16 weights
    (dict(M=None), -1), (dict(proj=1), -1),
])
def test_step_validation(lib, kw, status):
    a = dict(W=FAKE, ldw=1024, G=FAKE, M=FAKE, V=FAKE, n=1024, m=1024, r=128, seed=1, t=1,
             lr=1e-3, beta1=0.9, beta2=0.999, eps=1e-8, alpha=1.0, proj=0, dtype=1, w_dtype=1,
             ws=FAKE, ws_bytes=1 << 40, stream=None)
    a.update(kw)
    st = lib.compact_step(a["W"], a["ldw"], a["G"], a["M"], a["V"], a["n"], a["m"], a["r"],
                          a["seed"], a["t"], a["lr"], a["beta1"], a["beta2"], a["eps"], a["alpha"],
                          a["proj"], a["dtype"], a["w_dtype"], a["ws"], a["ws_bytes"], a["stream"])
    assert st == status


def test_projection_validation(lib):
    sparse = lambda s_: 2 | (s_ << 8)
    assert lib.compact_projection(1, 4, 4, sparse(65), FAKE, 4, None) == -1
    assert lib.compact_projection(1, 4, 4, sparse(8), None, 4, None) == -1
    assert lib.compact_projection(1, 4, 4, sparse(8), FAKE, 2, None) == -1
    assert lib.compact_projection(1, 4, 5, sparse(8), FAKE, 8, None) == -1      # r > n
    assert lib.compact_projection(1, 4, 3, 1, FAKE, 4, None) == -1              # identity needs r == n
    assert lib.compact_last_error()


def test_pstream_validation(lib):
    assert lib.compact_pstream(1, 0, 4, FAKE, 4, None) == -1
    assert lib.compact_pstream(1, 4, 4, None, 4, None) == -1
    assert lib.compact_pstream(1, 4, 4, FAKE, 2, None) == -1
    assert lib.compact_pstream_boxmuller(None, None, None, None, 0, None) == 0
    assert lib.compact_pstream_boxmuller(None, None, None, None, 5, None) == -1


def test_layer_batch_marshals_once_and_updates_seeds(lib):
    torch = pytest.importorskip("torch")
    import paper_2410_15352_amd as cp
    layers = [dict(W=torch.empty(64, 40, dtype=torch.bfloat16), G=torch.empty(8, 40), M=torch.empty(8, 40),
                   V=torch.empty(8, 40), seed=(i + 1) << 32, alpha=0.5) for i in range(3)]
    b = cp.prepare_layers(layers)
    assert b.count == 3
    assert [b.arr[i].seed for i in range(3)] == [(i + 1) << 32 for i in range(3)]
    assert [(b.arr[i].n, b.arr[i].m, b.arr[i].r) for i in range(3)] == [(64, 40, 8)] * 3
    b.set_seeds([7, 8, 9])
    assert [b.arr[i].seed for i in range(3)] == [7, 8, 9]
    # the workspace size is the same whether the layers come as a list or a batch
    assert cp.step_batched_workspace_bytes(b) == cp.step_batched_workspace_bytes(layers) > 0
    with pytest.raises(ValueError):
        b.set_seeds([1])
