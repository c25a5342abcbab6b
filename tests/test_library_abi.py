"""The C-ABI library loads, exports every declared entry point, and rejects bad
arguments on the host before launching anything. Nothing here needs a GPU:
only workspace-size queries and argument errors are exercised, and both return
before any HIP call."""
import ctypes
import os
import re

import pytest

import paper_2608_15241_amd as lk

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

OK, ERR_NULL, ERR_SHAPE, ERR_UNSUPPORTED, ERR_WORKSPACE = 0, 1, 2, 3, 4
# Never dereferenced: every call below either only queries a size (ws NULL)
# or fails argument validation, both of which return before any launch.
FAKE = ctypes.c_void_p(0x1000)


def declared_symbols():
    names = set()
    for fn in os.listdir(os.path.join(ROOT, "include")):
        if fn.endswith(".h"):
            text = open(os.path.join(ROOT, "include", fn)).read()
            names |= set(re.findall(r"^\s*(?:[\w\*]+\s+)+\**(local_\w+)\s*\(", text, re.M))
    return names


@pytest.fixture(scope="module")
def lib():
    return lk.load_library()


def test_every_declared_symbol_is_exported(lib):
    names = declared_symbols()
    assert {"local_lora_linear", "local_paged_attn_decode", "local_paged_attn_prefill",
            "local_block_version_check", "local_last_error", "local_version"} <= names
    for n in names:
        assert hasattr(lib, n), n
    assert set(lk.EXPORTS) == names


def _size(fn, *args):
    n = ctypes.c_size_t(0)
    st = fn(*args, None, ctypes.byref(n), None)
    return st, n.value


def test_lora_linear_workspace_and_errors(lib):
    f = lib.local_lora_linear
    # sizes only: T=32, K=N=4096, 8 adapters of rank 16
    st, n = _size(f, FAKE, 32, 4096, FAKE, 4096, FAKE, FAKE, 8, 16, None, FAKE, FAKE, None, FAKE)
    assert st == OK
    # decode sizes: fp32 base partial sums (4 K slices x T x N), then the
    # shrink's, fused into the base product (4 K slices x T x n_adapters*r_max)
    assert n == 4 * 32 * 4096 * 4 + 4 * 32 * 128 * 4
    # a shrink too wide to fuse (N = 64: two 48-row feature tiles for 256
    # stacked rows, 8 base K slices) runs on its own: 8 K slices x T x r_max
    st, n2 = _size(f, FAKE, 32, 4096, FAKE, 64, FAKE, FAKE, 16, 16, None, FAKE, FAKE, None, FAKE)
    assert st == OK and n2 == 8 * 32 * 64 * 4 + 8 * 32 * 16 * 4
    # above 256 tokens: the shrink's fp32 partial sums for each token's own
    # adapter, 8 K slices (the most; 5 tiles of 64 tokens) x T x r_max, then
    # a 32-byte adapter bitmap per 64-token tile, each part 256-byte aligned
    st, n1 = _size(f, FAKE, 300, 4096, FAKE, 4096, FAKE, FAKE, 8, 16, None, FAKE, FAKE, None, FAKE)
    assert st == OK and n1 == 8 * 300 * 16 * 4 + 256
    # 2048 tokens (32 tiles of 64): 8 slices fill the chip (fewer do not fit LDS)
    st, n2k = _size(f, FAKE, 2048, 4096, FAKE, 4096, FAKE, FAKE, 4, 16, None, FAKE, FAKE, None, FAKE)
    assert st == OK and n2k == 8 * 2048 * 16 * 4 + 32 * 32
    st, n0 = _size(f, FAKE, 32, 4096, FAKE, 4096, None, None, 0, 0, None, None, None, None, FAKE)
    assert st == OK and n0 == 4 * 32 * 4096 * 4
    assert _size(f, FAKE, 32, 100, FAKE, 4096, None, None, 0, 0, None, None, None, None, FAKE)[0] == ERR_UNSUPPORTED
    assert _size(f, FAKE, 32, 4096, FAKE, 4096, FAKE, FAKE, 8, 12, None, FAKE, FAKE, None, FAKE)[0] == ERR_UNSUPPORTED
    assert _size(f, FAKE, -1, 4096, FAKE, 4096, None, None, 0, 0, None, None, None, None, FAKE)[0] == ERR_SHAPE
    assert b"lora_linear" in lib.local_last_error()
    # NULL pointers are reported before any launch
    n = ctypes.c_size_t(1 << 30)
    st = f(None, 32, 4096, FAKE, 4096, None, None, 0, 0, None, None, None, None, FAKE,
           FAKE, ctypes.byref(n), None)
    assert st == ERR_NULL
    st = f(FAKE, 32, 4096, FAKE, 4096, FAKE, None, 8, 16, None, FAKE, FAKE, None, FAKE,
           FAKE, ctypes.byref(n), None)
    assert st == ERR_NULL
    # too small a workspace (adapters present, so one is needed)
    n = ctypes.c_size_t(16)
    st = f(FAKE, 32, 4096, FAKE, 4096, FAKE, FAKE, 8, 16, None, FAKE, FAKE, None, FAKE,
           FAKE, ctypes.byref(n), None)
    assert st == ERR_WORKSPACE
    assert f(FAKE, 32, 4096, FAKE, 4096, None, None, 0, 0, None, None, None, None, FAKE,
             FAKE, None, None) == ERR_WORKSPACE


def test_decode_workspace_and_errors(lib):
    f = lib.local_paged_attn_decode

    def call(B=32, Hq=32, Hkv=32, D=128, bs=16, mb=256, kn=FAKE, vn=FAKE, nblocks=5000):
        return _size(f, FAKE, B, Hq, Hkv, D, kn, vn, FAKE, FAKE, nblocks, bs, FAKE, mb, FAKE,
                     FAKE, FAKE, 0.088, FAKE, FAKE)

    st, n = call()
    assert st == OK and n == 32 * 32 * 8 * (128 + 2) * 4    # 8 partitions of 512 tokens
    assert call(Hq=32, Hkv=6)[0] == ERR_SHAPE
    assert call(D=96)[0] == ERR_UNSUPPORTED
    assert call(bs=32)[0] == ERR_UNSUPPORTED
    assert call(Hq=64, Hkv=2)[0] == ERR_UNSUPPORTED          # group 32 > 16
    assert call(kn=None)[0] == ERR_NULL                        # k_new without v_new


def test_prefill_and_version_check_errors(lib):
    st, n = _size(lib.local_paged_attn_prefill, FAKE, FAKE, 4, 2048, 32, 32, 128, FAKE, FAKE,
                  FAKE, FAKE, 352, 16, FAKE, 160, FAKE, FAKE, FAKE, 0.088, FAKE, FAKE)
    # partial results of split tiles: (T/128 + B) tiles x 32 heads x 4 key ranges x
    # 128 rows x (D + 2) floats; then the plan: 256 bytes of counts and the schedule:
    # two int4 per unit, 4 units per tile bound, then one int4 per split tile
    tiles = 2048 // 128 + 4
    parts = tiles * 32 * 4 * 128 * (128 + 2) * 4
    assert st == OK and n == (parts + 255) // 256 * 256 + 256 + tiles * 4 * 32 + tiles * 16
    ws = ctypes.c_size_t(n - 1)
    assert lib.local_paged_attn_prefill(FAKE, FAKE, 4, 2048, 32, 32, 128, FAKE, FAKE, FAKE,
                                        FAKE, 352, 16, FAKE, 160, FAKE, FAKE, FAKE, 0.088, FAKE,
                                        FAKE, FAKE, ctypes.byref(ws), None) == ERR_WORKSPACE
    st, _ = _size(lib.local_paged_attn_prefill, FAKE, FAKE, 4, 2048, 32, 32, 80, FAKE, FAKE,
                  FAKE, FAKE, 352, 16, FAKE, 160, FAKE, FAKE, FAKE, 0.088, FAKE, FAKE)
    assert st == ERR_UNSUPPORTED
    f = lib.local_block_version_check
    st, n = _size(f, FAKE, 128, 1024, FAKE, 16, FAKE, 70000, FAKE, FAKE, 1000, FAKE, FAKE)
    assert st == OK and n == 128 * 4
    assert _size(f, FAKE, 128, 1024, FAKE, 8, FAKE, 70000, FAKE, FAKE, 1000, FAKE,
                 FAKE)[0] == ERR_UNSUPPORTED
    assert _size(f, FAKE, 128, 0, FAKE, 16, FAKE, 70000, FAKE, FAKE, 1000, FAKE,
                 FAKE)[0] == ERR_SHAPE
    assert _size(f, FAKE, 128, 16, FAKE, 16, FAKE, 0, FAKE, FAKE, 1000, FAKE,
                 FAKE)[0] == ERR_SHAPE
    nn = ctypes.c_size_t(4096)
    assert f(FAKE, 128, 1024, FAKE, 16, FAKE, 70000, FAKE, None, 10, FAKE, FAKE, FAKE,
             ctypes.byref(nn), None) == ERR_NULL


def test_binding_refuses_cpu_tensors():
    import torch
    x = torch.zeros((4, 64), dtype=torch.bfloat16)
    with pytest.raises(ValueError, match="GPU"):
        lk.local_lora_linear(x, torch.zeros((64, 64), dtype=torch.bfloat16))


def test_lora_linear_grouped_workspace_and_errors(lib):
    f = lib.local_lora_linear_grouped
    P = ctypes.c_void_p
    ptrs = lambda n: (P * n)(*([FAKE] * n))
    Ns = (ctypes.c_int64 * 3)(4096, 4096, 4096)
    # q, k, v of a 7B layer at T=32 with 8 rank-16 adapters: one virtual weight
    # of 12288 rows in 96-row tiles, K in 2 slices (256 workgroups), the shrink
    # fused (3 x 128 stacked rows): base sums 2 x 32 x 12288 fp32, shrink sums
    # 2 x 32 x 384 fp32
    st, n = _size(f, FAKE, 32, 4096, 3, ptrs(3), Ns, ptrs(3), ptrs(3), 8, 16, None, FAKE,
                  FAKE, ptrs(3))
    assert st == OK and n == 2 * 32 * 12288 * 4 + 2 * 32 * 384 * 4
    # a 2048-token chunk: one launch over the three projections, the shrink's
    # partial sums per projection (8 K slices x T x r_max fp32 each), then the
    # adapter bitmaps (32 bytes per 64-token tile)
    st, n = _size(f, FAKE, 2048, 4096, 3, ptrs(3), Ns, ptrs(3), ptrs(3), 4, 16, None, FAKE,
                  FAKE, ptrs(3))
    assert st == OK and n == 3 * 8 * 2048 * 16 * 4 + 32 * 32
    assert _size(f, FAKE, 32, 4096, 0, ptrs(1), Ns, None, None, 0, 0, None, None, None,
                 ptrs(1))[0] == ERR_UNSUPPORTED
    assert _size(f, FAKE, 32, 4096, 5, ptrs(5), Ns, None, None, 0, 0, None, None, None,
                 ptrs(5))[0] == ERR_UNSUPPORTED
    assert _size(f, FAKE, 32, 4096, 3, None, Ns, None, None, 0, 0, None, None, None,
                 ptrs(3))[0] == ERR_NULL
    bad = (ctypes.c_int64 * 3)(4096, 100, 4096)
    assert _size(f, FAKE, 32, 4096, 3, ptrs(3), bad, None, None, 0, 0, None, None, None,
                 ptrs(3))[0] == ERR_UNSUPPORTED
    assert b"grouped" in lib.local_last_error()


def test_lora_grad_workspace_and_errors(lib):
    f = lib.local_lora_grad
    # T=300, K=512, N=640, 4 adapters of rank 16. Parts, each 256-byte aligned:
    # the bucketed token order (T int32), the adapter offsets and the unit
    # offsets (n+1 int32 each), the unit table (16 bytes for each of at most
    # T/64 + n 64-token units), B transposed (n x r_max x N bf16), the
    # shrinks' partial sums of x against A (8 K slices x T x r_max fp32) and of
    # dy against B^T (10 slices), each followed by 32 bytes of adapter bitmap
    # per 64-token tile, then the units' partial products (units x N x r_max
    # and units x K x r_max fp32).
    a = lambda v: (v + 255) // 256 * 256
    st, n = _size(f, FAKE, 300, 512, FAKE, 640, FAKE, FAKE, 4, 16, None, FAKE, FAKE, FAKE, FAKE)
    assert st == OK
    units = 300 // 64 + 4
    assert n == (a(300 * 4) + 2 * a(5 * 4) + a(units * 16) + a(4 * 16 * 640 * 2)
                 + a(8 * 300 * 16 * 4) + a(5 * 32) + a(10 * 300 * 16 * 4) + a(5 * 32)
                 + a(units * 640 * 16 * 4) + a(units * 512 * 16 * 4))
    st, n0 = _size(f, FAKE, 0, 512, FAKE, 640, FAKE, FAKE, 4, 16, None, FAKE, FAKE, FAKE, FAKE)
    assert st == OK and n0 > 0                     # T = 0 still runs the bucket and reduce passes
    assert _size(f, FAKE, 300, 512, FAKE, 640, FAKE, FAKE, 4, 12, None, FAKE, FAKE, FAKE,
                 FAKE)[0] == ERR_UNSUPPORTED
    assert _size(f, FAKE, 300, 100, FAKE, 640, FAKE, FAKE, 4, 16, None, FAKE, FAKE, FAKE,
                 FAKE)[0] == ERR_UNSUPPORTED
    assert _size(f, FAKE, 300, 512, FAKE, 640, FAKE, FAKE, 0, 16, None, FAKE, FAKE, FAKE,
                 FAKE)[0] == ERR_SHAPE
    assert b"lora_grad" in lib.local_last_error()
    big = ctypes.c_size_t(1 << 40)
    assert f(None, 300, 512, FAKE, 640, FAKE, FAKE, 4, 16, None, FAKE, FAKE, FAKE, FAKE, FAKE,
             ctypes.byref(big), None) == ERR_NULL
    assert f(FAKE, 300, 512, FAKE, 640, FAKE, FAKE, 4, 16, None, FAKE, FAKE, None, FAKE, FAKE,
             ctypes.byref(big), None) == ERR_NULL
    small = ctypes.c_size_t(n - 1)
    assert f(FAKE, 300, 512, FAKE, 640, FAKE, FAKE, 4, 16, None, FAKE, FAKE, FAKE, FAKE, FAKE,
             ctypes.byref(small), None) == ERR_WORKSPACE
    g = lib.local_lora_grad_input
    # the transposed adapters, then the forward projection's workspace for
    # x = dy [T, N] against the transposed weight [K, N]
    st, m = _size(g, FAKE, 300, 640, FAKE, 512, FAKE, FAKE, 4, 16, None, FAKE, FAKE, FAKE)
    st2, fw = _size(lib.local_lora_linear, FAKE, 300, 640, FAKE, 512, FAKE, FAKE, 4, 16, None,
                    FAKE, FAKE, None, FAKE)
    assert st == OK and st2 == OK
    assert m == a(4 * 16 * 640 * 2) + a(4 * 512 * 16 * 2) + fw
    assert g(FAKE, 300, 640, FAKE, 512, FAKE, FAKE, 4, 16, None, FAKE, FAKE, None, FAKE,
             ctypes.byref(big), None) == ERR_NULL


def test_lora_grad_grouped_workspace_and_errors(lib):
    f = lib.local_lora_grad_grouped
    P = ctypes.c_void_p
    ptrs = lambda n: (P * n)(*([FAKE] * n))
    Ns = (ctypes.c_int64 * 3)(4096, 1024, 1024)
    st, n = _size(f, FAKE, 2048, 4096, 3, ptrs(3), Ns, ptrs(3), ptrs(3), 4, 16, None, FAKE,
                  FAKE, ptrs(3), ptrs(3))
    assert st == OK
    # at least the three projections' partial products (units x (N_g + K) x r_max fp32)
    units = 2048 // 64 + 4
    assert n > units * (4096 + 1024 + 1024 + 3 * 4096) * 16 * 4
    assert _size(f, FAKE, 2048, 4096, 5, ptrs(5), Ns, ptrs(5), ptrs(5), 4, 16, None, FAKE,
                 FAKE, ptrs(5), ptrs(5))[0] == ERR_UNSUPPORTED
    assert _size(f, FAKE, 2048, 4096, 3, None, Ns, ptrs(3), ptrs(3), 4, 16, None, FAKE,
                 FAKE, ptrs(3), ptrs(3))[0] == ERR_NULL
    bad = (ctypes.c_int64 * 3)(4096, 100, 1024)
    assert _size(f, FAKE, 2048, 4096, 3, ptrs(3), bad, ptrs(3), ptrs(3), 4, 16, None, FAKE,
                 FAKE, ptrs(3), ptrs(3))[0] == ERR_UNSUPPORTED
    assert b"lora_grad_grouped" in lib.local_last_error()


def test_decode_noalloc_rejects_sizes_beyond_its_scratch(lib):
    # The no-workspace decode entry point holds a fixed scratch of
    # LOCAL_DECODE_NOALLOC_SCRATCH_BYTES; a call that would need more is
    # refused on the host, before any HIP call.
    f = lib.local_paged_attn_decode_noalloc
    limit = 68157440
    text = open(os.path.join(ROOT, "include", "local.h")).read()
    assert re.search(r"#define LOCAL_DECODE_NOALLOC_SCRATCH_BYTES \(\(size_t\)%d\)" % limit, text)

    def call(B=129, Hq=32, Hkv=8, D=128, mb=1024, bs=16, kn=FAKE, vn=FAKE):
        return f(FAKE, B, Hq, Hkv, D, kn, vn, FAKE, FAKE, 100000, bs, FAKE, mb, FAKE, FAKE,
                 FAKE, 0.088, FAKE, FAKE, None)

    # partitions of 32 blocks for tables up to 256 wide, 48 up to 512, 64 beyond
    assert 256 * 32 * 16 * (128 + 2) * 4 == limit      # 1024 blocks: 16 partitions
    assert call(B=257) == ERR_UNSUPPORTED               # one request more: refused
    assert b"scratch" in lib.local_last_error()
    assert 512 * 32 * 8 * (128 + 2) * 4 == limit       # 256 blocks: 8 partitions
    assert call(B=513, mb=256) == ERR_UNSUPPORTED
    assert 372 * 32 * 11 <= 131072 < 373 * 32 * 11      # 512 blocks: 11 partitions of 48
    assert call(B=373, mb=512) == ERR_UNSUPPORTED
    assert call(B=1, Hq=32, mb=64 * 4097) == ERR_UNSUPPORTED
    assert call(B=0) == OK                              # nothing to do, nothing launched
    assert call(Hq=32, Hkv=6) == ERR_SHAPE
    assert call(D=96) == ERR_UNSUPPORTED
    assert call(bs=8) == ERR_UNSUPPORTED
    assert call(kn=None) == ERR_NULL


def test_kv_pool_conversion_errors(lib):
    A, B, C, D_ = (ctypes.c_void_p(x) for x in (0x100000, 0x200000, 0x300000, 0x400000))
    for f in (lib.local_kv_pool_import, lib.local_kv_pool_export):
        # 0 blocks: nothing to do, nothing launched
        assert f(A, B, 0, 8, 128, 16, C, D_, None) == OK
        assert f(None, None, 0, 8, 128, 16, None, None, None) == OK
        assert f(None, B, 4, 8, 128, 16, C, D_, None) == ERR_NULL
        assert f(A, B, 4, 8, 128, 16, C, None, None) == ERR_NULL
        assert f(A, B, -1, 8, 128, 16, C, D_, None) == ERR_SHAPE
        assert f(A, B, 4, 0, 128, 16, C, D_, None) == ERR_SHAPE
        assert f(A, B, 4, 8, 96, 16, C, D_, None) == ERR_UNSUPPORTED
        assert f(A, B, 4, 8, 128, 8, C, D_, None) == ERR_UNSUPPORTED
        # 4 blocks x 8 heads x 4 KB = 128 KB per pool: these ranges overlap
        assert f(A, B, 4, 8, 128, 16, ctypes.c_void_p(0x110000), D_, None) == ERR_SHAPE
        assert f(A, B, 4, 8, 128, 16, C, ctypes.c_void_p(0x310000), None) == ERR_SHAPE
        assert b"overlap" in lib.local_last_error()
