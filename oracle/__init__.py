"""CPU oracle of the mixed-adapter LoRA step (test infrastructure only).

Only the tests, the smoke check and the benchmark's CPU-baseline leg may
import this package. The GPU library never calls it and it never calls the
GPU library: the two share nothing but the seeded inputs of `workloads`.

The arithmetic lives in `oracle.c` (plain loops, float64 accumulation). This
module builds it with gcc and marshals numpy arrays to it.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from typing import Optional, Tuple

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.c")
_LIB_PATH = os.path.join(_HERE, "liboracle.so")
_lib = None


def build(force: bool = True) -> str:
    """Compile oracle.c into liboracle.so (gcc, -O2, no fast-math)."""
    if force or not os.path.exists(_LIB_PATH):
        tmp = _LIB_PATH + ".tmp%d" % os.getpid()
        cmd = ["gcc", "-O2", "-std=c11", "-fopenmp", "-shared", "-fPIC",
               _SRC, "-o", tmp, "-lm"]
        subprocess.run(cmd, check=True)
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH):
        build(force=True)
    lib = ctypes.CDLL(_LIB_PATH)
    P = ctypes.c_void_p
    i32, i64, dbl = ctypes.c_int32, ctypes.c_int64, ctypes.c_double
    lib.oracle_num_threads.restype = ctypes.c_int
    lib.oracle_lora_linear.argtypes = [P, i64, i64, P, i64, P, P, i32, i32, P, P, P, P, P]
    lib.oracle_lora_linear.restype = None
    lib.oracle_block_version_check.argtypes = [P, i32, i32, P, P, i64, P, P, i64, P]
    lib.oracle_block_version_check.restype = i64
    lib.oracle_kv_append.argtypes = [P, P, i32, i32, P, i32, i64, i32, P, P, P, P]
    lib.oracle_kv_append.restype = None
    lib.oracle_paged_attn.argtypes = [P, P, i32, i32, i32, i32, P, P, P, i32, i64, P,
                                      P, P, dbl, P, P]
    lib.oracle_paged_attn.restype = None
    lib.oracle_to_bf16_array.argtypes = [P, i64, P]
    lib.oracle_to_bf16_array.restype = None
    _lib = lib
    return lib


def _p(a: Optional[np.ndarray]):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _c(a, dtype):
    if a is None:
        return None
    return np.ascontiguousarray(a, dtype=dtype)


def num_threads() -> int:
    return int(_load().oracle_num_threads())


def lora_linear(x, W, A=None, B=None, ranks=None, adapter_idx=None, scale=None,
                residual=None):
    """y = x W^T + scale * (x A_a^T) B_a^T (+ residual) per token, float64 [T, N].

    x [T,K], W [N,K], A [n_ad,r_max,K], B [n_ad,N,r_max], residual [T,N] as
    uint16 bf16 bits.
    """
    lib = _load()
    x = _c(x, np.uint16)
    W = _c(W, np.uint16)
    T, K = x.shape
    N = W.shape[0]
    assert W.shape[1] == K
    n_ad, r_max = 0, 8
    if A is not None:
        A = _c(A, np.uint16)
        B = _c(B, np.uint16)
        n_ad, r_max = A.shape[0], A.shape[1]
        assert A.shape[2] == K and B.shape == (n_ad, N, r_max)
        adapter_idx = _c(adapter_idx, np.int32)
        scale = _c(scale, np.float32)
        ranks = _c(ranks, np.int32)
        assert r_max <= 256
    res = _c(residual, np.uint16)
    if res is not None:
        assert res.shape == (T, N)
    y = np.empty((T, N), dtype=np.float64)
    lib.oracle_lora_linear(_p(x), T, K, _p(W), N, _p(A), _p(B), n_ad, r_max,
                           _p(ranks), _p(adapter_idx), _p(scale), _p(res), _p(y))
    return y


def block_version_check(block_table, ctx_lens, block_version, req_version,
                        cap: Optional[int] = None):
    """Returns (stale_pairs [min(n,cap),2] int32, n, valid_tokens [B] int32)."""
    lib = _load()
    bt = _c(block_table, np.int32)
    Bn, mb = bt.shape
    ctx = _c(ctx_lens, np.int32)
    bv = _c(block_version, np.int32)
    rv = _c(req_version, np.int32)
    if cap is None:
        cap = int(sum((int(L) + 15) // 16 for L in ctx))
    pairs = np.zeros((max(cap, 1), 2), dtype=np.int32)
    valid = np.zeros(Bn, dtype=np.int32)
    n = lib.oracle_block_version_check(_p(bt), Bn, mb, _p(ctx), _p(bv), bv.shape[0],
                                       _p(rv), _p(pairs), cap, _p(valid))
    return pairs[:min(n, cap)].copy(), int(n), valid


def kv_append(k_cache, v_cache, Hkv, D, block_table, q_indptr, ctx_lens,
              k_new, v_new):
    """In-place append of k_new/v_new [T,Hkv,D] into the uint16 pools."""
    lib = _load()
    assert k_cache.dtype == np.uint16 and k_cache.flags.c_contiguous
    assert v_cache.dtype == np.uint16 and v_cache.flags.c_contiguous
    bt = _c(block_table, np.int32)
    qi = _c(q_indptr, np.int32)
    ctx = _c(ctx_lens, np.int32)
    kn = _c(k_new, np.uint16)
    vn = _c(v_new, np.uint16)
    num_blocks = k_cache.size // (Hkv * 16 * D)
    lib.oracle_kv_append(_p(k_cache), _p(v_cache), Hkv, D, _p(bt), bt.shape[1], num_blocks,
                         bt.shape[0], _p(qi), _p(ctx), _p(kn), _p(vn))


def paged_attn(q, q_indptr, Hq, Hkv, D, k_cache, v_cache, block_table,
               ctx_lens, block_version, req_version, sm_scale) -> Tuple[np.ndarray, np.ndarray]:
    """Returns (out [T,Hq,D] float64, lse [T,Hq] float64)."""
    lib = _load()
    q = _c(q, np.uint16)
    qi = _c(q_indptr, np.int32)
    T = int(qi[-1])
    assert q.size == T * Hq * D
    kc = _c(k_cache, np.uint16)
    vc = _c(v_cache, np.uint16)
    bt = _c(block_table, np.int32)
    out = np.empty((T, Hq, D), dtype=np.float64)
    lse = np.empty((T, Hq), dtype=np.float64)
    num_blocks = kc.size // (Hkv * 16 * D)
    lib.oracle_paged_attn(_p(q), _p(qi), bt.shape[0], Hq, Hkv, D, _p(kc), _p(vc),
                          _p(bt), bt.shape[1], num_blocks, _p(_c(ctx_lens, np.int32)),
                          _p(_c(block_version, np.int32)),
                          _p(_c(req_version, np.int32)), float(sm_scale),
                          _p(out), _p(lse))
    return out, lse


def to_bf16(v: np.ndarray) -> np.ndarray:
    """float64 -> bf16 bits (uint16), round to nearest even through float32."""
    lib = _load()
    v = _c(v, np.float64)
    out = np.empty(v.shape, dtype=np.uint16)
    lib.oracle_to_bf16_array(_p(v), v.size, _p(out))
    return out


def bf16_to_f64(u: np.ndarray) -> np.ndarray:
    """bf16 bits (uint16) -> float64, exact."""
    u = np.ascontiguousarray(u, dtype=np.uint16)
    return (u.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
