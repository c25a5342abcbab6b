"""Test-side helpers: small paged pools built with numpy reshapes.

The pool layout is the one the library's interface documents:
    k_cache [num_blocks][Hkv][D/8][16][8],  v_cache [num_blocks][Hkv][D][16].
These helpers reach it through numpy reshape/transpose of dense arrays
[num_blocks][Hkv][16][D], which is a different computation from the oracle's
index arithmetic, so tests built on them pin that arithmetic.
"""
from __future__ import annotations

import numpy as np

BS = 16


def f32_to_bf16_bits(a: np.ndarray) -> np.ndarray:
    """Round float values to bf16 (nearest even) and return the uint16 bits."""
    f = np.ascontiguousarray(a, dtype=np.float32)
    u = f.view(np.uint32).astype(np.uint64)
    lsb = (u >> 16) & 1
    u = (u + 0x7FFF + lsb) >> 16
    return u.astype(np.uint16)


def bits_to_f64(u: np.ndarray) -> np.ndarray:
    u = np.ascontiguousarray(u, dtype=np.uint16)
    return (u.astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def rand_bf16(rng, shape, std=1.0) -> np.ndarray:
    return f32_to_bf16_bits(rng.standard_normal(shape).astype(np.float32) * std)


def dense_to_pool(kd: np.ndarray, vd: np.ndarray):
    """kd, vd [nb][Hkv][16][D] (uint16) -> (k_cache, v_cache) flat uint16."""
    nb, hkv, bs, D = kd.shape
    assert bs == BS
    kc = kd.reshape(nb, hkv, BS, D // 8, 8).transpose(0, 1, 3, 2, 4)
    vc = vd.transpose(0, 1, 3, 2)
    return np.ascontiguousarray(kc).reshape(-1), np.ascontiguousarray(vc).reshape(-1)


def pool_to_dense(kc: np.ndarray, vc: np.ndarray, nb: int, hkv: int, D: int):
    kd = kc.reshape(nb, hkv, D // 8, BS, 8).transpose(0, 1, 3, 2, 4).reshape(nb, hkv, BS, D)
    vd = vc.reshape(nb, hkv, D, BS).transpose(0, 1, 3, 2)
    return np.ascontiguousarray(kd), np.ascontiguousarray(vd)


def make_table(rng, ctx_lens, extra_blocks=0, max_blocks=None):
    """Random permutation block table; returns (table [B,mb], num_blocks)."""
    nbs = [(int(L) + BS - 1) // BS for L in ctx_lens]
    num = sum(nbs) + extra_blocks
    perm = rng.permutation(num).astype(np.int32)
    mb = max(1, max(nbs) if nbs else 1) if max_blocks is None else max_blocks
    table = np.zeros((len(ctx_lens), mb), dtype=np.int32)
    off = 0
    for b, n in enumerate(nbs):
        table[b, :n] = perm[off:off + n]
        off += n
    return table, num


def gather_request(kd, vd, table, b, L, g):
    """Dense K, V [L][D] (float64) of request b, KV head g."""
    pos = np.arange(L)
    blocks = table[b, pos // BS]
    slots = pos % BS
    return bits_to_f64(kd[blocks, g, slots, :]), bits_to_f64(vd[blocks, g, slots, :])
