"""Seeded synthetic inputs for the workloads in `configs`.

This module draws inputs only. It holds none of the method's arithmetic, and
both the kernels and the oracle consume what it produces.

* Integer metadata (context lengths, adapter assignment, the block-pool
  permutation and the stale draw) comes from numpy's PCG64. Each item gets
  its own child of `SeedSequence(seed)`, spawned in a fixed order, so adding
  an item never changes the others.
* Float tensors come from a seeded `torch.Generator` on the target device.
  They are drawn in float32 and rounded to bf16 (nearest even). Large pools
  are drawn chunk by chunk, so that no float32 copy of a whole pool exists.

Structure (how the readings of the paper are applied):
* Context lengths. In decode, ctx_lens[b] counts the token being decoded,
  whose K/V the step appends at position ctx_lens[b]-1. In prefill,
  ctx_lens[b] = prefix[b] + chunk.
* Adapter versions. Adapter a's committed version is 1000*(a+1). Tags are
  therefore unique across adapters, so one equality test checks both the
  adapter and the version components of the validity key (§5.1). A request
  binds the committed version of its adapter (§4.2).
* Stale draw. A stale block carries version - 1 (the superseded version, §1
  challenge (2)). The stale entries are round(frac * #entries) block-table
  entries drawn without replacement. Each request's last block is excluded,
  because it is the block the step appends to under the current version.
* Block pool. num_blocks = sum_b ceil(ctx_lens[b]/16). Physical ids are a
  random permutation, handed out in (b, j) order. Table entries past a
  request's blocks are 0 and are never read.
"""
from __future__ import annotations

import math
from dataclasses import dataclass
from typing import Dict, List, Optional

import numpy as np

from .configs import BLOCK_SIZE, LORA_SCALE, Workload

VERSION_STRIDE = 1000

# Order in which SeedSequence children are spawned (never reorder).
_META_ITEMS = ("ctx", "adapter", "perm", "stale")


def adapter_version(a: int) -> int:
    return VERSION_STRIDE * (a + 1)


@dataclass
class Meta:
    """Host-side integer metadata of one step (identical for every layer)."""
    ctx_lens: np.ndarray        # [B] int32
    n_new: np.ndarray           # [B] int32 tokens appended this step
    q_indptr: np.ndarray        # [B+1] int32
    request_adapter: np.ndarray  # [B] int32
    req_version: np.ndarray     # [B] int32
    block_table: np.ndarray     # [B, max_blocks] int32
    block_version: np.ndarray   # [num_blocks] int32
    num_blocks: int
    max_blocks: int
    stale_entries: np.ndarray   # [n, 2] int32 (b, j) in lexicographic order
    token_adapter: np.ndarray   # [T] int32 adapter of each token
    token_scale: np.ndarray     # [T] float32

    @property
    def T(self) -> int:
        return int(self.q_indptr[-1])

    @property
    def B(self) -> int:
        return int(self.ctx_lens.shape[0])


def _children(seed: int):
    ss = np.random.SeedSequence(seed)
    kids = ss.spawn(len(_META_ITEMS))
    return {name: np.random.Generator(np.random.PCG64(k))
            for name, k in zip(_META_ITEMS, kids)}


def _draw_ctx(w: Workload, rng) -> np.ndarray:
    kind = w.ctx[0]
    if kind == "fixed":
        base = np.asarray(w.ctx[1], dtype=np.int64)
        assert base.shape[0] == w.batch
    elif kind == "uniform":
        lo, hi = w.ctx[1], w.ctx[2]
        base = rng.integers(lo, hi, size=w.batch, endpoint=True)
    elif kind == "loguniform":
        lo, hi = w.ctx[1], w.ctx[2]
        base = np.rint(np.exp(rng.uniform(math.log(lo), math.log(hi),
                                          size=w.batch))).astype(np.int64)
        base = np.clip(base, lo, hi)
    else:
        raise ValueError(kind)
    if w.kind == "prefill":
        return (base + w.chunk).astype(np.int32)
    return base.astype(np.int32)


def _draw_adapters(w: Workload, rng, B: int) -> np.ndarray:
    if w.n_adapters == 0:
        return np.full(B, -1, dtype=np.int32)
    if w.assignment == "uniform":
        return rng.integers(0, w.n_adapters, size=B).astype(np.int32)
    if w.assignment == "zipf":
        k = np.arange(w.n_adapters, dtype=np.float64)
        p = (k + 1.0) ** (-w.zipf_s)
        p /= p.sum()
        return rng.choice(w.n_adapters, size=B, p=p).astype(np.int32)
    raise ValueError(w.assignment)


def make_meta(w: Workload, seed: int = 0,
              ctx_override: Optional[np.ndarray] = None,
              max_blocks: Optional[int] = None) -> Meta:
    rngs = _children(seed)
    ctx = _draw_ctx(w, rngs["ctx"])
    if ctx_override is not None:
        ctx = np.asarray(ctx_override, dtype=np.int32)
    B = int(ctx.shape[0])
    adapters = _draw_adapters(w, rngs["adapter"], B)
    nb = (ctx.astype(np.int64) + BLOCK_SIZE - 1) // BLOCK_SIZE
    num_blocks = int(nb.sum())
    mb = int(max(1, nb.max() if B else 1)) if max_blocks is None else max_blocks
    assert mb >= (nb.max() if B else 0)
    perm = rngs["perm"].permutation(num_blocks).astype(np.int32)
    table = np.zeros((B, mb), dtype=np.int32)
    off = 0
    for b in range(B):
        table[b, :nb[b]] = perm[off:off + nb[b]]
        off += nb[b]
    req_version = np.array([adapter_version(a) if a >= 0 else 0
                            for a in adapters], dtype=np.int32)
    block_version = np.zeros(num_blocks, dtype=np.int32)
    for b in range(B):
        block_version[table[b, :nb[b]]] = req_version[b]
    # stale draw: entries other than each request's last block
    stale = np.zeros((0, 2), dtype=np.int32)
    if w.stale_frac > 0 and B:
        cand = np.array([(b, j) for b in range(B) for j in range(nb[b] - 1)],
                        dtype=np.int64).reshape(-1, 2)
        n_st = int(round(w.stale_frac * num_blocks))
        n_st = min(n_st, cand.shape[0])
        pick = rngs["stale"].choice(cand.shape[0], size=n_st, replace=False)
        stale = cand[np.sort(pick)]
        order = np.lexsort((stale[:, 1], stale[:, 0]))
        stale = stale[order].astype(np.int32)
        for b, j in stale:
            block_version[table[b, j]] = req_version[b] - 1
    if w.kind == "prefill":
        n_new = np.full(B, w.chunk, dtype=np.int32)
    else:
        n_new = np.ones(B, dtype=np.int32)
    q_indptr = np.zeros(B + 1, dtype=np.int32)
    q_indptr[1:] = np.cumsum(n_new)
    token_adapter = np.repeat(adapters, n_new).astype(np.int32)
    token_scale = np.where(token_adapter >= 0, LORA_SCALE, 0.0).astype(np.float32)
    return Meta(ctx_lens=ctx, n_new=n_new, q_indptr=q_indptr,
                request_adapter=adapters, req_version=req_version,
                block_table=table, block_version=block_version,
                num_blocks=num_blocks, max_blocks=mb, stale_entries=stale,
                token_adapter=token_adapter, token_scale=token_scale)


# ---------------------------------------------------------------- floats

def _gen(device, seed: int):
    import torch
    g = torch.Generator(device=device)
    g.manual_seed(int(seed))
    return g


def randn_bf16(shape, std: float, device, seed: int, chunk_elems: int = 1 << 28):
    """N(0, std^2) drawn in float32 and rounded to bf16, chunk by chunk."""
    import torch
    out = torch.empty(shape, dtype=torch.bfloat16, device=device)
    flat = out.view(-1)
    g = _gen(device, seed)
    n = flat.numel()
    for s in range(0, n, chunk_elems):
        e = min(n, s + chunk_elems)
        tmp = torch.randn(e - s, generator=g, device=device, dtype=torch.float32)
        if std != 1.0:
            tmp.mul_(std)
        flat[s:e].copy_(tmp)
        del tmp
    return out


def make_adapters(w: Workload, proj: str, device, seed: int):
    """Stacked A [n_ad][r_max][K] and B [n_ad][N][r_max]; zero beyond rank."""
    import torch
    N, K = w.proj_shape(proj)
    r_max = w.r_max
    A = torch.zeros((w.n_adapters, r_max, K), dtype=torch.bfloat16, device=device)
    Bm = torch.zeros((w.n_adapters, N, r_max), dtype=torch.bfloat16, device=device)
    for a, r in enumerate(w.ranks):
        A[a, :r] = randn_bf16((r, K), 1.0 / math.sqrt(r), device, seed + 2 * a)
        Bm[a, :, :r] = randn_bf16((N, r), 0.01, device, seed + 2 * a + 1)
    ranks = torch.tensor(list(w.ranks), dtype=torch.int32, device=device)
    return A, Bm, ranks


def make_layer_weights(w: Workload, layer: int, device, seed: int) -> Dict:
    """Base weights and (for LoRA targets) adapters of one layer."""
    out = {}
    for i, proj in enumerate(("q", "k", "v", "o")):
        N, K = w.proj_shape(proj)
        s = seed * 1_000_003 + layer * 10_007 + i * 1009
        out["W_" + proj] = randn_bf16((N, K), 0.02, device, s)
        if proj in w.lora_targets and w.n_adapters > 0:
            A, Bm, ranks = make_adapters(w, proj, device, s + 101)
            out["A_" + proj], out["B_" + proj], out["ranks_" + proj] = A, Bm, ranks
    return out


def make_kv_pool(w: Workload, meta: Meta, device, seed: int, n_layers: Optional[int] = None):
    """KV pool [n_layers][2][num_blocks][Hkv][16*D] bf16, N(0,1).

    Index [l][0] is layer l's K pool and [l][1] its V pool; each block row
    is reinterpreted in the in-block order of the library's layout.
    """
    L = w.n_layers if n_layers is None else n_layers
    shape = (L, 2, meta.num_blocks, w.hkv, BLOCK_SIZE * w.head_dim)
    return randn_bf16(shape, 1.0, device, seed * 7919 + 17)


def to_host_u16(t) -> np.ndarray:
    """bf16 tensor -> numpy uint16 array of the same bits (host copy)."""
    import torch
    return t.detach().contiguous().view(torch.int16).cpu().numpy().view(np.uint16)
