"""Stale-coverage prefill under a staged adapter version, then publication
(§5.3), end to end: the host KV manager plans and records coverage, the
kernels compute it, the oracle checks it.

  1. Eight prefixes are prefilled under the committed version c and recorded.
  2. Requests heat them unevenly; the trained adapter is staged as s.
  3. The manager's plan lists them; they are re-prefilled under s in chunks of
     128 tokens (8 blocks), with the staged adapter weights and req_version s,
     into fresh private blocks tagged s. Between rounds a foreground request
     bound to c decodes over committed coverage, with a staged block forced
     into its table: the tag test must drop it.
  4. Publication: a request bound to s now matches the warmed blocks; its
     decode equals the oracle's decode over K/V computed from scratch under
     the staged weights (the chunked re-prefill wrote the same K/V as one
     full prefill), and the superseded blocks are stale for it.
"""
import math

import numpy as np
import pytest
import torch

import oracle
import oracle.chain as ochain
import paper_2608_15241_amd as lk
import workloads
from paper_2608_15241_amd.step import Step, meta_to_device
from gpu_helpers import assert_rel, f64, host_u16, say

pytestmark = pytest.mark.gpu

W = workloads.TINY_DECODE          # hidden 256, 4 x 64 MHA, rank-8 adapters on q and v
AD, C, S = 1, 2000, 2001           # the adapter, its committed and staged versions
CHUNK_BLOCKS = 8                   # 128-token re-prefill chunks
BS = lk.BLOCK_SIZE


def _meta(tables, ctx, n_new, tags, req_version):
    B = len(ctx)
    mb = max(1, max(len(t) for t in tables))
    table = np.zeros((B, mb), dtype=np.int32)
    for b, t in enumerate(tables):
        table[b, :len(t)] = t
    q_indptr = np.zeros(B + 1, dtype=np.int32)
    q_indptr[1:] = np.cumsum(n_new)
    T = int(q_indptr[-1])
    return workloads.generate.Meta(
        ctx_lens=np.asarray(ctx, np.int32), n_new=np.asarray(n_new, np.int32),
        q_indptr=q_indptr, request_adapter=np.full(B, AD, np.int32),
        req_version=np.full(B, req_version, np.int32), block_table=table,
        block_version=np.asarray(tags, np.int32), num_blocks=len(tags), max_blocks=mb,
        stale_entries=np.zeros((0, 2), np.int32), token_adapter=np.full(T, AD, np.int32),
        token_scale=np.full(T, workloads.configs.LORA_SCALE, np.float32))


def _prefill(pool, weights, x, meta):
    st = Step("prefill", x, [weights], meta_to_device(meta, "cuda"), pool, W.hq, W.hkv,
              W.head_dim, residual=False)
    st()
    torch.cuda.synchronize()


def _host_weights(lw):
    return {k: (host_u16(v) if v.dtype == torch.bfloat16 else v.cpu().numpy())
            for k, v in lw.items()}


def test_stale_coverage_prefill_then_publish():
    rng = np.random.default_rng(5)
    D, hkv, hq = W.head_dim, W.hkv, W.hq
    vocab, num_blocks = 512, 320
    emb = workloads.randn_bf16((vocab, W.hidden), 1.0, "cuda", 71)
    committed = workloads.make_layer_weights(W, 0, "cuda", 72)
    trained = workloads.make_layer_weights(W, 0, "cuda", 73)
    staged = dict(committed)
    for k in trained:
        if k[:2] in ("A_", "B_") or k.startswith("ranks_"):
            staged[k] = trained[k]
    pool = workloads.randn_bf16((1, 2, num_blocks, hkv, BS * D), 1.0, "cuda", 74)
    lens = [8, 12, 16, 20, 24, 10, 14, 6]                      # blocks per prefix
    paths = [rng.integers(0, vocab, size=BS * n).astype(np.int32) for n in lens]

    def embed(tokens):
        return emb[torch.as_tensor(np.asarray(tokens, np.int64), device="cuda")].contiguous()

    m = lk.KVManager(num_blocks)
    m.set_committed(AD, C)

    # 1. committed coverage: the eight prefixes as one prefill step under c
    say("committed prefill")
    blocks_c = []
    for p in paths:
        assert len(m.lookup(0, AD, C, p)) == 0
        blocks_c.append(m.alloc(len(p) // BS, C))
    meta = _meta(blocks_c, [len(p) for p in paths], [len(p) for p in paths], m.tags(), C)
    _prefill(pool, committed, embed(np.concatenate(paths)), meta)
    for p, b in zip(paths, blocks_c):
        assert list(m.insert(0, AD, C, p, b)) == [1] * len(b)

    # 2. uneven heat, then the trained version is staged
    for i, p in enumerate(paths):
        for _ in range(i % 4 + 1):
            assert np.array_equal(m.lookup(0, AD, C, p), blocks_c[i])
    m.stage(AD, S)
    plan = m.plan_stale_prefill(AD, 8)
    assert sorted(tot for _, _, tot in plan) == sorted(lens)
    assert all(cov == 0 for _, cov, _ in plan)
    plan_paths = [m.path(node)[1] for node, _, _ in plan]
    for pp in plan_paths:
        assert any(np.array_equal(pp, p) for p in paths)

    # 3. re-prefill in 128-token chunks under s, foreground decode in between
    kpool_c = host_u16(pool[0, 0]).reshape(-1).copy()     # committed K/V as written
    vpool_c = host_u16(pool[0, 1]).reshape(-1).copy()
    rounds = 0
    while True:
        reqs = []
        for pp in plan_paths:
            have = m.lookup(0, AD, S, pp)
            if len(have) < len(pp) // BS:
                reqs.append((pp, have))
        if not reqs:
            break
        rounds += 1
        tables, ctx, n_new, toks, fresh = [], [], [], [], []
        for pp, have in reqs:
            nb = min(CHUNK_BLOCKS, len(pp) // BS - len(have))
            new = m.alloc(nb, S)
            tables.append(np.concatenate([have, new]))
            ctx.append(BS * (len(have) + nb))
            n_new.append(BS * nb)
            toks.append(pp[BS * len(have):BS * (len(have) + nb)])
            fresh.append((pp, len(have), new))
        say("re-prefill round", rounds, "requests", len(reqs))
        meta = _meta(tables, ctx, n_new, m.tags(), S)
        _prefill(pool, staged, embed(np.concatenate(toks)), meta)
        for pp, first, new in fresh:
            assert list(m.insert(0, AD, S, pp, new, first=first)) == [1] * len(new)
        # foreground, bound to c: a staged block in its table is dropped
        q = workloads.randn_bf16((1, hq, D), 1.0, "cuda", 80 + rounds)
        fg = np.concatenate([blocks_c[2], fresh[0][2][:1]])
        L = BS * len(fg)
        md = meta_to_device(_meta([fg], [L], [1], m.tags(), C), "cuda")
        out, lse = lk.local_paged_attn_decode(q, pool[0, 0], pool[0, 1], md.block_table,
                                              md.ctx_lens, md.block_version, md.req_version,
                                              1 / math.sqrt(D), Hkv=hkv)
        torch.cuda.synchronize()
        ro, rl = oracle.paged_attn(host_u16(q), np.array([0, 1], np.int32), hq, hkv, D,
                                   kpool_c, vpool_c, fg[None, :].astype(np.int32),
                                   np.array([L], np.int32), m.tags(),
                                   np.array([C], np.int32), 1 / math.sqrt(D))
        assert_rel(f64(out), ro, "foreground decode during re-prefill")
    assert rounds == max(math.ceil(n / CHUNK_BLOCKS) for n in lens)

    # 4. publication
    assert m.publish(AD) == C
    hs = _host_weights(staged)
    kh = host_u16(pool[0, 0]).reshape(-1)
    vh = host_u16(pool[0, 1]).reshape(-1)
    for i, p in enumerate(paths):
        warmed = m.lookup(0, AD, S, p)
        assert len(warmed) == len(p) // BS
        assert not set(warmed.tolist()) & set(blocks_c[i].tolist())
        # oracle: K/V of the whole prefix from scratch under the staged weights,
        # written into a copy of the pool at the warmed blocks
        L = len(p)
        T = L
        x = host_u16(embed(p))
        ta = np.full(T, AD, np.int32)
        ts = np.full(T, workloads.configs.LORA_SCALE, np.float32)
        kb = oracle.to_bf16(ochain.project(x, hs, "k", ta, ts)).reshape(T, hkv, D)
        vb = oracle.to_bf16(ochain.project(x, hs, "v", ta, ts)).reshape(T, hkv, D)
        ko, vo = kh.copy(), vh.copy()
        oracle.kv_append(ko, vo, hkv, D, warmed[None, :].astype(np.int32),
                         np.array([0, T], np.int32), np.array([L], np.int32), kb, vb)
        q = workloads.randn_bf16((1, hq, D), 1.0, "cuda", 90 + i)
        md = meta_to_device(_meta([warmed], [L], [1], m.tags(), S), "cuda")
        out, lse = lk.local_paged_attn_decode(q, pool[0, 0], pool[0, 1], md.block_table,
                                              md.ctx_lens, md.block_version, md.req_version,
                                              1 / math.sqrt(D), Hkv=hkv)
        torch.cuda.synchronize()
        ro, rl = oracle.paged_attn(host_u16(q), np.array([0, 1], np.int32), hq, hkv, D, ko, vo,
                                   warmed[None, :].astype(np.int32), np.array([L], np.int32),
                                   m.tags(), np.array([S], np.int32), 1 / math.sqrt(D))
        assert_rel(f64(out), ro, "decode after publication, prefix %d" % i)
        # the superseded coverage is stale for a request bound to s
        _, n_stale, _ = oracle.block_version_check(blocks_c[i][None, :].astype(np.int32),
                                                   np.array([L], np.int32), m.tags(),
                                                   np.array([S], np.int32))
        assert n_stale == len(blocks_c[i])
    # and it is the first to go under memory pressure
    freed = m.evict(m.stats()[0] + sum(lens))
    assert sorted(freed) == sorted(np.concatenate(blocks_c).tolist())
