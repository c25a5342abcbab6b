"""Full-size workloads on the GPU against the oracle.

Decode workloads run the whole step (version check, q/k/v projections,
appending attention, output projection; in the 32-layer workload each layer's
output is the next layer's input), for all requests or a seeded sample of them
(requests are independent within a step, so a sample is exact). Each compared
layer is checked stage by stage with the oracle fed the GPU's own bf16 input of
that stage (teacher forcing), and the step's final output against the
oracle's own chain through every layer. The chunked-prefill step runs whole
at full size and is checked the same way on sampled rows. Integer outputs and
appended pools are compared bit for bit.
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
from tests.gpu_helpers import (assert_attn, assert_lse, assert_rel, dev, f64, gather_requests,
                               host_u16, say)

pytestmark = pytest.mark.gpu


def _host_weights(lw):
    out = {}
    for k, v in lw.items():
        out[k] = host_u16(v) if v.dtype == torch.bfloat16 else v.cpu().numpy()
    return out


def _setup(w, seed=0):
    say("generate", w.name)
    meta = workloads.make_meta(w, seed)
    weights = [workloads.make_layer_weights(w, l, "cuda", seed) for l in range(w.n_layers)]
    pool = workloads.make_kv_pool(w, meta, "cuda", seed)
    x = workloads.randn_bf16((meta.T, w.hidden), 1.0, "cuda", seed * 31 + 5)
    torch.cuda.synchronize()
    return meta, weights, pool, x


def _stage_check(l, w, hw, buf, reqs, x_in, pool_l, table, bv, ctx, rv, tok_a, tok_s, qi,
                 gpu_pool_after):
    """Layer l checked stage by stage, each stage of the oracle fed the GPU's
    own bf16 input of that stage (teacher forcing): q, k, v from the layer
    input, the appended pool and attention from the GPU's q, k, v, and the
    output projection from the GPU's attention output."""
    D, T = w.head_dim, len(reqs)
    for name in ("q", "k", "v"):
        ref = ochain.project(x_in, hw, name, tok_a, tok_s)
        assert_rel(f64(buf[name])[reqs], ref, "layer %d %s" % (l, name))
    kh, vh = pool_l[0].copy(), pool_l[1].copy()
    kq = host_u16(buf["k"])[reqs].reshape(T, w.hkv, D)
    vq = host_u16(buf["v"])[reqs].reshape(T, w.hkv, D)
    oracle.kv_append(kh, vh, w.hkv, D, table, qi, ctx, kq, vq)
    assert np.array_equal(gpu_pool_after[0], kh), "layer %d appended K pool differs" % l
    assert np.array_equal(gpu_pool_after[1], vh), "layer %d appended V pool differs" % l
    qq = host_u16(buf["q"])[reqs].reshape(T, w.hq, D)
    ro, rl = oracle.paged_attn(qq, qi, w.hq, w.hkv, D, kh, vh, table, ctx, bv, rv,
                               1.0 / math.sqrt(D))
    assert_attn(f64(buf["o"])[reqs], ro.reshape(T, w.hq * D), "layer %d o" % l, D)
    assert_lse(buf["lse"].cpu().numpy()[reqs], rl, "layer %d lse" % l)
    ref = ochain.project(host_u16(buf["o"])[reqs], hw, "o", tok_a, tok_s)
    assert_rel(f64(buf["y"])[reqs], ref, "layer %d y" % l)


def _decode_chain_check(w, reqs, seed=0, layers_to_compare=None):
    meta, weights, pool, x = _setup(w, seed)
    D = w.head_dim
    reqs = np.asarray(reqs)
    # host copies of the sampled requests' blocks, taken before the GPU step
    pools = []
    for l in range(w.n_layers):
        kh, vh, table, bv = gather_requests(pool[l, 0], pool[l, 1], w.hkv, D,
                                            meta.block_table, meta.ctx_lens,
                                            meta.block_version, reqs)
        pools.append((kh, vh))
    x_host = host_u16(x)[reqs]
    say("GPU step", w.name, "layers", w.n_layers)
    st = Step("decode", x, weights, meta_to_device(meta, "cuda"), pool, w.hq, w.hkv, D,
              residual=False)
    st()
    torch.cuda.synchronize()
    # version check of the step: bit-exact
    pairs, n, valid = st.version_outputs
    ep, en, ev = oracle.block_version_check(meta.block_table, meta.ctx_lens,
                                            meta.block_version, meta.req_version)
    assert int(n.item()) == en
    assert np.array_equal(pairs[:en].cpu().numpy(), ep)
    assert np.array_equal(valid.cpu().numpy(), ev)
    ctx = meta.ctx_lens[reqs]
    rv = meta.req_version[reqs]
    tok_a = meta.token_adapter[reqs]
    tok_s = meta.token_scale[reqs]
    qi = np.arange(len(reqs) + 1, dtype=np.int32)
    compare = set(range(w.n_layers)) if layers_to_compare is None else set(layers_to_compare)
    # per layer, stage by stage, with the GPU's own inputs of each stage
    for l in sorted(compare):
        say("stage check", w.name, "layer", l)
        after = gather_requests(pool[l, 0], pool[l, 1], w.hkv, D, meta.block_table,
                                meta.ctx_lens, meta.block_version, reqs)[:2]
        _stage_check(l, w, _host_weights(weights[l]), st.buffers[l], reqs,
                     host_u16(st.buffers[l]["x"])[reqs], pools[l], table, bv, ctx, rv, tok_a,
                     tok_s, qi, after)
    # the oracle's own chain through every layer, against the step's output
    say("oracle chain", w.name, "requests", len(reqs))
    xo = x_host
    for l in range(w.n_layers):
        lw = _host_weights(weights[l])
        kh, vh = pools[l]
        xo, _ = ochain.layer(xo, lw, kh, vh, w.hq, w.hkv, D, table, qi, ctx, bv, rv, tok_a,
                             tok_s, residual=False)
    assert_rel(f64(st.out)[reqs], oracle.bf16_to_f64(xo), "final output")
    del st, pool, weights
    torch.cuda.empty_cache()


def test_tiny_decode_step():
    w = workloads.TINY_DECODE
    _decode_chain_check(w, np.arange(w.batch))


def test_decode_7b_step():
    w = workloads.DECODE_7B
    _decode_chain_check(w, np.arange(w.batch))


def test_gqa_skew_step():
    w = workloads.GQA_SKEW
    _decode_chain_check(w, np.arange(w.batch))


def test_churn_32_layer_step_sampled():
    w = workloads.CHURN_32L
    rng = np.random.default_rng(2024)
    reqs = np.sort(rng.choice(w.batch, size=4, replace=False))
    _decode_chain_check(w, reqs, layers_to_compare=(0, 1, 15, 31))


def test_prefill_7b_sampled():
    w = workloads.PREFILL_7B
    meta = workloads.make_meta(w, 0)
    D, T = w.head_dim, meta.T
    rng = np.random.default_rng(7)
    rows = np.unique(np.concatenate([meta.q_indptr[:-1], meta.q_indptr[1:] - 1,
                                     rng.choice(T, size=40, replace=False)]))
    # --- projections at full size (q and o shapes), sampled rows
    lw = workloads.make_layer_weights(w, 0, "cuda", 0)
    x = workloads.randn_bf16((T, w.hidden), 1.0, "cuda", 11)
    md = meta_to_device(meta, "cuda")
    for name in ("q", "o"):
        say("prefill projection", name)
        y = lk.local_lora_linear(x, lw["W_" + name], lw["A_" + name], lw["B_" + name],
                                 lw["ranks_" + name], md.token_adapter, md.token_scale)
        torch.cuda.synchronize()
        hw = _host_weights(lw)
        ref = ochain.project(host_u16(x)[rows], hw, name, meta.token_adapter[rows],
                             meta.token_scale[rows])
        assert_rel(f64(y)[rows], ref, "proj " + name)
    # --- appending causal attention at full size, sampled query rows
    pool = workloads.make_kv_pool(w, meta, "cuda", 0)
    q = workloads.randn_bf16((T, w.hq, D), 1.0, "cuda", 21)
    kn = workloads.randn_bf16((T, w.hkv, D), 1.0, "cuda", 22)
    vn = workloads.randn_bf16((T, w.hkv, D), 1.0, "cuda", 23)
    kh, vh = host_u16(pool[0, 0]).reshape(-1), host_u16(pool[0, 1]).reshape(-1)
    say("prefill attention")
    out, lse = lk.local_paged_attn_prefill(q, md.q_indptr, pool[0, 0], pool[0, 1],
                                           md.block_table, md.ctx_lens, md.block_version,
                                           md.req_version, 1 / math.sqrt(D), k_new=kn,
                                           v_new=vn, Hkv=w.hkv)
    torch.cuda.synchronize()
    oracle.kv_append(kh, vh, w.hkv, D, meta.block_table, meta.q_indptr, meta.ctx_lens,
                     host_u16(kn), host_u16(vn))
    assert np.array_equal(host_u16(pool[0, 0]).reshape(-1), kh)
    assert np.array_equal(host_u16(pool[0, 1]).reshape(-1), vh)
    # row r of request b at position P_b + i attends over positions <= P_b + i:
    # the one-row problem with context P_b + i + 1 (a decode of that row)
    b_of = np.searchsorted(meta.q_indptr, rows, side="right") - 1
    pos = meta.ctx_lens[b_of] - meta.n_new[b_of] + (rows - meta.q_indptr[b_of])
    ro, rl = oracle.paged_attn(host_u16(q)[rows], np.arange(len(rows) + 1, dtype=np.int32),
                               w.hq, w.hkv, D, kh, vh, meta.block_table[b_of],
                               (pos + 1).astype(np.int32), meta.block_version,
                               meta.req_version[b_of], 1 / math.sqrt(D))
    assert_attn(f64(out)[rows], ro, "prefill out", D)
    assert_lse(lse.cpu().numpy()[rows], rl, "prefill lse")
    del pool
    torch.cuda.empty_cache()


def test_prefill_7b_step():
    # The whole prefill step as the benchmark runs it (version check; q, k, v
    # as one grouped call at T = 2048, K = 4096; appending causal attention;
    # o), checked stage by stage on sampled rows with the oracle fed the
    # GPU's own input of each stage, and the appended pool bit for bit.
    w = workloads.PREFILL_7B
    meta, weights, pool, x = _setup(w, 5)
    D, T = w.head_dim, meta.T
    rng = np.random.default_rng(8)
    starts = meta.q_indptr[:-1]
    rows = np.unique(np.concatenate([starts, meta.q_indptr[1:] - 1, starts + 127, starts + 128,
                                     rng.choice(T, size=32, replace=False)]))
    kh, vh = host_u16(pool[0, 0]).reshape(-1), host_u16(pool[0, 1]).reshape(-1)
    say("GPU prefill step", w.name)
    st = Step("prefill", x, weights, meta_to_device(meta, "cuda"), pool, w.hq, w.hkv, D,
              residual=False)
    st()
    torch.cuda.synchronize()
    pairs, n, valid = st.version_outputs
    ep, en, ev = oracle.block_version_check(meta.block_table, meta.ctx_lens,
                                            meta.block_version, meta.req_version)
    assert int(n.item()) == en and np.array_equal(valid.cpu().numpy(), ev)
    buf = st.buffers[0]
    hw = _host_weights(weights[0])
    tok_a, tok_s = meta.token_adapter[rows], meta.token_scale[rows]
    xh = host_u16(x)[rows]
    for name in ("q", "k", "v"):
        say("prefill step stage", name)
        ref = ochain.project(xh, hw, name, tok_a, tok_s)
        assert_rel(f64(buf[name])[rows], ref, "step " + name)
    say("prefill step append + attention")
    oracle.kv_append(kh, vh, w.hkv, D, meta.block_table, meta.q_indptr, meta.ctx_lens,
                     host_u16(buf["k"]).reshape(T, w.hkv, D),
                     host_u16(buf["v"]).reshape(T, w.hkv, D))
    assert np.array_equal(host_u16(pool[0, 0]).reshape(-1), kh), "appended K pool differs"
    assert np.array_equal(host_u16(pool[0, 1]).reshape(-1), vh), "appended V pool differs"
    b_of = np.searchsorted(meta.q_indptr, rows, side="right") - 1
    pos = meta.ctx_lens[b_of] - meta.n_new[b_of] + (rows - meta.q_indptr[b_of])
    qh = host_u16(buf["q"]).reshape(T, w.hq, D)[rows]
    ro, rl = oracle.paged_attn(qh, np.arange(len(rows) + 1, dtype=np.int32), w.hq, w.hkv, D,
                               kh, vh, meta.block_table[b_of], (pos + 1).astype(np.int32),
                               meta.block_version, meta.req_version[b_of], 1 / math.sqrt(D))
    assert_attn(f64(buf["o"])[rows], ro.reshape(len(rows), w.hq * D), "step o", D)
    assert_lse(buf["lse"].cpu().numpy()[rows], rl, "step lse")
    say("prefill step stage y")
    ref = ochain.project(host_u16(buf["o"])[rows], hw, "o", tok_a, tok_s)
    assert_rel(f64(buf["y"])[rows], ref, "step y")
    del st, pool, weights
    torch.cuda.empty_cache()


def test_step_graph_replays_match_eager():
    # The whole decode step captured into a HIP graph: every replay, with
    # eager work and synchronisations in between, equals the eager step.
    say("step graph")
    w = workloads.GQA_SKEW
    meta, weights, pool, x = _setup(w, 3)
    st = Step("decode", x, weights, meta_to_device(meta, "cuda"), pool, w.hq, w.hkv,
              w.head_dim, residual=False)
    st()
    torch.cuda.synchronize()
    ref = {k: v.clone() for k, v in st.buffers[0].items()}
    ref_pairs = [t.clone() for t in st.version_outputs]
    g = st.capture()
    for rep in range(4):
        for k in ("q", "o", "y", "lse"):
            st.buffers[0][k].fill_(float("nan") if k == "lse" else 7.0)
        st.version_outputs[2].fill_(-1)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for k, v in ref.items():
            assert torch.equal(st.buffers[0][k].view(torch.int16) if v.dtype == torch.bfloat16
                               else st.buffers[0][k], v.view(torch.int16)
                               if v.dtype == torch.bfloat16 else v), (rep, k)
        for a_, b_ in zip(st.version_outputs, ref_pairs):
            assert torch.equal(a_, b_), rep
    del st, pool, weights
    torch.cuda.empty_cache()
