#!/usr/bin/env python3
"""Benchmark of the mixed-adapter LoRA decode step on one MI355X.

One step = one pass of the whole path over one batch: the version check, the
q/k/v LoRA projections, the appending, version-masked paged decode attention,
and the output LoRA projection, for the 7B-class single-layer decode workload
(hidden 4096, 32x128 MHA, batch 32, context U[256,4096], 8 rank-16 adapters on
q/k/v/o). Inputs are seeded synthetic tensors already resident in HBM. Two
independent input sets (weights, KV pools, activations) alternate between
steps, so that the last-level cache cannot serve one step's weights to the
next.

Prints ONE JSON line. `value` is decode tokens/s. `roofline` is for the
dominant kernel (decode attention), timed with HIP events around its launches
inside the timed region. `prefill` reports the matrix-core utilisation of the
LoRA-fused projections of the chunked-prefill workload, timed the same way.
`cpu_baseline` is the CPU oracle timed on this host on the same workload.

`--workload gqa_skew_b64 | churn_32l_b128 | tiny_decode` times the decode step
of another workload the same way (without the prefill and CPU legs; the
32-layer one with a single input set, since its KV pool is 146 GB).
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

import numpy as np

HBM_PEAK_GBPS = 8000.0          # MI355X HBM3E
BF16_PEAK_TFLOPS = 2500.0       # MI355X dense bf16 matrix cores


def say(*a):
    """Progress on stderr (the JSON line alone goes to stdout)."""
    print("bench:", *a, file=sys.stderr, flush=True)


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=200)
    p.add_argument("--warmup", type=int, default=20)
    p.add_argument("--sets", type=int, default=2, help="input sets rotated across steps")
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--no-prefill", action="store_true")
    p.add_argument("--cpu-budget-s", type=float, default=15.0)
    p.add_argument("--workload", default="decode_7b_mha_b32",
                   choices=("tiny_decode", "decode_7b_mha_b32", "gqa_skew_b64",
                            "churn_32l_b128"),
                   help="decode workload of the step; prefill and cpu_baseline are reported "
                        "with the default one only. The 32-layer workload uses one input set "
                        "(its KV pool is 146 GB)")
    p.add_argument("--traffic-probe", action="store_true",
                   help="only run, eagerly, a 256 MiB device copy (the calibration of the "
                        "HBM byte counters) and 5 decode attention launches of the workload; "
                        "for rocprofv3 --pmc runs")
    return p.parse_args()


TRAFFIC_FILE = os.path.join(os.path.dirname(os.path.abspath(__file__)), "profiles",
                            "decode_attn_traffic_decode_7b_mha_b32.md")
DECODE_SOURCES = ("paper_2608_15241_amd/csrc/paged_attn_decode.hip",
                  "paper_2608_15241_amd/csrc/common.hpp")


def decode_source_hash():
    """sha256 over the sources of the decode attention kernels."""
    import hashlib
    h = hashlib.sha256()
    root = os.path.dirname(os.path.abspath(__file__))
    for rel in DECODE_SOURCES:
        with open(os.path.join(root, rel), "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def measured_traffic():
    """HBM bytes per decode attention launch from the committed counter summary,
    or None when it is missing or was taken on other kernel sources."""
    try:
        text = open(TRAFFIC_FILE).read()
    except OSError:
        return None
    vals = {}
    for line in text.splitlines():
        if line.startswith("- ") and ": " in line:
            k, v = line[2:].split(": ", 1)
            vals[k.strip()] = v.strip().strip("`")
    if vals.get("source_sha256") != decode_source_hash():
        return None
    try:
        return int(vals["traffic_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


def decode_bytes(w, meta):
    """Algorithmic HBM bytes of one layer's attention launch and of one decode
    step over all layers (each layer reads its own KV pool and weights)."""
    D, hq, hkv, H = w.head_dim, w.hq, w.hkv, w.hidden
    B = meta.B
    nb = (meta.ctx_lens.astype(np.int64) + 15) // 16
    # valid KV tokens: live tokens of non-stale blocks (version check rule)
    valid_tokens = 0
    for b in range(B):
        L = int(meta.ctx_lens[b])
        tags = meta.block_version[meta.block_table[b, :nb[b]]]
        live = np.minimum(16, L - 16 * np.arange(nb[b]))
        valid_tokens += int(live[tags == meta.req_version[b]].sum())
    kv = valid_tokens * hkv * D * 2 * 2
    attn = (kv + B * hq * D * 2 * 2 + B * hq * 4      # q, out, lse
            + B * hkv * D * 2 * 2 * 2                  # k_new/v_new read + append write
            + int(nb.sum()) * 8)                       # table entry + tag
    present = np.unique(meta.token_adapter[meta.token_adapter >= 0])
    proj = 0
    for name in ("q", "k", "v", "o"):
        N, K = w.proj_shape(name)
        proj += N * K * 2 + B * (K + N) * 2
        if name in w.lora_targets:
            for a in present:
                r = w.ranks[a]
                proj += r * K * 2 + N * r * 2
    vc = int(nb.sum()) * 8 + B * 4 * 3
    return attn, w.n_layers * (attn + proj) + vc, valid_tokens


def context_text(w):
    kind = w.ctx[0]
    if kind == "fixed":
        return "fixed %s" % (list(w.ctx[1]),)
    return "%s[%d,%d]" % ({"uniform": "U", "loguniform": "logU"}[kind], w.ctx[1], w.ctx[2])


def adapters_text(w):
    ranks = sorted(set(w.ranks))
    r = "rank %d" % ranks[0] if len(ranks) == 1 else "ranks %s" % ranks
    return "%d x %s on %s (%s)" % (w.n_adapters, r, "/".join(w.lora_targets), w.assignment)


def prefill_gemm_flops(w, meta):
    T = meta.T
    f = 0
    for name in ("q", "k", "v", "o"):
        N, K = w.proj_shape(name)
        f += 2 * T * K * N
        if name in w.lora_targets:
            r = w.r_max
            f += 2 * T * r * (K + N)
    return f


def main():
    args = parse()
    if args.gpus != 1:
        print("bench.py: the library runs on one GPU; --gpus %d is not supported "
              "(sharding across GPUs is not implemented)" % args.gpus,
              file=sys.stderr)
        sys.exit(2)
    import torch
    import workloads
    import paper_2608_15241_amd as lk
    from paper_2608_15241_amd.step import Step, meta_to_device

    lk.load_library()
    dev = "cuda:0"
    torch.cuda.set_device(0)
    w = workloads.BY_NAME[args.workload]
    primary = w.name == workloads.DECODE_7B.name
    meta = workloads.make_meta(w, seed=0)
    md = meta_to_device(meta, dev)
    if args.traffic_probe:
        traffic_probe(torch, workloads, w, meta, md, dev)
        return
    n_sets = args.sets if w.n_layers == 1 else 1
    sets = []
    for s in range(n_sets):
        say("input set", s, "of", w.name)
        weights = [workloads.make_layer_weights(w, l, dev, seed=100 + s)
                   for l in range(w.n_layers)]
        pool = workloads.make_kv_pool(w, meta, dev, seed=100 + s)
        x = workloads.randn_bf16((meta.T, w.hidden), 1.0, dev, seed=200 + s)
        st = Step("decode", x, weights, md, pool, w.hq, w.hkv, w.head_dim, residual=False)
        sets.append((st, pool, weights, x))
    torch.cuda.synchronize()

    stream = torch.cuda.current_stream()
    # warmup (eager: sets kernel attributes on first launch), then one HIP
    # graph per input set; a step is one graph replay
    for i in range(max(args.warmup, len(sets))):
        sets[i % len(sets)][0]()
    torch.cuda.synchronize()
    graphs = [st.capture() for st, *_ in sets]
    for i in range(args.warmup):
        graphs[i % len(graphs)].replay()
    torch.cuda.synchronize()

    say("timed steps")
    K = args.steps
    t_start = torch.cuda.Event(enable_timing=True)
    t_end = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t_start.record(stream)
    for i in range(K):
        graphs[i % len(graphs)].replay()
    t_end.record(stream)
    torch.cuda.synchronize()
    total_ms = t_start.elapsed_time(t_end)
    ms_per_step = total_ms / K

    # the dominant kernel (decode attention), timed with HIP events around
    # each of its launches (every layer) in K eager steps on the same stream
    ev_a = [torch.cuda.Event(enable_timing=True) for _ in range(K * w.n_layers)]
    ev_b = [torch.cuda.Event(enable_timing=True) for _ in range(K * w.n_layers)]
    e_start = torch.cuda.Event(enable_timing=True)
    e_end = torch.cuda.Event(enable_timing=True)
    e_start.record(stream)
    for i in range(K):
        st = sets[i % len(sets)][0]
        st.version_check()
        for l, lc in enumerate(st.layer_calls):
            for c in lc["in"]:
                c()
            ev_a[i * w.n_layers + l].record(stream)
            lc["attn"]()
            ev_b[i * w.n_layers + l].record(stream)
            lc["o"]()
    e_end.record(stream)
    torch.cuda.synchronize()
    eager_ms = e_start.elapsed_time(e_end) / K
    attn_ms = float(np.mean([a.elapsed_time(b) for a, b in zip(ev_a, ev_b)]))

    attn_bytes, step_bytes, valid_tokens = decode_bytes(w, meta)
    tokens_per_s = meta.B / (ms_per_step / 1e3)
    attn_gbps = attn_bytes / (attn_ms / 1e3) / 1e9
    step_gbps = step_bytes / (ms_per_step / 1e3) / 1e9

    result = {
        "metric": "decode tokens/s + achieved HBM GB/s (% peak); prefill LoRA-GEMM MFMA util",
        "value": round(tokens_per_s, 1),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": w.name, "layers": w.n_layers, "hidden": w.hidden,
                   "heads": "%dq/%dkv x %d" % (w.hq, w.hkv, w.head_dim), "batch": meta.B,
                   "context": context_text(w), "sum_context": int(meta.ctx_lens.sum()),
                   "valid_kv_tokens": valid_tokens, "stale_frac": w.stale_frac,
                   "adapters": adapters_text(w), "input_sets": n_sets},
        "roofline": {"kernel": "local_paged_attn_decode", "bound": "hbm",
                     "achieved": round(attn_gbps, 1), "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                     "frac": round(attn_gbps / HBM_PEAK_GBPS, 4),
                     "traffic": measured_traffic() if primary else None,
                     "bytes_per_launch": attn_bytes, "ms_per_launch": round(attn_ms, 5)},
        "hbm_step": {"bytes_per_step": step_bytes, "achieved": round(step_gbps, 1),
                     "unit": "GB/s", "frac": round(step_gbps / HBM_PEAK_GBPS, 4)},
        "step_launch": {"mode": "hip_graph_replay", "eager_ms_per_step": round(eager_ms, 5)},
    }

    if primary and not args.no_prefill:
        say("prefill projections")
        result["prefill"] = bench_prefill(torch, workloads, lk, dev)
        say("prefill attention")
        result["prefill_attn"] = bench_prefill_attn(torch, workloads, lk, dev)
        say("stale-coverage prefill")
        result["reprefill"] = bench_reprefill(torch, workloads, lk, dev)
        say("lora backward")
        result["lora_grad"] = bench_lora_grad(torch, workloads, lk, dev)

    if primary and not args.no_cpu_baseline:
        say("cpu baseline")
        result["cpu_baseline"] = cpu_baseline(torch, workloads, w, meta, sets[0], args)

    del sets
    print(json.dumps(result), flush=True)


def traffic_probe(torch, workloads, w, meta, md, dev):
    """A plain copy of known size, then decode attention launches, eagerly."""
    from paper_2608_15241_amd.step import Step
    weights = [workloads.make_layer_weights(w, 0, dev, seed=100)]
    pool = workloads.make_kv_pool(w, meta, dev, seed=100)
    x = workloads.randn_bf16((meta.T, w.hidden), 1.0, dev, seed=200)
    st = Step("decode", x, weights, md, pool, w.hq, w.hkv, w.head_dim, residual=False)
    st()
    torch.cuda.synchronize()
    n = 256 << 20
    src = torch.ones(n // 2, dtype=torch.bfloat16, device=dev)
    dst = torch.empty_like(src)
    for _ in range(3):
        torch.mul(src, 1.0, out=dst)       # elementwise kernel: reads n bytes, writes n
    torch.cuda.synchronize()
    for _ in range(5):
        st.layer_calls[0]["attn"]()
    torch.cuda.synchronize()
    attn_bytes, _, _ = decode_bytes(w, meta)
    print(json.dumps({"traffic_probe": {"copy_read_bytes": n, "copy_write_bytes": n,
                                        "copy_kernel": "torch.mul(src, 1.0, out=dst), bf16",
                                        "attn_launches": 5,
                                        "attn_algorithmic_bytes": attn_bytes,
                                        "decode_source_sha256": decode_source_hash()}}),
          flush=True)


def bench_prefill(torch, workloads, lk, dev, reps=20):
    """Matrix-core utilisation of the 4 LoRA-fused projections (prefill workload)."""
    from paper_2608_15241_amd.step import meta_to_device
    w = workloads.PREFILL_7B
    meta = workloads.make_meta(w, seed=0)
    md = meta_to_device(meta, dev)
    # the projections as a decode or prefill step issues them: q, k, v of one x
    # as one grouped call, then o
    calls = []
    for s in range(2):
        lw = workloads.make_layer_weights(w, 0, dev, seed=300 + s)
        x = workloads.randn_bf16((meta.T, w.hidden), 1.0, dev, seed=400 + s)
        ws = lk.Workspace(dev)
        qkv = ("q", "k", "v")
        outs = [torch.empty((meta.T, w.proj_shape(n)[0]), dtype=torch.bfloat16, device=dev)
                for n in qkv]
        calls.append(lk.prepare_lora_linear_grouped(
            x, [lw["W_" + n] for n in qkv], [lw["A_" + n] for n in qkv],
            [lw["B_" + n] for n in qkv], [lw["ranks_" + n] for n in qkv],
            md.token_adapter, md.token_scale, outs=outs, workspace=ws))
        N, K = w.proj_shape("o")
        inp = torch.empty((meta.T, K), dtype=torch.bfloat16, device=dev).normal_()
        out = torch.empty((meta.T, N), dtype=torch.bfloat16, device=dev)
        calls.append(lk.prepare_lora_linear(inp, lw["W_o"], lw["A_o"], lw["B_o"], lw["ranks_o"],
                                            md.token_adapter, md.token_scale, out=out,
                                            workspace=ws))
    per_set = 2
    for c in calls:
        c()
    torch.cuda.synchronize()
    graphs = []
    for sidx in range(2):
        g = torch.cuda.CUDAGraph()
        s = torch.cuda.Stream()
        s.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(s):
            with torch.cuda.graph(g, stream=s):
                for c in calls[sidx * per_set:(sidx + 1) * per_set]:
                    c()
        torch.cuda.current_stream().wait_stream(s)
        graphs.append(g)
    for g in graphs:
        g.replay()
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()
    a = torch.cuda.Event(enable_timing=True)
    b = torch.cuda.Event(enable_timing=True)
    a.record(stream)
    for r in range(reps):
        graphs[r % 2].replay()
    b.record(stream)
    torch.cuda.synchronize()
    ms = a.elapsed_time(b) / reps
    flops = prefill_gemm_flops(w, meta)
    tflops = flops / (ms / 1e3) / 1e12
    return {"workload": w.name,
            "kernel": "local_lora_linear_grouped (q,k,v) + local_lora_linear (o), T=%d" % meta.T,
            "bound": "mfma", "flops_per_step": flops, "ms_per_step": round(ms, 5),
            "achieved": round(tflops, 1), "peak": BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
            "frac": round(tflops / BF16_PEAK_TFLOPS, 4)}


def prefill_attn_flops(w, meta):
    """2 * 2 * D flop per (query, key) pair attended: query i of request b at
    position P_b + i sees keys 0 .. P_b + i, for every query head."""
    pairs = 0
    for b in range(meta.B):
        n = int(meta.n_new[b])
        P = int(meta.ctx_lens[b]) - n
        pairs += n * P + n * (n + 1) // 2
    return 4 * w.head_dim * w.hq * pairs


def bench_prefill_attn(torch, workloads, lk, dev, reps=20):
    """Matrix-core utilisation of the appending, version-masked paged prefill
    attention of the prefill workload (4 chunks of 512 on prefixes
    {0, 512, 1024, 2048}), timed as graph replays over two input sets."""
    from paper_2608_15241_amd.step import meta_to_device
    w = workloads.PREFILL_7B
    meta = workloads.make_meta(w, seed=0)
    md = meta_to_device(meta, dev)
    D, T = w.head_dim, meta.T
    calls, keep = [], []
    for s in range(2):
        pool = workloads.make_kv_pool(w, meta, dev, seed=600 + s)
        q = workloads.randn_bf16((T, w.hq, D), 1.0, dev, seed=610 + s)
        kn = workloads.randn_bf16((T, w.hkv, D), 1.0, dev, seed=620 + s)
        vn = workloads.randn_bf16((T, w.hkv, D), 1.0, dev, seed=630 + s)
        keep += [pool, q, kn, vn]
        calls.append(lk.prepare_paged_attn_prefill(
            q, md.q_indptr, pool[0, 0], pool[0, 1], md.block_table, md.ctx_lens,
            md.block_version, md.req_version, 1 / math.sqrt(D), k_new=kn, v_new=vn, Hkv=w.hkv))
    for c in calls:
        c()
    torch.cuda.synchronize()
    graphs = []
    for c in calls:
        g = torch.cuda.CUDAGraph()
        st = torch.cuda.Stream()
        st.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(st):
            with torch.cuda.graph(g, stream=st):
                c()
        torch.cuda.current_stream().wait_stream(st)
        graphs.append(g)
    for g in graphs:
        g.replay()
    torch.cuda.synchronize()
    a = torch.cuda.Event(enable_timing=True)
    b = torch.cuda.Event(enable_timing=True)
    a.record()
    for r in range(reps):
        graphs[r % 2].replay()
    b.record()
    torch.cuda.synchronize()
    ms = a.elapsed_time(b) / reps
    flops = prefill_attn_flops(w, meta)
    tflops = flops / (ms / 1e3) / 1e12
    return {"workload": w.name, "kernel": "local_paged_attn_prefill (append + attention)",
            "bound": "mfma", "flops_per_call": flops, "ms_per_call": round(ms, 5),
            "achieved": round(tflops, 1), "peak": BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
            "frac": round(tflops / BF16_PEAK_TFLOPS, 4)}


def bench_reprefill(torch, workloads, lk, dev, n_prefix=8, prefix_blocks=64, chunk_blocks=8):
    """Stale-coverage prefill (§5.3) at the prefill workload's shapes: eight hot
    prefixes of 1024 tokens, recorded under the committed version, re-prefilled
    under the staged version in 128-token chunks (one prefill step per round,
    every prefix advancing one chunk), the KV manager planning, matching,
    allocating and recording on the host between rounds. Reports the warm-up's
    throughput, the matrix-core utilisation of its projections, and the host
    time of the manager."""
    from paper_2608_15241_amd.step import Step, meta_to_device
    w = workloads.PREFILL_7B
    D, BS = w.head_dim, lk.BLOCK_SIZE
    AD, C, S = 0, workloads.adapter_version(0), workloads.adapter_version(0) + 1
    rng = np.random.default_rng(17)
    num_blocks = 2 * n_prefix * prefix_blocks
    lw = workloads.make_layer_weights(w, 0, dev, seed=500)
    pool = workloads.randn_bf16((1, 2, num_blocks, w.hkv, BS * D), 1.0, dev, seed=501)
    emb = workloads.randn_bf16((4096, w.hidden), 1.0, dev, seed=502)
    paths = [rng.integers(0, 4096, size=BS * prefix_blocks).astype(np.int32)
             for _ in range(n_prefix)]
    m = lk.KVManager(num_blocks)
    m.set_committed(AD, C)
    for p in paths:  # committed coverage (its KV content does not matter here)
        m.insert(0, AD, C, p, m.alloc(prefix_blocks, C))
        m.lookup(0, AD, C, p)
    m.stage(AD, S)

    def round_inputs():
        t0 = time.perf_counter()
        plan = m.plan_stale_prefill(AD, n_prefix)
        tables, ctx, n_new, toks, fresh = [], [], [], [], []
        for node, cov, tot in plan:
            pp = m.path(node)[1]
            have = m.lookup(0, AD, S, pp)
            nb = min(chunk_blocks, tot - len(have))
            new = m.alloc(nb, S)
            tables.append(np.concatenate([have, new]))
            ctx.append(BS * (len(have) + nb))
            n_new.append(BS * nb)
            toks.append(pp[BS * len(have):BS * (len(have) + nb)])
            fresh.append((pp, len(have), new))
        host = time.perf_counter() - t0
        if not plan:
            return None, host
        B = len(plan)
        table = np.zeros((B, max(len(t) for t in tables)), dtype=np.int32)
        for b, t in enumerate(tables):
            table[b, :len(t)] = t
        q_indptr = np.zeros(B + 1, dtype=np.int32)
        q_indptr[1:] = np.cumsum(n_new)
        T = int(q_indptr[-1])
        meta = workloads.Meta(
            ctx_lens=np.asarray(ctx, np.int32), n_new=np.asarray(n_new, np.int32),
            q_indptr=q_indptr, request_adapter=np.full(B, AD, np.int32),
            req_version=np.full(B, S, np.int32), block_table=table,
            block_version=m.tags(), num_blocks=num_blocks, max_blocks=table.shape[1],
            stale_entries=np.zeros((0, 2), np.int32), token_adapter=np.full(T, AD, np.int32),
            token_scale=np.full(T, workloads.configs.LORA_SCALE, np.float32))
        x = emb[torch.as_tensor(np.concatenate(toks).astype(np.int64), device=dev)].contiguous()
        st = Step("prefill", x, [lw], meta_to_device(meta, dev), pool, w.hq, w.hkv, D,
                  residual=False)
        return (st, fresh, T, meta), host

    rounds, tokens, host_s, gpu_ms, flops = 0, 0, 0.0, 0.0, 0
    ev_a, ev_b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    while True:
        r, h = round_inputs()
        host_s += h
        if r is None:
            break
        st, fresh, T, meta = r
        st()  # sets kernel attributes; then the round as one HIP graph, replayed
        torch.cuda.synchronize()  # (it only rewrites the same slots)
        g = st.capture()
        g.replay()
        torch.cuda.synchronize()
        ev_a.record()
        g.replay()
        ev_b.record()
        torch.cuda.synchronize()
        gpu_ms += ev_a.elapsed_time(ev_b)
        del g
        t0 = time.perf_counter()
        for pp, first, new in fresh:
            m.insert(0, AD, S, pp, new, first=first)
        host_s += time.perf_counter() - t0
        rounds += 1
        tokens += T
        flops += prefill_gemm_flops(w, meta)
    m.publish(AD)
    tflops = flops / (gpu_ms / 1e3) / 1e12
    return {"workload": "reprefill_7b_8x1024", "prefixes": n_prefix,
            "prefix_tokens": BS * prefix_blocks, "chunk_tokens": BS * chunk_blocks,
            "rounds": rounds, "tokens": tokens, "gpu_ms": round(gpu_ms, 4),
            "tokens_per_s": round(tokens / (gpu_ms / 1e3), 1),
            "projection_flops": flops, "step_tflops": round(tflops, 1),
            "step_frac_of_mfma_peak": round(tflops / BF16_PEAK_TFLOPS, 4),
            "host_manager_us_per_round": round(host_s / max(rounds, 1) * 1e6, 1),
            "note": "each round is one whole prefill step (version check, q/k/v, appending "
                    "causal attention, o) timed as a HIP graph replay; step_tflops counts the "
                    "projections' flops only"}


def lora_grad_bytes(w, T):
    """Algorithmic HBM bytes of the adapter gradients of a layer's projections:
    the q/k/v input read once for the three (they share it) and the o input
    once, every dy once (bf16), the token routing once per call (int32 index
    and fp32 scale per token), every adapter's A and B read once (bf16) and
    dA, dB written once (fp32)."""
    total = 0
    for proj in ("q", "k", "v", "o"):
        N, K = w.proj_shape(proj)
        total += 2 * T * N + w.n_adapters * w.r_max * (K + N) * (2 + 4)
    total += 2 * T * w.proj_shape("q")[1] + 2 * T * w.proj_shape("o")[1]  # the two inputs
    total += 2 * 8 * T  # routing, once per call
    return total


def lora_grad_input_flops(w, T):
    """2 T N K per projection for dy W, plus 2 T r (N + K) for the adapter term."""
    total = 0
    for proj in ("q", "k", "v", "o"):
        N, K = w.proj_shape(proj)
        total += 2 * T * N * K + 2 * T * w.r_max * (N + K)
    return total


def bench_lora_grad(torch, workloads, lk, dev, reps=20):
    """The LoRA backward of one training chunk at the prefill workload's shapes
    (2048 tokens over 4 rank-16 adapters, q/k/v/o of a 4096-wide layer): the
    adapter gradients (HBM-bound; q, k and v share their input and run as one
    grouped call) and the input gradient (matrix-core bound) of the four
    projections, each timed as graph replays over two input sets."""
    from paper_2608_15241_amd.step import meta_to_device
    w = workloads.PREFILL_7B
    meta = workloads.make_meta(w, seed=0)
    md = meta_to_device(meta, dev)
    T = meta.T
    grads, inputs, keep = [], [], []
    for s in range(2):
        lw = workloads.make_layer_weights(w, 0, dev, seed=700 + s)
        ws = lk.Workspace(dev)
        g_calls, i_calls = [], []
        route = (md.token_adapter, md.token_scale)
        # q, k, v share their input: one grouped call; o has its own
        x_in = workloads.randn_bf16((T, w.proj_shape("q")[1]), 1.0, dev, seed=710 + 10 * s)
        x_o = workloads.randn_bf16((T, w.proj_shape("o")[1]), 1.0, dev, seed=711 + 10 * s)
        dys = {}
        for i, proj in enumerate(("q", "k", "v", "o")):
            N, K = w.proj_shape(proj)
            dys[proj] = workloads.randn_bf16((T, N), 1.0, dev, seed=750 + 10 * s + i)
            Wt = lw["W_" + proj].t().contiguous()
            keep += [dys[proj], Wt]
            i_calls.append(lk.prepare_lora_grad_input(
                dys[proj], Wt, lw["A_" + proj], lw["B_" + proj], lw["ranks_" + proj], *route,
                workspace=ws))
        qkv = ("q", "k", "v")
        g_calls.append(lk.prepare_lora_grad_grouped(
            x_in, [dys[n] for n in qkv], [lw["A_" + n] for n in qkv], [lw["B_" + n] for n in qkv],
            [lw["ranks_" + n] for n in qkv], *route, workspace=ws))
        g_calls.append(lk.prepare_lora_grad(x_o, dys["o"], lw["A_o"], lw["B_o"], lw["ranks_o"],
                                            *route, workspace=ws))
        keep += [lw, x_in, x_o]
        grads.append(g_calls)
        inputs.append(i_calls)

    def graphs_of(sets):
        out = []
        for calls in sets:
            for c in calls:
                c()
            torch.cuda.synchronize()
            g = torch.cuda.CUDAGraph()
            st = torch.cuda.Stream()
            st.wait_stream(torch.cuda.current_stream())
            with torch.cuda.stream(st):
                with torch.cuda.graph(g, stream=st):
                    for c in calls:
                        c()
            torch.cuda.current_stream().wait_stream(st)
            out.append(g)
        return out

    def time_graphs(gs):
        for g in gs:
            g.replay()
        torch.cuda.synchronize()
        a = torch.cuda.Event(enable_timing=True)
        b = torch.cuda.Event(enable_timing=True)
        a.record()
        for r in range(reps):
            gs[r % 2].replay()
        b.record()
        torch.cuda.synchronize()
        return a.elapsed_time(b) / reps

    ms_g = time_graphs(graphs_of(grads))
    ms_i = time_graphs(graphs_of(inputs))
    gb = lora_grad_bytes(w, T)
    fl = lora_grad_input_flops(w, T)
    gbps = gb / (ms_g / 1e3) / 1e9
    tflops = fl / (ms_i / 1e3) / 1e12
    return {"workload": "lora_backward_7b_t%d_4x_r16" % T,
            "adapter_grads": {"kernel": "local_lora_grad_grouped (q,k,v) + local_lora_grad (o)",
                              "bound": "hbm",
                              "bytes_per_pass": gb, "ms_per_pass": round(ms_g, 5),
                              "achieved": round(gbps, 1), "peak": HBM_PEAK_GBPS,
                              "unit": "GB/s", "frac": round(gbps / HBM_PEAK_GBPS, 4)},
            "input_grad": {"kernel": "local_lora_grad_input x 4 (q,k,v,o)", "bound": "mfma",
                           "flops_per_pass": fl, "ms_per_pass": round(ms_i, 5),
                           "achieved": round(tflops, 1), "peak": BF16_PEAK_TFLOPS,
                           "unit": "TFLOP/s", "frac": round(tflops / BF16_PEAK_TFLOPS, 4)}}


def cpu_baseline(torch, workloads, w, meta, set0, args):
    """The oracle (float64 C, OpenMP) on the same decode step, on this host."""
    import oracle
    import oracle.chain as ochain
    st, pool, weights, x = set0
    D = w.head_dim

    def h(t):
        return t.detach().contiguous().view(torch.int16).cpu().numpy().view(np.uint16)

    lw = {k: (h(v) if v.dtype == torch.bfloat16 else v.cpu().numpy())
          for k, v in weights[0].items()}
    kpool = h(pool[0, 0]).reshape(-1)
    vpool = h(pool[0, 1]).reshape(-1)
    xh = h(x)
    qi = np.arange(meta.B + 1, dtype=np.int32)
    times = []
    t_budget = time.time() + args.cpu_budget_s
    n_req = meta.B
    while True:
        kc, vc = kpool.copy(), vpool.copy()
        t0 = time.perf_counter()
        oracle.block_version_check(meta.block_table, meta.ctx_lens, meta.block_version,
                                   meta.req_version)
        ochain.layer(xh, lw, kc, vc, w.hq, w.hkv, D, meta.block_table, qi, meta.ctx_lens,
                     meta.block_version, meta.req_version, meta.token_adapter,
                     meta.token_scale, residual=False)
        times.append(time.perf_counter() - t0)
        if time.time() > t_budget or len(times) >= 5:
            break
    t = float(np.median(times))
    return {"value": round(n_req / t, 2), "unit": "tokens/s", "cores": oracle.num_threads(),
            "kind": "oracle", "sample": "the whole decode step of the same workload "
            "(%d requests, 1 layer), median of %d runs" % (n_req, len(times)),
            "s_per_step": round(t, 3)}


if __name__ == "__main__":
    main()
