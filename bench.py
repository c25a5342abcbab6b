#!/usr/bin/env python3
"""Benchmark of the mixed-adapter LoRA step on one MI355X, every workload.

A decode step is one pass of the whole path over one batch: the version
check, the q/k/v LoRA projections (one grouped call), the appending,
version-masked paged decode attention and the output LoRA projection, for
every layer. A prefill step is the same with a chunk of tokens per request
and causal prefill attention. Inputs are seeded synthetic tensors already
resident in HBM; a step is one HIP-graph replay, timed with an event pair per
step, and the median is reported.

Prints ONE JSON line:
* the headline is the largest single-GPU workload, `churn_32l_b128` (32
  layers, 32q/8kv x 128, batch 128, contexts U[1024,16384], 32 rank-16
  adapters, 10% of block-table entries stale): `value` is its decode tokens/s,
  `roofline` its dominant kernel (decode attention, HIP events around every
  layer's launch), `hbm_step` the whole step's algorithmic bytes over the step
  time, and `cpu_baseline` the oracle on a seeded sample of 8 of the 128
  requests through all 32 layers (its rate, and the 128-request step time it
  extrapolates to, labelled as such);
* `workloads` holds the same record for the other four workloads:
  `tiny_decode` (absolute time), `decode_7b_mha_b32` and `gqa_skew_b64`
  (decode steps; two input sets alternate so that the last-level cache
  cannot serve one step's weights to the next), and `prefill_7b_4x512` (the
  whole prefill step, its LoRA-fused projections and its attention against
  the matrix-core peak); each with the oracle timed on the whole step;
* `reprefill` (stale-coverage prefill under a staged version) and
  `lora_grad` (the LoRA backward of a training chunk).

`--workload NAME` runs one workload alone (its record as the headline, no
CPU leg, no other legs): for profiling runs.
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
HEADLINE = "churn_32l_b128"
CPU_SAMPLE_REQUESTS = 8         # oracle sample of the 32-layer workload


def say(*a):
    """Progress on stderr (the JSON line alone goes to stdout)."""
    print("bench:", *a, file=sys.stderr, flush=True)


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=50)
    p.add_argument("--warmup", type=int, default=10)
    p.add_argument("--sets", type=int, default=2,
                   help="input sets rotated across steps (single-layer workloads)")
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--cpu-budget-s", type=float, default=20.0,
                   help="repeat a workload's oracle run (at most 3 times after a warm-up run) "
                        "while the total stays within this budget")
    p.add_argument("--workload", default="all",
                   choices=("all", "tiny_decode", "decode_7b_mha_b32", "gqa_skew_b64",
                            "churn_32l_b128", "prefill_7b_4x512"),
                   help="one workload alone (no CPU leg, no other legs)")
    p.add_argument("--traffic-probe", action="store_true",
                   help="only run, eagerly, a 256 MiB device copy (the calibration of the "
                        "HBM byte counters) and 5 decode attention launches of the workload "
                        "(layer 0); for rocprofv3 --pmc runs")
    return p.parse_args()


ROOT = os.path.dirname(os.path.abspath(__file__))
DECODE_SOURCES = ("paper_2608_15241_amd/csrc/paged_attn_decode.hip",
                  "paper_2608_15241_amd/csrc/common.hpp")


def traffic_file(workload):
    return os.path.join(ROOT, "profiles", "decode_attn_traffic_%s.md" % workload)


def decode_source_hash():
    """sha256 over the sources of the decode attention kernels."""
    import hashlib
    h = hashlib.sha256()
    for rel in DECODE_SOURCES:
        with open(os.path.join(ROOT, rel), "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def measured_traffic(workload):
    """HBM bytes per decode attention launch of `workload` from the committed
    counter summary, or None when it is missing or was taken on other kernel
    sources."""
    try:
        text = open(traffic_file(workload)).read()
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
    D, hq, hkv = w.head_dim, w.hq, w.hkv
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


def workload_config(w, meta, n_sets, valid_tokens=None):
    c = {"workload": w.name, "layers": w.n_layers, "hidden": w.hidden,
         "heads": "%dq/%dkv x %d" % (w.hq, w.hkv, w.head_dim), "batch": meta.B,
         "context": context_text(w), "sum_context": int(meta.ctx_lens.sum()),
         "stale_frac": w.stale_frac, "adapters": adapters_text(w), "input_sets": n_sets}
    if w.kind == "prefill":
        c["chunk_tokens"] = w.chunk
        c["tokens_per_step"] = meta.T
    if valid_tokens is not None:
        c["valid_kv_tokens"] = valid_tokens
    return c


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


def cpu_cores():
    """(threads the oracle runs on, CPUs in this process's affinity mask)."""
    import oracle
    return oracle.num_threads(), len(os.sched_getaffinity(0))


def time_graph_steps(torch, graphs, steps, warmup):
    """Replays graphs[i % n] `warmup` times, then times `steps` replays with
    one event pair around each. Returns (median ms, mean ms over the
    bracketed region)."""
    for i in range(warmup):
        graphs[i % len(graphs)].replay()
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(steps + 1)]
    torch.cuda.synchronize()
    ev[0].record(stream)
    for i in range(steps):
        graphs[i % len(graphs)].replay()
        ev[i + 1].record(stream)
    torch.cuda.synchronize()
    per = [ev[i].elapsed_time(ev[i + 1]) for i in range(steps)]
    return float(np.median(per)), ev[0].elapsed_time(ev[-1]) / steps


def bench_decode(torch, workloads, lk, w, args, with_cpu):
    """Decode step of workload w: graph replays, attention launches, bytes, and
    (with_cpu) the oracle on the same step. Frees its inputs before returning."""
    from paper_2608_15241_amd.step import Step, meta_to_device
    dev = "cuda:0"
    meta = workloads.make_meta(w, seed=0)
    md = meta_to_device(meta, dev)
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
    # eager steps first (they set kernel attributes), then one graph per set
    for i in range(max(2, len(sets))):
        sets[i % len(sets)][0]()
    torch.cuda.synchronize()
    graphs = [st.capture() for st, *_ in sets]
    say("timed steps", w.name)
    K = args.steps
    ms_med, ms_mean = time_graph_steps(torch, graphs, K, args.warmup)

    # the dominant kernel (decode attention): every layer's attention call of
    # a step (a single-layer step's call 8 times) captured back to back in one
    # graph per input set, and HIP events on the same stream around replays
    # of those graphs; per launch = the median replay time / launches per replay
    stream = torch.cuda.current_stream()
    per_graph = w.n_layers if w.n_layers > 1 else 8
    attn_graphs = []
    for st, *_ in sets:
        calls = [lc["attn"] for lc in st.layer_calls] * (per_graph // w.n_layers)
        g = torch.cuda.CUDAGraph()
        cs = torch.cuda.Stream()
        cs.wait_stream(stream)
        with torch.cuda.stream(cs):
            with torch.cuda.graph(g, stream=cs):
                for c in calls:
                    c()
        stream.wait_stream(cs)
        attn_graphs.append(g)
    for g in attn_graphs:
        g.replay()
    torch.cuda.synchronize()
    n_rep = max(4, min(K, 20))
    ev_a = [torch.cuda.Event(enable_timing=True) for _ in range(n_rep)]
    ev_b = [torch.cuda.Event(enable_timing=True) for _ in range(n_rep)]
    for i in range(n_rep):
        ev_a[i].record(stream)
        attn_graphs[i % len(attn_graphs)].replay()
        ev_b[i].record(stream)
    torch.cuda.synchronize()
    attn_ms = float(np.median([a.elapsed_time(b) for a, b in zip(ev_a, ev_b)])) / per_graph
    del attn_graphs

    attn_bytes, step_bytes, valid_tokens = decode_bytes(w, meta)
    attn_gbps = attn_bytes / (attn_ms / 1e3) / 1e9
    step_gbps = step_bytes / (ms_med / 1e3) / 1e9
    rec = {
        "tokens_per_s": round(meta.B / (ms_med / 1e3), 1),
        "ms_per_step": round(ms_med, 5),
        "ms_per_step_mean": round(ms_mean, 5),
        "config": workload_config(w, meta, n_sets, valid_tokens),
        "roofline": {"kernel": ("local_paged_attn_decode_checked (the step's version check "
                                "folded in)" if w.n_layers == 1 else
                                "local_paged_attn_decode (layer 0: _checked, the step's "
                                "version check folded in)"), "bound": "hbm",
                     "achieved": round(attn_gbps, 1), "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                     "frac": round(attn_gbps / HBM_PEAK_GBPS, 4),
                     "traffic": measured_traffic(w.name),
                     "bytes_per_launch": attn_bytes, "ms_per_launch": round(attn_ms, 5),
                     "launches_timed": n_rep * per_graph,
                     "timing": "graph replays of back-to-back launches of the entry point "
                               "(decode kernel + merge), median per replay / launches"},
        "hbm_step": {"bytes_per_step": step_bytes, "achieved": round(step_gbps, 1),
                     "unit": "GB/s", "frac": round(step_gbps / HBM_PEAK_GBPS, 4)},
    }
    if w.name == "tiny_decode":
        rec["note"] = ("launch-latency bound (the whole step's data fits in the last-level "
                       "cache): the absolute step time is the figure; the fractions are not "
                       "meaningful")
    if with_cpu:
        say("cpu baseline", w.name)
        rec["cpu_baseline"] = cpu_decode(torch, workloads, w, meta, sets[0], args)
    del graphs, sets, md
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    return rec


def _h(torch, t):
    return t.detach().contiguous().view(torch.int16).cpu().numpy().view(np.uint16)


def _gather_blocks(torch, pool_l, hkv, D, meta, reqs):
    """Host copies of the K and V blocks of `reqs` in one layer's pool, with
    block ids renumbered in the order the requests own them. Returns
    (k, v, table, block_version)."""
    nb = [(int(meta.ctx_lens[b]) + 15) // 16 for b in reqs]
    ids = np.concatenate([meta.block_table[b, :n] for b, n in zip(reqs, nb)]).astype(np.int64)
    idx = torch.from_numpy(ids).to(pool_l.device)
    per = hkv * 16 * D
    k = _h(torch, pool_l[0].reshape(-1, per).index_select(0, idx)).reshape(-1)
    v = _h(torch, pool_l[1].reshape(-1, per).index_select(0, idx)).reshape(-1)
    table = np.zeros((len(reqs), max(nb)), np.int32)
    off = 0
    for i, n in enumerate(nb):
        table[i, :n] = np.arange(off, off + n)
        off += n
    return k, v, table, meta.block_version[ids].astype(np.int32)


def cpu_decode(torch, workloads, w, meta, set0, args):
    """The oracle (float64 C, OpenMP) on the decode step of w on this host:
    every request of a single-layer workload; for the 32-layer workload a
    seeded sample of requests through every layer (the oracle's cost is linear
    in the requests: each one reads every weight and its own KV), each layer's
    blocks and weights copied to the host before its timed part."""
    import oracle
    import oracle.chain as ochain
    st, pool, weights, x = set0
    D = w.head_dim
    if w.n_layers > 1:
        rng = np.random.default_rng(2025)
        reqs = np.sort(rng.choice(meta.B, size=CPU_SAMPLE_REQUESTS, replace=False))
    else:
        reqs = np.arange(meta.B)
    ctx, rv = meta.ctx_lens[reqs], meta.req_version[reqs]
    tok_a, tok_s = meta.token_adapter[reqs], meta.token_scale[reqs]
    qi = np.arange(len(reqs) + 1, dtype=np.int32)

    def run_once():
        xo = _h(torch, x)[reqs]
        t = 0.0
        for l in range(w.n_layers):
            lw = {k: (_h(torch, v) if v.dtype == torch.bfloat16 else v.cpu().numpy())
                  for k, v in weights[l].items()}
            kh, vh, table, bv = _gather_blocks(torch, pool[l], w.hkv, D, meta, reqs)
            t0 = time.perf_counter()
            if l == 0:
                oracle.block_version_check(meta.block_table, meta.ctx_lens,
                                           meta.block_version, meta.req_version)
            xo, _ = ochain.layer(xo, lw, kh, vh, w.hq, w.hkv, D, table, qi, ctx, bv, rv,
                                 tok_a, tok_s, residual=False)
            t += time.perf_counter() - t0
        return t

    times = repeat_within_budget(run_once, args.cpu_budget_s)
    t = float(np.median(times))
    threads, affinity = cpu_cores()
    rec = {"value": round(len(reqs) / t, 2), "unit": "tokens/s", "cores": threads,
           "affinity_cpus": affinity, "kind": "oracle", "s_per_step": round(t, 4),
           "runs": len(times)}
    if w.n_layers > 1:
        rec["sample"] = ("%d of %d requests (seeded) through all %d layers; timed part: the "
                         "oracle's version check and layer steps, not the device-to-host "
                         "copies of each layer's blocks and weights" %
                         (len(reqs), meta.B, w.n_layers))
        rec["extrapolated_s_per_step_%d_requests" % meta.B] = round(t * meta.B / len(reqs), 2)
        rec["extrapolation"] = "linear in requests (labelled extrapolation, not measured)"
    else:
        rec["sample"] = "the whole decode step (%d requests, 1 layer)" % meta.B
    return rec


def repeat_within_budget(fn, budget_s):
    """Runs fn once; if that run took under a quarter of the budget it was a
    warm-up, and fn runs up to 3 more times while the total stays within the
    budget. Returns the timed runs."""
    t0 = time.time()
    first = fn()
    if first * 4 > budget_s:
        return [first]
    times = []
    while len(times) < 3 and (time.time() - t0) + first <= budget_s:
        times.append(fn())
    return times or [first]


def bench_prefill_step(torch, workloads, lk, args, with_cpu):
    """The whole prefill step of prefill_7b_4x512 (version check, grouped
    q/k/v, appending causal attention, o) as graph replays over two input
    sets, plus its projections and its attention alone, and the oracle on the
    same step."""
    from paper_2608_15241_amd.step import Step, meta_to_device
    w = workloads.PREFILL_7B
    dev = "cuda:0"
    meta = workloads.make_meta(w, seed=0)
    md = meta_to_device(meta, dev)
    sets = []
    for s in range(2):
        say("prefill input set", s)
        weights = [workloads.make_layer_weights(w, 0, dev, seed=800 + s)]
        pool = workloads.make_kv_pool(w, meta, dev, seed=800 + s)
        x = workloads.randn_bf16((meta.T, w.hidden), 1.0, dev, seed=810 + s)
        st = Step("prefill", x, weights, md, pool, w.hq, w.hkv, w.head_dim, residual=False)
        sets.append((st, pool, weights, x))
    for st, *_ in sets:
        st()  # the step rewrites the same slots with the same values on every replay
    torch.cuda.synchronize()
    graphs = [st.capture() for st, *_ in sets]
    ms_med, ms_mean = time_graph_steps(torch, graphs, args.steps, args.warmup)
    gemm = prefill_gemm_flops(w, meta)
    attn = prefill_attn_flops(w, meta)
    tflops = (gemm + attn) / (ms_med / 1e3) / 1e12
    rec = {"tokens_per_s": round(meta.T / (ms_med / 1e3), 1),
           "ms_per_step": round(ms_med, 5), "ms_per_step_mean": round(ms_mean, 5),
           "config": workload_config(w, meta, 2),
           "mfma_step": {"flops_per_step": gemm + attn, "achieved": round(tflops, 1),
                         "peak": BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
                         "frac": round(tflops / BF16_PEAK_TFLOPS, 4)}}
    if with_cpu:
        say("cpu baseline", w.name)
        rec["cpu_baseline"] = cpu_prefill(torch, w, meta, sets[0], args)
    del graphs, sets, md
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    say("prefill projections")
    rec["projections"] = bench_prefill(torch, workloads, lk, dev)
    say("prefill attention")
    rec["attention"] = bench_prefill_attn(torch, workloads, lk, dev)
    return rec


def cpu_prefill(torch, w, meta, set0, args):
    """The oracle on the whole prefill step (2048 tokens, 1 layer)."""
    import oracle
    import oracle.chain as ochain
    st, pool, weights, x = set0
    lw = {k: (_h(torch, v) if v.dtype == torch.bfloat16 else v.cpu().numpy())
          for k, v in weights[0].items()}
    kh, vh = _h(torch, pool[0, 0]).reshape(-1), _h(torch, pool[0, 1]).reshape(-1)
    xh = _h(torch, x)

    def run_once():
        t0 = time.perf_counter()
        oracle.block_version_check(meta.block_table, meta.ctx_lens, meta.block_version,
                                   meta.req_version)
        ochain.layer(xh, lw, kh, vh, w.hq, w.hkv, w.head_dim, meta.block_table,
                     meta.q_indptr, meta.ctx_lens, meta.block_version, meta.req_version,
                     meta.token_adapter, meta.token_scale, residual=False)
        return time.perf_counter() - t0

    times = repeat_within_budget(run_once, args.cpu_budget_s)
    t = float(np.median(times))
    threads, affinity = cpu_cores()
    return {"value": round(meta.T / t, 2), "unit": "tokens/s", "cores": threads,
            "affinity_cpus": affinity, "kind": "oracle", "s_per_step": round(t, 3),
            "runs": len(times),
            "sample": "the whole prefill step (%d tokens, 1 layer)" % meta.T}


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

    lk.load_library()
    torch.cuda.set_device(0)
    if args.traffic_probe:
        traffic_probe(torch, workloads, workloads.BY_NAME[
            HEADLINE if args.workload == "all" else args.workload], "cuda:0")
        return
    alone = args.workload != "all"
    head_name = HEADLINE if not alone else args.workload
    with_cpu = not alone and not args.no_cpu_baseline

    if head_name == "prefill_7b_4x512":
        head = bench_prefill_step(torch, workloads, lk, args, False)
        unit_tokens = "prefill tokens/s"
    else:
        head = bench_decode(torch, workloads, lk, workloads.BY_NAME[head_name], args,
                            with_cpu)
        unit_tokens = "tokens/s"
    result = {
        "metric": "decode tokens/s + achieved HBM GB/s (% peak); prefill LoRA-GEMM MFMA util",
        "value": head["tokens_per_s"],
        "unit": unit_tokens,
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": head["ms_per_step"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
    }
    for k, v in head.items():
        if k not in ("tokens_per_s", "ms_per_step"):
            result[k] = v
    result["ms_per_step_note"] = "median of per-step event times over the timed graph replays"

    if not alone:
        subs = {}
        for name in ("decode_7b_mha_b32", "gqa_skew_b64", "tiny_decode"):
            subs[name] = bench_decode(torch, workloads, lk, workloads.BY_NAME[name], args,
                                      with_cpu)
        subs["prefill_7b_4x512"] = bench_prefill_step(torch, workloads, lk, args, with_cpu)
        result["workloads"] = subs
        say("stale-coverage prefill")
        result["reprefill"] = bench_reprefill(torch, workloads, lk, "cuda:0")
        say("lora backward")
        result["lora_grad"] = bench_lora_grad(torch, workloads, lk, "cuda:0")
    print(json.dumps(result), flush=True)


def traffic_probe(torch, workloads, w, dev):
    """A plain copy of known size, then decode attention launches of layer 0
    of workload w, eagerly."""
    from paper_2608_15241_amd.step import Step, meta_to_device
    meta = workloads.make_meta(w, seed=0)
    md = meta_to_device(meta, dev)
    weights = [workloads.make_layer_weights(w, 0, dev, seed=100)]
    pool = workloads.make_kv_pool(w, meta, dev, seed=100, n_layers=1)
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
    print(json.dumps({"traffic_probe": {"workload": w.name, "copy_read_bytes": n,
                                        "copy_write_bytes": n,
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
    del graphs
    return {"workload": w.name,
            "kernel": "local_lora_linear_grouped (q,k,v) + local_lora_linear (o), T=%d" % meta.T,
            "bound": "mfma", "flops_per_step": flops, "ms_per_step": round(ms, 5),
            "achieved": round(tflops, 1), "peak": BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
            "frac": round(tflops / BF16_PEAK_TFLOPS, 4),
            "yardstick": library_gemm_yardstick(torch, w, meta, dev, reps)}


def library_gemm_yardstick(torch, w, meta, dev, reps):
    """The same base products (x W_qkv^T and o W_o^T, no adapters) through
    torch.mm, i.e. the vendor GEMM library, timed the same way: a reference
    for what the matrix cores give a plain GEMM of these shapes on this machine."""
    sets = []
    for s in range(2):
        wq = [torch.empty(w.proj_shape(n), dtype=torch.bfloat16, device=dev).normal_()
              for n in ("q", "k", "v")]
        wqkv_t = torch.cat(wq, 0).t().contiguous()   # [K, Nq + Nk + Nv]
        N, K = w.proj_shape("o")
        wo_t = torch.empty((N, K), dtype=torch.bfloat16, device=dev).normal_().t().contiguous()
        x = torch.empty((meta.T, w.hidden), dtype=torch.bfloat16, device=dev).normal_()
        o = torch.empty((meta.T, K), dtype=torch.bfloat16, device=dev).normal_()
        y1 = torch.empty((meta.T, wqkv_t.shape[1]), dtype=torch.bfloat16, device=dev)
        y2 = torch.empty((meta.T, N), dtype=torch.bfloat16, device=dev)
        sets.append((x, wqkv_t, y1, o, wo_t, y2))
    for x, wt, y1, o, wo, y2 in sets:
        torch.mm(x, wt, out=y1)
        torch.mm(o, wo, out=y2)
    torch.cuda.synchronize()
    graphs = []
    for x, wt, y1, o, wo, y2 in sets:
        g = torch.cuda.CUDAGraph()
        st = torch.cuda.Stream()
        st.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(st):
            with torch.cuda.graph(g, stream=st):
                torch.mm(x, wt, out=y1)
                torch.mm(o, wo, out=y2)
        torch.cuda.current_stream().wait_stream(st)
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
    flops = 2 * meta.T * (w.hidden * sets[0][1].shape[1] + sets[0][3].shape[1] * sets[0][5].shape[1])
    tflops = flops / (ms / 1e3) / 1e12
    del graphs, sets
    return {"kernel": "torch.mm (the vendor GEMM library): the same base products, no adapters",
            "flops_per_step": flops, "ms_per_step": round(ms, 5), "achieved": round(tflops, 1),
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
    {0, 512, 1024, 2048}), timed as graph replays of back-to-back calls over two
    input sets."""
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
    # one graph of back-to-back calls, the two input sets in turn (as the
    # decode attention is timed): the figure is a call's time inside a step,
    # without the gap between graph launches
    per_graph = 8
    g = torch.cuda.CUDAGraph()
    st = torch.cuda.Stream()
    st.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(st):
        with torch.cuda.graph(g, stream=st):
            for i in range(per_graph):
                calls[i % 2]()
    torch.cuda.current_stream().wait_stream(st)
    g.replay()
    torch.cuda.synchronize()
    times = []
    for r in range(reps):
        a = torch.cuda.Event(enable_timing=True)
        b = torch.cuda.Event(enable_timing=True)
        a.record()
        g.replay()
        b.record()
        torch.cuda.synchronize()
        times.append(a.elapsed_time(b) / per_graph)
    ms = float(np.median(times))
    del g
    flops = prefill_attn_flops(w, meta)
    tflops = flops / (ms / 1e3) / 1e12
    return {"workload": w.name, "kernel": "local_paged_attn_prefill (append + attention)",
            "bound": "mfma", "flops_per_call": flops, "ms_per_call": round(ms, 5),
            "achieved": round(tflops, 1), "peak": BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
            "frac": round(tflops / BF16_PEAK_TFLOPS, 4), "launches_timed": reps * per_graph,
            "timing": "graph replays of %d back-to-back calls (two input sets in turn), "
                      "median per replay / calls" % per_graph}


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


if __name__ == "__main__":
    main()
