"""One step of the mixed-adapter LoRA transformer path, as prepared C-ABI calls.

A step is the version check (once per step, it is the same for every layer;
in decode it is folded into the first layer's attention call,
local_paged_attn_decode_checked, which reads the same tags anyway) followed,
per layer, by
    q, k, v = LoRA projections of x            (local_lora_linear x3)
    o       = paged attention over the cache   (local_paged_attn_decode/_prefill,
              which first appends this step's k, v)
    y       = LoRA projection of o             (local_lora_linear, with the
              residual x added when layers are chained)
and the next layer's input is y. Nothing here computes: it only lays out the
buffers and replays the prepared calls, in order on the current stream, so
the whole step can also be captured into a HIP graph by the caller. The q, k
and v projections read the same x, so those with the same adapter setup run
as one grouped call (local_lora_linear_grouped): one pass of launches over
their concatenated weights.
"""
from __future__ import annotations

import math
from dataclasses import dataclass
from typing import Dict, List, Optional

import torch

from . import binding as bd

PROJECTIONS = ("q", "k", "v", "o")


@dataclass
class StepMeta:
    """Device copies of a step's integer metadata."""
    block_table: torch.Tensor   # [B, max_blocks] int32
    ctx_lens: torch.Tensor      # [B] int32
    block_version: torch.Tensor  # [num_blocks] int32
    req_version: torch.Tensor   # [B] int32
    q_indptr: torch.Tensor      # [B+1] int32
    token_adapter: torch.Tensor  # [T] int32
    token_scale: torch.Tensor   # [T] float32
    T: int
    B: int


def meta_to_device(m, device) -> StepMeta:
    """Copy a host metadata record (numpy arrays) to the device."""
    def t(a, dt=torch.int32):
        return torch.from_numpy(a.copy()).to(device=device, dtype=dt)
    return StepMeta(block_table=t(m.block_table), ctx_lens=t(m.ctx_lens),
                    block_version=t(m.block_version), req_version=t(m.req_version),
                    q_indptr=t(m.q_indptr), token_adapter=t(m.token_adapter),
                    token_scale=t(m.token_scale, torch.float32), T=m.T, B=m.B)


class Step:
    """Prepared calls of one step over `n_layers` layers.

    weights[l] maps "W_q", "A_q", "B_q", "ranks_q", ... to device tensors
    (adapter entries only for projections that carry adapters).
    kv_pool is [n_layers, 2, num_blocks, Hkv, 16*D] bf16.
    """

    def __init__(self, kind: str, x: torch.Tensor, weights: List[Dict[str, torch.Tensor]],
                 meta: StepMeta, kv_pool: torch.Tensor, hq: int, hkv: int, head_dim: int,
                 residual: bool, stale_cap: Optional[int] = None):
        assert kind in ("decode", "prefill")
        dev = x.device
        T, H = x.shape
        D = head_dim
        self.kind = kind
        self.n_layers = len(weights)
        self.inputs = (x, weights, meta, kv_pool)  # owned for the step's lifetime
        self.ws = bd.Workspace(dev)
        self.calls: List[bd.Call] = []
        self.buffers = {}
        cap = stale_cap if stale_cap is not None else meta.block_table.numel()
        self.version_check = None  # a separate call only in prefill
        if kind == "prefill":
            self.version_check = bd.prepare_block_version_check(
                meta.block_table, meta.ctx_lens, meta.block_version, meta.req_version, cap=cap,
                workspace=self.ws)
            self.calls.append(self.version_check)
            self.version_outputs = self.version_check.outputs
        else:
            self.version_outputs = (
                torch.empty((max(cap, 1), 2), dtype=torch.int32, device=dev),
                torch.empty((1,), dtype=torch.int32, device=dev),
                torch.empty((meta.B,), dtype=torch.int32, device=dev))
        sm_scale = 1.0 / math.sqrt(D)
        xs = [x]
        self.layer_calls = []
        for l, lw in enumerate(weights):
            xin = xs[-1]
            q = torch.empty((T, hq * D), dtype=torch.bfloat16, device=dev)
            k = torch.empty((T, hkv * D), dtype=torch.bfloat16, device=dev)
            v = torch.empty((T, hkv * D), dtype=torch.bfloat16, device=dev)
            o = torch.empty((T, hq * D), dtype=torch.bfloat16, device=dev)
            y = torch.empty((T, H), dtype=torch.bfloat16, device=dev)
            lse = torch.empty((T, hq), dtype=torch.float32, device=dev)
            lc = {"in": self._in_proj(lw, xin, {"q": q, "k": k, "v": v}, meta)}
            kc, vc = kv_pool[l, 0], kv_pool[l, 1]
            if kind == "decode" and l == 0:
                pairs, n_stale, valid = self.version_outputs
                lc["attn"] = bd.prepare_paged_attn_decode_checked(
                    q.view(T, hq, D), kc, vc, meta.block_table, meta.ctx_lens,
                    meta.block_version, meta.req_version, sm_scale,
                    k_new=k.view(T, hkv, D), v_new=v.view(T, hkv, D), Hkv=hkv,
                    out=o.view(T, hq, D), lse=lse, cap=cap, stale_pairs=pairs,
                    n_stale=n_stale, valid_tokens=valid, workspace=self.ws)
            elif kind == "decode":
                lc["attn"] = bd.prepare_paged_attn_decode(
                    q.view(T, hq, D), kc, vc, meta.block_table, meta.ctx_lens,
                    meta.block_version, meta.req_version, sm_scale,
                    k_new=k.view(T, hkv, D), v_new=v.view(T, hkv, D), Hkv=hkv,
                    out=o.view(T, hq, D), lse=lse, workspace=self.ws)
            else:
                lc["attn"] = bd.prepare_paged_attn_prefill(
                    q.view(T, hq, D), meta.q_indptr, kc, vc, meta.block_table, meta.ctx_lens,
                    meta.block_version, meta.req_version, sm_scale,
                    k_new=k.view(T, hkv, D), v_new=v.view(T, hkv, D), Hkv=hkv,
                    out=o.view(T, hq, D), lse=lse, workspace=self.ws)
            lc["o"] = self._proj(lw, "o", o, y, meta, xin if residual else None)
            self.calls += lc["in"] + [lc["attn"], lc["o"]]
            self.layer_calls.append(lc)
            self.buffers[l] = dict(x=xin, q=q, k=k, v=v, o=o, y=y, lse=lse)
            xs.append(y)
        self.out = xs[-1]

    def _proj(self, lw, name, inp, outp, meta, residual):
        if ("A_" + name) in lw:
            return bd.prepare_lora_linear(
                inp, lw["W_" + name], lw["A_" + name], lw["B_" + name], lw["ranks_" + name],
                meta.token_adapter, meta.token_scale, residual=residual, out=outp,
                workspace=self.ws)
        return bd.prepare_lora_linear(inp, lw["W_" + name], residual=residual, out=outp,
                                      workspace=self.ws)

    def _in_proj(self, lw, x, outs, meta) -> List[bd.Call]:
        """Calls for the q, k, v projections of x: one grouped call per set of
        projections with the same adapter setup."""
        calls = []
        with_ad = [n for n in ("q", "k", "v") if ("A_" + n) in lw]
        without = [n for n in ("q", "k", "v") if ("A_" + n) not in lw]
        if len({tuple(lw["A_" + n].shape[:2]) for n in with_ad}) > 1:
            # adapter sets of different shapes: those projections one by one
            calls += [self._proj(lw, n, x, outs[n], meta, None) for n in with_ad]
            with_ad = []
        for names, ad in ((with_ad, True), (without, False)):
            if not names:
                continue
            if len(names) == 1:
                calls.append(self._proj(lw, names[0], x, outs[names[0]], meta, None))
            elif ad:
                calls.append(bd.prepare_lora_linear_grouped(
                    x, [lw["W_" + n] for n in names], [lw["A_" + n] for n in names],
                    [lw["B_" + n] for n in names], [lw["ranks_" + n] for n in names],
                    meta.token_adapter, meta.token_scale, outs=[outs[n] for n in names],
                    workspace=self.ws))
            else:
                calls.append(bd.prepare_lora_linear_grouped(
                    x, [lw["W_" + n] for n in names], outs=[outs[n] for n in names],
                    workspace=self.ws))
        return calls

    def __call__(self):
        for c in self.calls:
            c()
        return self.out

    def capture(self):
        """Capture the step into a HIP graph; returns the torch.cuda.CUDAGraph.

        Run the step eagerly at least once first (kernel attributes are set on
        first launch). The library records no memset, so replays are exact.
        """
        g = torch.cuda.CUDAGraph()
        s = torch.cuda.Stream()
        s.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(s):
            with torch.cuda.graph(g, stream=s):
                self()
        torch.cuda.current_stream().wait_stream(s)
        return g
