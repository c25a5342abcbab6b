"""One step of the mixed-adapter LoRA transformer path, as prepared C-ABI calls.

A step is the version check (once per step, it is the same for every layer)
followed, per layer, by
    q, k, v = LoRA projections of x            (local_lora_linear x3)
    o       = paged attention over the cache   (local_paged_attn_decode/_prefill,
              which first appends this step's k, v)
    y       = LoRA projection of o             (local_lora_linear, with the
              residual x added when layers are chained)
and the next layer's input is y. Nothing here computes: it only lays out the
buffers and replays the prepared calls, in order on the current stream, so
the whole step can also be captured into a HIP graph. A graph may instead be
captured with what does not depend on each other on parallel branches: the
version check (its stale list is for the host; attention checks the tags
itself) beside the whole step, and the k and v projections beside the q
projection. On the 7B decode step the joins cost more than the overlap
gains, so the in-order graph is the default.
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
        # calls that may run concurrently get workspaces of their own
        self.ws_k, self.ws_v, self.ws_vc = (bd.Workspace(dev) for _ in range(3))
        self.calls: List[bd.Call] = []
        self.buffers = {}
        cap = stale_cap if stale_cap is not None else meta.block_table.numel()
        self.version_check = bd.prepare_block_version_check(
            meta.block_table, meta.ctx_lens, meta.block_version, meta.req_version, cap=cap,
            workspace=self.ws_vc)
        self.calls.append(self.version_check)
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
            lc = {}
            for name, inp, outp, ws in (("q", xin, q, self.ws), ("k", xin, k, self.ws_k),
                                        ("v", xin, v, self.ws_v)):
                lc[name] = self._proj(lw, name, inp, outp, meta, None, ws)
            kc, vc = kv_pool[l, 0], kv_pool[l, 1]
            if kind == "decode":
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
            lc["o"] = self._proj(lw, "o", o, y, meta, xin if residual else None, self.ws)
            for name in ("q", "k", "v", "attn", "o"):
                self.calls.append(lc[name])
            self.layer_calls.append(lc)
            self.buffers[l] = dict(x=xin, q=q, k=k, v=v, o=o, y=y, lse=lse)
            xs.append(y)
        self.out = xs[-1]

    def _proj(self, lw, name, inp, outp, meta, residual, ws):
        if ("A_" + name) in lw:
            return bd.prepare_lora_linear(
                inp, lw["W_" + name], lw["A_" + name], lw["B_" + name], lw["ranks_" + name],
                meta.token_adapter, meta.token_scale, residual=residual, out=outp,
                workspace=ws)
        return bd.prepare_lora_linear(inp, lw["W_" + name], residual=residual, out=outp,
                                      workspace=ws)

    def __call__(self):
        for c in self.calls:
            c()
        return self.out

    def _run_branched(self, side):
        """The step with its independent calls on the side streams (capture)."""
        cur = torch.cuda.current_stream()
        s_vc, s_k, s_v = side
        s_vc.wait_stream(cur)
        with torch.cuda.stream(s_vc):
            self.version_check()
        for lc in self.layer_calls:
            s_k.wait_stream(cur)
            s_v.wait_stream(cur)
            lc["q"]()
            with torch.cuda.stream(s_k):
                lc["k"]()
            with torch.cuda.stream(s_v):
                lc["v"]()
            cur.wait_stream(s_k)
            cur.wait_stream(s_v)
            lc["attn"]()
            lc["o"]()
        cur.wait_stream(s_vc)

    def capture(self, parallel: bool = False):
        """Capture the step into a HIP graph; returns the torch.cuda.CUDAGraph.

        With `parallel`, independent calls become parallel branches of the
        graph (see the module docstring); otherwise the graph is the eager
        order. Run the step eagerly at least once first (kernel attributes are
        set on first launch). The library records no memset, so replays are
        exact.
        """
        g = torch.cuda.CUDAGraph()
        s = torch.cuda.Stream()
        side = [torch.cuda.Stream() for _ in range(3)]
        s.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(s):
            with torch.cuda.graph(g, stream=s):
                if parallel:
                    self._run_branched(side)
                else:
                    self()
        torch.cuda.current_stream().wait_stream(s)
        self._side = side  # the graph's branches were recorded on these
        return g
