"""The oracle's layer step: its own functions composed in the step's order.

TEST INFRASTRUCTURE ONLY (see the package docstring).

Per layer (the mixed-adapter LoRA transformer path): q, k, v are LoRA
projections of the layer input; this step's k, v are appended to the paged
cache; attention with the version mask gives o; the output projection of o,
plus the layer input when layers are chained through a residual stream,
gives the next layer's input. Every stage's output is bf16 by definition of
the library interface, so the chain rounds each stage's float64 result to
bf16 (nearest even) before the next stage consumes it.
"""
from __future__ import annotations

import math
from typing import Dict, Optional

import numpy as np

from . import kv_append, lora_linear, paged_attn, to_bf16


def project(x, lw: Dict[str, np.ndarray], name: str, token_adapter, token_scale,
            residual=None):
    if ("A_" + name) in lw:
        return lora_linear(x, lw["W_" + name], lw["A_" + name], lw["B_" + name],
                           lw["ranks_" + name], token_adapter, token_scale, residual)
    return lora_linear(x, lw["W_" + name], residual=residual)


def layer(x, lw, k_pool, v_pool, hq, hkv, D, block_table, q_indptr, ctx_lens,
          block_version, req_version, token_adapter, token_scale, residual: bool):
    """One layer on host arrays; k_pool/v_pool (uint16) are appended in place.

    Returns (y_bf16, stages) with stages holding every intermediate (float64
    before rounding).
    """
    T = x.shape[0]
    st = {}
    for name in ("q", "k", "v"):
        st[name] = project(x, lw, name, token_adapter, token_scale)
    qb, kb, vb = (to_bf16(st[n]) for n in ("q", "k", "v"))
    kv_append(k_pool, v_pool, hkv, D, block_table, q_indptr, ctx_lens,
              kb.reshape(T, hkv, D), vb.reshape(T, hkv, D))
    o, lse = paged_attn(qb.reshape(T, hq, D), q_indptr, hq, hkv, D, k_pool, v_pool,
                        block_table, ctx_lens, block_version, req_version, 1.0 / math.sqrt(D))
    st["o"], st["lse"] = o.reshape(T, hq * D), lse
    ob = to_bf16(st["o"])
    st["y"] = project(ob, lw, "o", token_adapter, token_scale,
                      residual=x if residual else None)
    return to_bf16(st["y"]), st
