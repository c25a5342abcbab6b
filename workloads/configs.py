"""The five workloads of the mixed-adapter LoRA step, as frozen records.

They are seeded synthetic stand-ins shaped like the paper's 7B-class
deployment (§7.1: a 7B model served with LoRA adapters on one GPU). The paper
measures on an agent benchmark with trained adapters; none of that is needed
here: every tensor is drawn from the distributions stated below, and the
structure (context-length mix, adapter mix, stale blocks) is what the kernels
see.

Value distributions (shared by every workload): activations N(0,1), base
weights N(0,0.02^2), adapter A ~ N(0, 1/r) with r that adapter's rank,
adapter B ~ N(0, 0.01^2), KV cache N(0,1); every float is drawn in float32
and rounded to bf16 (nearest even). LoRA scale s = 2.0 for every routed
token. KV block size 16.

Layers of the multi-layer workload are chained output-to-input (layer l+1
consumes layer l's output projection). The paper defines no normalisation
and no residual stream for this path, and without a normalisation a residual
sum of these distributions grows by orders of magnitude over 32 layers
(attention collapses onto the newest token), so none is added.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Optional, Tuple

BLOCK_SIZE = 16
LORA_SCALE = 2.0


@dataclass(frozen=True)
class Workload:
    name: str
    kind: str                      # "decode" or "prefill"
    n_layers: int
    hidden: int
    hq: int                        # query heads
    hkv: int                       # KV heads
    head_dim: int
    batch: int                     # requests
    # context lengths: ("fixed", (L0, L1, ...)) | ("uniform", lo, hi)
    #                  | ("loguniform", lo, hi); for prefill the cached prefix
    #                  lengths are ("fixed", (...)) and `chunk` tokens follow.
    ctx: tuple
    n_adapters: int
    ranks: Tuple[int, ...]         # one per adapter
    lora_targets: Tuple[str, ...]  # subset of ("q", "k", "v", "o")
    assignment: str                # "uniform" or "zipf"
    zipf_s: float = 0.0
    chunk: int = 0                 # prefill tokens per request
    stale_frac: float = 0.0        # fraction of block-table entries made stale
    description: str = ""

    @property
    def r_max(self) -> int:
        return max(self.ranks) if self.ranks else 8

    def proj_shape(self, proj: str) -> Tuple[int, int]:
        """(N, K) of a projection weight W[N][K]."""
        h, d = self.hidden, self.head_dim
        return {
            "q": (self.hq * d, h),
            "k": (self.hkv * d, h),
            "v": (self.hkv * d, h),
            "o": (h, self.hq * d),
        }[proj]


TINY_DECODE = Workload(
    name="tiny_decode",
    kind="decode", n_layers=1, hidden=256, hq=4, hkv=4, head_dim=64,
    batch=4, ctx=("fixed", (17, 64, 100, 128)),
    n_adapters=3, ranks=(8, 8, 8), lora_targets=("q", "v"),
    assignment="uniform",
    description="1 layer, hidden 256, 4x64 MHA, 4 requests of context "
                "{17,64,100,128}, 3 rank-8 adapters on q and v",
)

DECODE_7B = Workload(
    name="decode_7b_mha_b32",
    kind="decode", n_layers=1, hidden=4096, hq=32, hkv=32, head_dim=128,
    batch=32, ctx=("uniform", 256, 4096),
    n_adapters=8, ranks=(16,) * 8, lora_targets=("q", "k", "v", "o"),
    assignment="uniform",
    description="7B-class single-layer decode: hidden 4096, 32x128 MHA, "
                "batch 32, context U[256,4096], 8 rank-16 adapters on q/k/v/o",
)

PREFILL_7B = Workload(
    name="prefill_7b_4x512",
    kind="prefill", n_layers=1, hidden=4096, hq=32, hkv=32, head_dim=128,
    batch=4, ctx=("fixed", (0, 512, 1024, 2048)), chunk=512,
    n_adapters=4, ranks=(16,) * 4, lora_targets=("q", "k", "v", "o"),
    assignment="uniform",
    description="7B-class single-layer chunked prefill: 4 requests each adding "
                "512 tokens on prefixes {0,512,1024,2048}, 4 rank-16 adapters",
)

GQA_SKEW = Workload(
    name="gqa_skew_b64",
    kind="decode", n_layers=1, hidden=4096, hq=32, hkv=8, head_dim=128,
    batch=64, ctx=("loguniform", 512, 8192),
    n_adapters=16, ranks=tuple((8, 16, 32, 64)[i % 4] for i in range(16)),
    lora_targets=("q", "k", "v", "o"),
    assignment="zipf", zipf_s=1.1,
    description="GQA decode 32q/8kv x128, batch 64, context log-uniform "
                "[512,8192], 16 adapters of ranks {8,16,32,64}, Zipf(1.1)",
)

CHURN_32L = Workload(
    name="churn_32l_b128",
    kind="decode", n_layers=32, hidden=4096, hq=32, hkv=8, head_dim=128,
    batch=128, ctx=("uniform", 1024, 16384),
    n_adapters=32, ranks=(16,) * 32, lora_targets=("q", "k", "v", "o"),
    assignment="uniform", stale_frac=0.10,
    description="32-layer GQA decode, batch 128, context U[1024,16384], "
                "32 rank-16 adapters, 10% of block-table entries stale",
)

ALL = (TINY_DECODE, DECODE_7B, PREFILL_7B, GQA_SKEW, CHURN_32L)
BY_NAME = {w.name: w for w in ALL}
