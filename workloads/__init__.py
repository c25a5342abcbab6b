"""Seeded synthetic workloads shared by the kernels' tests, the oracle's
tests and the benchmark. Input generation only: no arithmetic of the method."""
from .configs import (ALL, BLOCK_SIZE, BY_NAME, CHURN_32L, DECODE_7B, GQA_SKEW,
                      LORA_SCALE, PREFILL_7B, TINY_DECODE, Workload)
from .generate import (Meta, adapter_version, make_adapters, make_kv_pool,
                       make_layer_weights, make_meta, randn_bf16, to_host_u16)
