"""The seeded input generator: determinism, shapes and distributions."""
import math

import numpy as np
import pytest
import torch

import workloads
from workloads import BLOCK_SIZE


@pytest.mark.parametrize("w", workloads.ALL, ids=lambda w: w.name)
def test_meta_is_deterministic_and_consistent(w):
    m1 = workloads.make_meta(w, seed=0)
    m2 = workloads.make_meta(w, seed=0)
    for f in ("ctx_lens", "block_table", "block_version", "req_version",
              "token_adapter", "stale_entries"):
        assert np.array_equal(getattr(m1, f), getattr(m2, f))
    assert m1.B == w.batch
    nb = (m1.ctx_lens + BLOCK_SIZE - 1) // BLOCK_SIZE
    assert m1.num_blocks == nb.sum()
    used = np.concatenate([m1.block_table[b, :nb[b]] for b in range(m1.B)])
    assert np.array_equal(np.sort(used), np.arange(m1.num_blocks))   # a permutation
    assert m1.T == (w.batch * w.chunk if w.kind == "prefill" else w.batch)
    if w.n_adapters:
        assert np.all((m1.request_adapter >= 0) & (m1.request_adapter < w.n_adapters))
        assert np.array_equal(m1.req_version, 1000 * (m1.request_adapter + 1))


def test_context_ranges():
    m = workloads.make_meta(workloads.DECODE_7B, 0)
    assert m.ctx_lens.min() >= 256 and m.ctx_lens.max() <= 4096
    m = workloads.make_meta(workloads.GQA_SKEW, 0)
    assert m.ctx_lens.min() >= 512 and m.ctx_lens.max() <= 8192
    m = workloads.make_meta(workloads.CHURN_32L, 0)
    assert m.ctx_lens.min() >= 1024 and m.ctx_lens.max() <= 16384
    m = workloads.make_meta(workloads.PREFILL_7B, 0)
    assert m.ctx_lens.tolist() == [512, 1024, 1536, 2560]
    assert workloads.make_meta(workloads.TINY_DECODE, 0).ctx_lens.tolist() == [17, 64, 100, 128]


def test_loguniform_and_zipf_shapes():
    # Many draws from the same recipe: log-lengths are uniform and adapter
    # frequencies follow (k+1)^-1.1.
    w = workloads.GQA_SKEW
    logs, ads = [], []
    for seed in range(60):
        m = workloads.make_meta(w, seed)
        logs.append(np.log(m.ctx_lens))
        ads.append(m.request_adapter)
    logs = np.concatenate(logs)
    u = (logs - math.log(512)) / (math.log(8192) - math.log(512))
    assert abs(u.mean() - 0.5) < 0.03 and abs(u.var() - 1 / 12) < 0.01
    ads = np.concatenate(ads)
    p = (np.arange(16) + 1.0) ** -1.1
    p /= p.sum()
    freq = np.bincount(ads, minlength=16) / ads.size
    assert abs(freq[0] - p[0]) < 0.03 and freq[0] > freq[3] > freq[15]


def test_stale_draw_spares_last_block():
    m = workloads.make_meta(workloads.CHURN_32L, 0)
    nb = (m.ctx_lens + 15) // 16
    assert np.all(m.stale_entries[:, 1] < nb[m.stale_entries[:, 0]] - 1)
    bt = m.block_table
    for b, j in m.stale_entries[:50]:
        assert m.block_version[bt[b, j]] == m.req_version[b] - 1


def test_float_distributions_cpu():
    w = workloads.TINY_DECODE
    lw = workloads.make_layer_weights(w, 0, "cpu", seed=0)
    W = lw["W_q"].float()
    assert W.shape == (256, 256)
    assert abs(W.std().item() - 0.02) < 0.002
    A, B = lw["A_q"].float(), lw["B_q"].float()
    assert abs(A.std().item() - 1 / math.sqrt(8)) < 0.02
    assert abs(B.std().item() - 0.01) < 0.001
    assert "A_k" not in lw and "A_o" not in lw      # LoRA on q and v only
    x = workloads.randn_bf16((64, 256), 1.0, "cpu", 3).float()
    assert abs(x.std().item() - 1.0) < 0.02
    again = workloads.randn_bf16((64, 256), 1.0, "cpu", 3)
    assert torch.equal(again.float(), x)


def test_ragged_rank_adapters_are_zero_padded():
    w = workloads.GQA_SKEW
    A, B, ranks = workloads.make_adapters(w, "k", "cpu", seed=5)
    assert A.shape == (16, 64, 4096) and B.shape == (16, 1024, 64)
    for a, r in enumerate(w.ranks):
        assert ranks[a].item() == r
        assert torch.count_nonzero(A[a, r:]) == 0
        assert torch.count_nonzero(B[a, :, r:]) == 0
        assert torch.count_nonzero(A[a, :r]) > 0
