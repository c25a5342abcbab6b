"""GPU parity of local_block_version_check: bit-exact against the oracle."""
import numpy as np
import pytest
import torch

import oracle
import paper_2608_15241_amd as lk
import workloads
from tests.gpu_helpers import dev, say
from tests.pool_helpers import make_table

pytestmark = pytest.mark.gpu


def _gpu(table, ctx, bv, rv, cap):
    pairs, n, valid = lk.local_block_version_check(dev(table), dev(ctx), dev(bv), dev(rv),
                                                   cap=cap)
    torch.cuda.synchronize()
    n = int(n.item())
    return pairs[:min(n, cap)].cpu().numpy(), n, valid.cpu().numpy()


def _compare(table, ctx, bv, rv, cap=None):
    if cap is None:
        cap = int(table.size)
    ep, en, ev = oracle.block_version_check(table, ctx, bv, rv, cap)
    gp, gn, gv = _gpu(table, ctx, bv, rv, cap)
    assert gn == en
    assert np.array_equal(gp, ep)
    assert np.array_equal(gv, ev)
    return en


@pytest.mark.parametrize("w", [workloads.TINY_DECODE, workloads.DECODE_7B,
                               workloads.PREFILL_7B, workloads.GQA_SKEW,
                               workloads.CHURN_32L], ids=lambda w: w.name)
def test_workload_metadata(w):
    say("version check", w.name)
    m = workloads.make_meta(w, seed=0)
    n = _compare(m.block_table, m.ctx_lens, m.block_version, m.req_version)
    assert n == m.stale_entries.shape[0]


def test_random_tags_and_ragged_tables():
    rng = np.random.default_rng(123)
    for trial in range(12):
        B = int(rng.integers(1, 300))
        ctx = rng.integers(0, 3000, size=B).astype(np.int32)
        ctx[rng.random(B) < 0.1] = 0
        table, num = make_table(rng, ctx, extra_blocks=5,
                                max_blocks=int((ctx.max() + 15) // 16) + int(rng.integers(1, 9)))
        rv = (rng.integers(1, 20, size=B) * 1000).astype(np.int32)
        bv = np.zeros(num, np.int32)
        for b in range(B):
            nb = (ctx[b] + 15) // 16
            bv[table[b, :nb]] = rv[b] + rng.choice([0, 0, 0, -1, 1, 7000], size=nb)
        say("version check random trial", trial, "B", B)
        _compare(table, ctx, bv, rv)


def test_truncated_list_and_full_count():
    m = workloads.make_meta(workloads.CHURN_32L, seed=1)
    for cap in (0, 1, 100, 7000):
        say("version check cap", cap)
        _compare(m.block_table, m.ctx_lens, m.block_version, m.req_version, cap=cap)


def test_everything_stale_and_empty_batch():
    rng = np.random.default_rng(5)
    ctx = np.array([1, 16, 17, 4096, 0], np.int32)
    table, num = make_table(rng, ctx)
    rv = np.array([1, 2, 3, 4, 5], np.int32)
    bv = np.full(num, 99, np.int32)
    n = _compare(table, ctx, bv, rv)
    assert n == sum((int(L) + 15) // 16 for L in ctx)
    empty = lk.local_block_version_check(dev(np.zeros((0, 4), np.int32)),
                                         dev(np.zeros(0, np.int32)),
                                         dev(np.array([1], np.int32)),
                                         dev(np.zeros(0, np.int32)), cap=4)
    torch.cuda.synchronize()
    assert int(empty[1].item()) == 0


def test_tags_are_never_written():
    m = workloads.make_meta(workloads.GQA_SKEW, seed=0)
    bv = dev(m.block_version)
    before = bv.clone()
    lk.local_block_version_check(dev(m.block_table), dev(m.ctx_lens), bv, dev(m.req_version))
    torch.cuda.synchronize()
    assert torch.equal(bv, before)


def test_small_tables():
    # Small tables: random stale tags, empty contexts, truncated lists.
    rng = np.random.default_rng(77)
    for trial in range(10):
        B = int(rng.integers(1, 33))
        mb = int(rng.integers(1, 8192 // B + 1))
        ctx = rng.integers(0, 16 * mb + 1, size=B).astype(np.int32)
        ctx[rng.random(B) < 0.15] = 0
        table, num = make_table(rng, ctx, extra_blocks=3, max_blocks=mb)
        rv = (rng.integers(1, 20, size=B) * 1000).astype(np.int32)
        bv = np.zeros(num, np.int32)
        for b in range(B):
            nb = (ctx[b] + 15) // 16
            bv[table[b, :nb]] = rv[b] + rng.choice([0, 0, 0, -1, 1], size=nb)
        say("version check small table", trial, "B", B, "mb", mb)
        n = _compare(table, ctx, bv, rv)
        for cap in (0, 1, max(0, n // 2)):
            _compare(table, ctx, bv, rv, cap=cap)
