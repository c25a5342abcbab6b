"""Pins of the oracle's version check.

Hand-worked cases, the two extreme cases, and a token-level brute force (a
different counting than the oracle's block-level loop). The generator's own
bookkeeping of which entries it staled is a further independent record.
"""
import numpy as np

import oracle
import workloads
from tests.golden import load_golden
from tests.pool_helpers import make_table


def _check(table, ctx, bv, rv, cap=None):
    return oracle.block_version_check(table, ctx, bv, rv, cap)


def test_hand_example_partial_block():
    # L = 17 covers two blocks (16 + 1 live tokens); staling block 1 leaves 16.
    table = np.array([[5, 2]], np.int32)
    bv = np.array([7, 7, 6, 7, 7, 7], np.int32)
    pairs, n, valid = _check(table, [17], bv, [7])
    assert n == 1 and pairs.tolist() == [[0, 1]] and valid.tolist() == [16]


def test_golden_cases():
    for case in load_golden("version_check_cases.json"):
        pairs, n, valid = _check(np.array(case["block_table"], np.int32),
                                 case["ctx_lens"], case["block_version"],
                                 case["req_version"])
        assert n == case["n_stale"], case["name"]
        assert pairs.tolist() == case["stale_pairs"], case["name"]
        assert valid.tolist() == case["valid_tokens"], case["name"]


def test_all_valid_and_fully_stale():
    rng = np.random.default_rng(0)
    ctx = [1, 15, 16, 17, 100, 256]
    table, num = make_table(rng, ctx)
    rv = np.arange(len(ctx), dtype=np.int32) * 10 + 10
    bv = np.zeros(num, np.int32)
    for b, L in enumerate(ctx):
        bv[table[b, :(L + 15) // 16]] = rv[b]
    pairs, n, valid = _check(table, ctx, bv, rv)
    assert n == 0 and valid.tolist() == ctx
    pairs, n, valid = _check(table, ctx, bv + 1, rv)   # every tag newer
    expect = [[b, j] for b, L in enumerate(ctx) for j in range((L + 15) // 16)]
    assert n == len(expect) and pairs.tolist() == expect
    assert valid.tolist() == [0] * len(ctx)


def test_token_level_brute_force():
    rng = np.random.default_rng(11)
    for trial in range(20):
        B = int(rng.integers(1, 9))
        ctx = rng.integers(0, 200, size=B)
        table, num = make_table(rng, ctx, extra_blocks=3)
        rv = rng.integers(1, 5, size=B).astype(np.int32) * 100
        bv = rng.integers(0, 6, size=num).astype(np.int32) * 100
        # some blocks match exactly, some older, some newer
        pairs, n, valid = _check(table, ctx, bv, rv)
        v_bf = [sum(1 for pi in range(int(L)) if bv[table[b, pi // 16]] == rv[b])
                for b, L in enumerate(ctx)]
        stale_bf = sorted({(b, pi // 16) for b, L in enumerate(ctx)
                           for pi in range(int(L)) if bv[table[b, pi // 16]] != rv[b]})
        assert valid.tolist() == v_bf
        assert n == len(stale_bf)
        assert [tuple(p) for p in pairs.tolist()] == stale_bf


def test_truncated_list_reports_full_count():
    table = np.array([[0, 1, 2], [3, 4, 5]], np.int32)
    bv = np.array([1, 1, 1, 9, 9, 9], np.int32)
    pairs, n, valid = _check(table, [48, 40], bv, [2, 2], cap=4)
    assert n == 6
    assert pairs.tolist() == [[0, 0], [0, 1], [0, 2], [1, 0]]
    assert valid.tolist() == [0, 0]


def test_empty_context_and_empty_batch():
    pairs, n, valid = _check(np.zeros((2, 1), np.int32), [0, 0],
                             np.array([3], np.int32), [1, 2])
    assert n == 0 and valid.tolist() == [0, 0]
    pairs, n, valid = _check(np.zeros((0, 1), np.int32), [], np.array([3], np.int32), [])
    assert n == 0 and valid.shape == (0,)


def test_churn_workload_matches_generator_record():
    # The 32-layer churn workload stales 10% of its block-table entries. The
    # generator records which; the oracle must recover exactly that list, and
    # the per-request valid count is the context minus the staled blocks'
    # 16 tokens each (the last block is never staled).
    w = workloads.CHURN_32L
    m = workloads.make_meta(w, seed=0)
    pairs, n, valid = _check(m.block_table, m.ctx_lens, m.block_version, m.req_version)
    assert n == round(0.1 * m.num_blocks) == m.stale_entries.shape[0]
    assert np.array_equal(pairs, m.stale_entries)
    per_req = np.bincount(m.stale_entries[:, 0], minlength=m.B)
    assert np.array_equal(valid, m.ctx_lens - 16 * per_req)


def test_out_of_range_ids_and_table_width():
    # An id outside [0, num_blocks) is stale and never read; a request owns at
    # most max_blocks blocks even if its context says more.
    table = np.array([[0, 7, 1], [2, -3, 3]], np.int32)
    bv = np.array([5, 5, 6, 6], np.int32)           # num_blocks = 4
    pairs, n, valid = _check(table, [48, 64], bv, [5, 6])
    assert pairs.tolist() == [[0, 1], [1, 1]] and n == 2
    assert valid.tolist() == [32, 32]               # request 1 owns 3 of 4 blocks
