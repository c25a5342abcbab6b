"""Pins of the oracle's paged attention and KV append.

References that are not the oracle: torch's float64 CPU scaled-dot-product
attention over KV gathered with numpy reshapes of the documented pool layout,
closed forms (uniform scores give the mean of V, one key gives its V row,
no key gives zero output), and invariances (physical block permutation,
stale exclusion equal to deleting the stale tokens, chunking of prefill).
"""
import math

import numpy as np
import pytest
import torch

import oracle
from tests.pool_helpers import (BS, bits_to_f64, dense_to_pool, gather_request,
                                make_table, pool_to_dense, rand_bf16)


def _pool(rng, num, hkv, D):
    kd = rand_bf16(rng, (num, hkv, BS, D))
    vd = rand_bf16(rng, (num, hkv, BS, D))
    return kd, vd


def _valid_tags(table, ctx, rv, num):
    bv = np.full(num, -5, np.int32)
    for b, L in enumerate(ctx):
        bv[table[b, :(L + BS - 1) // BS]] = rv[b]
    return bv


def _sdpa_reference(q, q_indptr, ctx, kd, vd, table, bv, rv, Hq, Hkv, D, scale):
    """torch float64 SDPA per request over gathered dense K/V with a mask."""
    T = q.shape[0]
    out = np.zeros((T, Hq, D))
    lse = np.full((T, Hq), -np.inf)
    qf = bits_to_f64(q).reshape(T, Hq, D)
    for b in range(len(ctx)):
        L = int(ctx[b])
        r0, r1 = int(q_indptr[b]), int(q_indptr[b + 1])
        n = r1 - r0
        if n == 0:
            continue
        pos = np.arange(L)
        keep = bv[table[b, pos // BS]] == rv[b] if L else np.zeros(0, bool)
        qpos = L - n + np.arange(n)
        mask = (pos[None, :] <= qpos[:, None]) & keep[None, :]   # [n, L]
        for h in range(Hq):
            g = h // (Hq // Hkv)
            K, V = gather_request(kd, vd, table, b, L, g)
            qt = torch.from_numpy(qf[r0:r1, h])                  # [n, D]
            Kt, Vt = torch.from_numpy(K), torch.from_numpy(V)
            m = torch.from_numpy(mask)
            rows = m.any(dim=1)
            if rows.any():
                o = torch.nn.functional.scaled_dot_product_attention(
                    qt[rows][None], Kt[None], Vt[None], attn_mask=m[rows][None],
                    scale=scale)[0]
                out[r0:r1][rows.numpy(), h] = o.numpy()
                s = (qt[rows] @ Kt.T) * scale
                s = s.masked_fill(~m[rows], -math.inf)
                lse[r0:r1][rows.numpy(), h] = torch.logsumexp(s, dim=1).numpy()
    return out, lse


def _run(q, q_indptr, ctx, kd, vd, table, bv, rv, Hq, Hkv, D, scale):
    kc, vc = dense_to_pool(kd, vd)
    return oracle.paged_attn(q, q_indptr, Hq, Hkv, D, kc, vc, table, ctx, bv, rv, scale)


@pytest.mark.parametrize("Hq,Hkv,D", [(4, 4, 64), (8, 2, 128), (6, 3, 64)])
def test_decode_matches_torch_sdpa(Hq, Hkv, D):
    rng = np.random.default_rng(Hq * 100 + D)
    ctx = np.array([1, 16, 17, 45, 96, 130], np.int32)
    table, num = make_table(rng, ctx, extra_blocks=2)
    rv = np.array([1000, 2000, 1000, 3000, 2000, 1000], np.int32)
    bv = _valid_tags(table, ctx, rv, num)
    # stale a few interior blocks, with older and newer tags
    bv[table[3, 1]] = rv[3] - 1
    bv[table[5, 0]] = rv[5] + 1
    bv[table[5, 3]] = rv[5] - 1
    kd, vd = _pool(rng, num, Hkv, D)
    q = rand_bf16(rng, (len(ctx), Hq, D))
    qi = np.arange(len(ctx) + 1, dtype=np.int32)
    scale = 1 / math.sqrt(D)
    out, lse = _run(q, qi, ctx, kd, vd, table, bv, rv, Hq, Hkv, D, scale)
    ref, ref_lse = _sdpa_reference(q, qi, ctx, kd, vd, table, bv, rv, Hq, Hkv, D, scale)
    np.testing.assert_allclose(out, ref, rtol=1e-9, atol=1e-10)
    np.testing.assert_allclose(lse, ref_lse, rtol=1e-9, atol=1e-10)


def test_prefill_causal_matches_torch_sdpa():
    rng = np.random.default_rng(42)
    Hq, Hkv, D = 4, 2, 64
    prefix = np.array([0, 20, 33], np.int32)
    n_new = np.array([5, 17, 3], np.int32)
    ctx = prefix + n_new
    table, num = make_table(rng, ctx)
    rv = np.array([10, 20, 30], np.int32)
    bv = _valid_tags(table, ctx, rv, num)
    bv[table[1, 0]] = 19            # stale prefix block of request 1
    kd, vd = _pool(rng, num, Hkv, D)
    qi = np.concatenate([[0], np.cumsum(n_new)]).astype(np.int32)
    q = rand_bf16(rng, (int(qi[-1]), Hq, D))
    out, lse = _run(q, qi, ctx, kd, vd, table, bv, rv, Hq, Hkv, D, 0.125)
    ref, ref_lse = _sdpa_reference(q, qi, ctx, kd, vd, table, bv, rv, Hq, Hkv, D, 0.125)
    np.testing.assert_allclose(out, ref, rtol=1e-9, atol=1e-10)
    np.testing.assert_allclose(lse, ref_lse, rtol=1e-9, atol=1e-10)


def test_uniform_scores_give_mean_of_valid_v():
    # q = 0 makes every score 0: out is the plain mean of V over the valid
    # keys and lse = log(#valid keys).
    rng = np.random.default_rng(3)
    Hq = Hkv = 2
    D = 64
    ctx = np.array([16, 50], np.int32)       # one block; four blocks
    table, num = make_table(rng, ctx)
    rv = np.array([1, 2], np.int32)
    bv = _valid_tags(table, ctx, rv, num)
    bv[table[1, 2]] = 7                      # stale block: tokens 32..47
    kd, vd = _pool(rng, num, Hkv, D)
    q = np.zeros((2, Hq, D), np.uint16)
    out, lse = _run(q, np.arange(3, dtype=np.int32), ctx, kd, vd, table, bv, rv,
                    Hq, Hkv, D, 0.1)
    for b, L in enumerate(ctx):
        keep = [pi for pi in range(L) if bv[table[b, pi // BS]] == rv[b]]
        for h in range(Hq):
            V = bits_to_f64(vd[table[b, np.array(keep) // BS], h, np.array(keep) % BS])
            np.testing.assert_allclose(out[b, h], V.mean(axis=0), rtol=1e-12, atol=1e-13)
            assert lse[b, h] == pytest.approx(math.log(len(keep)), rel=1e-12)


def test_single_valid_key_returns_its_value_row():
    rng = np.random.default_rng(4)
    Hq, Hkv, D = 4, 1, 128
    ctx = np.array([33], np.int32)           # blocks 0,1 stale; block 2 has 1 key
    table, num = make_table(rng, ctx)
    rv = np.array([5], np.int32)
    bv = np.full(num, 4, np.int32)
    bv[table[0, 2]] = 5
    kd, vd = _pool(rng, num, Hkv, D)
    q = rand_bf16(rng, (1, Hq, D))
    out, lse = _run(q, np.array([0, 1], np.int32), ctx, kd, vd, table, bv, rv,
                    Hq, Hkv, D, 0.2)
    p, s = table[0, 2], 0
    V = bits_to_f64(vd[p, 0, s])
    K = bits_to_f64(kd[p, 0, s])
    for h in range(Hq):
        np.testing.assert_array_equal(out[0, h], V)
        assert lse[0, h] == pytest.approx(0.2 * float(bits_to_f64(q[0, h]) @ K), rel=1e-12)


def test_fully_stale_gives_zero_and_minus_inf():
    rng = np.random.default_rng(5)
    Hq, Hkv, D = 2, 2, 64
    ctx = np.array([40, 7], np.int32)
    table, num = make_table(rng, ctx)
    rv = np.array([3, 4], np.int32)
    bv = np.full(num, 99, np.int32)
    kd, vd = _pool(rng, num, Hkv, D)
    q = rand_bf16(rng, (2, Hq, D))
    out, lse = _run(q, np.arange(3, dtype=np.int32), ctx, kd, vd, table, bv, rv,
                    Hq, Hkv, D, 0.1)
    assert np.all(out == 0.0)
    assert np.all(np.isneginf(lse))


def test_stale_exclusion_equals_deleting_stale_tokens():
    # Attention with stale blocks masked equals attention over a new request
    # that holds only the surviving blocks (a shorter, all-valid context).
    rng = np.random.default_rng(6)
    Hq, Hkv, D = 4, 2, 64
    ctx = np.array([80], np.int32)            # 5 full blocks
    table, num = make_table(rng, ctx)
    rv = np.array([9], np.int32)
    bv = _valid_tags(table, ctx, rv, num)
    bv[table[0, 1]] = 8
    bv[table[0, 3]] = 8
    kd, vd = _pool(rng, num, Hkv, D)
    q = rand_bf16(rng, (1, Hq, D))
    qi = np.array([0, 1], np.int32)
    out, lse = _run(q, qi, ctx, kd, vd, table, bv, rv, Hq, Hkv, D, 0.125)
    keep = table[0, [0, 2, 4]][None, :]
    out2, lse2 = _run(q, qi, np.array([48], np.int32), kd, vd, keep, bv, rv,
                      Hq, Hkv, D, 0.125)
    np.testing.assert_allclose(out, out2, rtol=1e-13, atol=1e-14)
    np.testing.assert_allclose(lse, lse2, rtol=1e-13)


def test_physical_block_permutation_invariance():
    rng = np.random.default_rng(7)
    Hq, Hkv, D = 4, 4, 64
    ctx = np.array([30, 64, 5], np.int32)
    table, num = make_table(rng, ctx)
    rv = np.array([1, 2, 3], np.int32)
    bv = _valid_tags(table, ctx, rv, num)
    bv[table[1, 2]] = 0
    kd, vd = _pool(rng, num, Hkv, D)
    q = rand_bf16(rng, (3, Hq, D))
    qi = np.arange(4, dtype=np.int32)
    out, lse = _run(q, qi, ctx, kd, vd, table, bv, rv, Hq, Hkv, D, 0.1)
    perm = rng.permutation(num)             # new id of old block p = perm[p]
    kd2, vd2, bv2 = np.empty_like(kd), np.empty_like(vd), np.empty_like(bv)
    kd2[perm], vd2[perm], bv2[perm] = kd, vd, bv
    table2 = perm[table].astype(np.int32)
    out2, lse2 = _run(q, qi, ctx, kd2, vd2, table2, bv2, rv, Hq, Hkv, D, 0.1)
    np.testing.assert_array_equal(out, out2)
    np.testing.assert_array_equal(lse, lse2)


def test_gqa_head_to_group_mapping():
    # V constant g+1 in KV head g and q = 0: query head h must return
    # h // (Hq/Hkv) + 1, which fails for any other grouping.
    Hq, Hkv, D = 8, 2, 64
    rng = np.random.default_rng(8)
    ctx = np.array([20], np.int32)
    table, num = make_table(rng, ctx)
    rv = np.array([1], np.int32)
    bv = _valid_tags(table, ctx, rv, num)
    kd = rand_bf16(rng, (num, Hkv, BS, D))
    vd = np.zeros((num, Hkv, BS, D), np.uint16)
    from tests.pool_helpers import f32_to_bf16_bits
    for g in range(Hkv):
        vd[:, g] = f32_to_bf16_bits(np.full((num, BS, D), g + 1.0, np.float32))
    q = np.zeros((1, Hq, D), np.uint16)
    out, _ = _run(q, np.array([0, 1], np.int32), ctx, kd, vd, table, bv, rv,
                  Hq, Hkv, D, 0.1)
    for h in range(Hq):
        np.testing.assert_allclose(out[0, h], h // (Hq // Hkv) + 1.0, rtol=1e-14)


def test_lse_normalises_the_weights():
    rng = np.random.default_rng(9)
    Hq = Hkv = 1
    D = 64
    ctx = np.array([37], np.int32)
    table, num = make_table(rng, ctx)
    rv = np.array([1], np.int32)
    bv = _valid_tags(table, ctx, rv, num)
    kd, vd = _pool(rng, num, Hkv, D)
    q = rand_bf16(rng, (1, Hq, D))
    _, lse = _run(q, np.array([0, 1], np.int32), ctx, kd, vd, table, bv, rv,
                  Hq, Hkv, D, 0.3)
    K, _ = gather_request(kd, vd, table, 0, 37, 0)
    s = 0.3 * (K @ bits_to_f64(q[0, 0]))
    assert np.exp(s - lse[0, 0]).sum() == pytest.approx(1.0, rel=1e-12)


def _append_then_attend(kd, vd, table, prefix, chunks, q_rows, k_rows, v_rows, rv, bv,
                        Hq, Hkv, D, scale):
    """Run successive chunks: append each chunk then attend its queries."""
    num = kd.shape[0]
    kc, vc = dense_to_pool(kd, vd)
    outs, lses = [], []
    done = 0
    pos = prefix
    for n in chunks:
        qi = np.array([0, n], np.int32)
        ctx = np.array([pos + n], np.int32)
        oracle.kv_append(kc, vc, Hkv, D, table, qi, ctx, k_rows[done:done + n],
                         v_rows[done:done + n])
        o, l = oracle.paged_attn(q_rows[done:done + n], qi, Hq, Hkv, D, kc, vc,
                                 table, ctx, bv, rv, scale)
        outs.append(o)
        lses.append(l)
        done += n
        pos += n
    return np.concatenate(outs), np.concatenate(lses), kc, vc


def test_prefill_chunking_and_decode_equivalence():
    # One 24-token chunk == two 12-token chunks == 24 one-token decode steps.
    rng = np.random.default_rng(10)
    Hq, Hkv, D = 4, 2, 64
    prefix, n = 19, 24
    ctx_end = np.array([prefix + n], np.int32)
    table, num = make_table(rng, ctx_end)
    rv = np.array([4], np.int32)
    bv = _valid_tags(table, ctx_end, rv, num)
    bv[table[0, 0]] = 3
    kd, vd = _pool(rng, num, Hkv, D)
    q = rand_bf16(rng, (n, Hq, D))
    kn = rand_bf16(rng, (n, Hkv, D))
    vn = rand_bf16(rng, (n, Hkv, D))
    args = (q, kn, vn, rv, bv, Hq, Hkv, D, 0.125)
    o1, l1, kc1, vc1 = _append_then_attend(kd, vd, table, prefix, [24], *args)
    o2, l2, kc2, vc2 = _append_then_attend(kd, vd, table, prefix, [12, 12], *args)
    o3, l3, kc3, vc3 = _append_then_attend(kd, vd, table, prefix, [1] * 24, *args)
    for o, l in ((o2, l2), (o3, l3)):
        np.testing.assert_array_equal(o, o1)
        np.testing.assert_array_equal(l, l1)
    assert np.array_equal(kc1, kc2) and np.array_equal(kc1, kc3)
    assert np.array_equal(vc1, vc3)


def test_kv_append_writes_documented_slots():
    rng = np.random.default_rng(12)
    Hkv, D = 2, 64
    ctx = np.array([18, 33], np.int32)
    n_new = np.array([3, 1], np.int32)
    table, num = make_table(rng, ctx)
    kd, vd = _pool(rng, num, Hkv, D)
    kc, vc = dense_to_pool(kd, vd)
    qi = np.array([0, 3, 4], np.int32)
    kn = rand_bf16(rng, (4, Hkv, D))
    vn = rand_bf16(rng, (4, Hkv, D))
    oracle.kv_append(kc, vc, Hkv, D, table, qi, ctx, kn, vn)
    kd2, vd2 = pool_to_dense(kc, vc, num, Hkv, D)
    written = {}
    for b in range(2):
        for i in range(n_new[b]):
            pos = ctx[b] - n_new[b] + i
            written[(table[b, pos // BS], pos % BS)] = qi[b] + i
    for p in range(num):
        for s in range(BS):
            if (p, s) in written:
                r = written[(p, s)]
                assert np.array_equal(kd2[p, :, s], kn[r])
                assert np.array_equal(vd2[p, :, s], vn[r])
            else:
                assert np.array_equal(kd2[p, :, s], kd[p, :, s])
                assert np.array_equal(vd2[p, :, s], vd[p, :, s])


def test_out_of_range_id_equals_stale_block():
    # An id outside the pool excludes its block exactly like a stale tag.
    rng = np.random.default_rng(13)
    Hq, Hkv, D = 4, 2, 64
    ctx = np.array([40], np.int32)
    table, num = make_table(rng, ctx)
    rv = np.array([3], np.int32)
    bv = _valid_tags(table, ctx, rv, num)
    kd, vd = _pool(rng, num, Hkv, D)
    q = rand_bf16(rng, (1, Hq, D))
    qi = np.array([0, 1], np.int32)
    bad = table.copy()
    bad[0, 1] = num + 5
    out1, lse1 = _run(q, qi, ctx, kd, vd, bad, bv, rv, Hq, Hkv, D, 0.125)
    bv2 = bv.copy()
    bv2[table[0, 1]] = 2
    out2, lse2 = _run(q, qi, ctx, kd, vd, table, bv2, rv, Hq, Hkv, D, 0.125)
    np.testing.assert_array_equal(out1, out2)
    np.testing.assert_array_equal(lse1, lse2)
