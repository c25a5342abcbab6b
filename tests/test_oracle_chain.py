"""Pins of the oracle's layer step (oracle/chain.py): the order of its stages.

With W_q = 0 and no adapter on q, every score is 0, so the attention output
is the plain mean of V over the valid keys, and that set includes the token
the step itself appended (its value row is v = x W_v^T). The closed form
below fails if the chain attends before appending, appends k and v swapped,
routes the wrong projection into the cache, or skips the output projection.
"""
import math

import numpy as np

import oracle
import oracle.chain as ochain
from tests.pool_helpers import (BS, bits_to_f64, dense_to_pool, make_table, pool_to_dense,
                                rand_bf16)


def test_chain_with_zero_query_weights_is_mean_of_values():
    rng = np.random.default_rng(21)
    H, hq, hkv, D = 128, 2, 2, 64
    ctx = np.array([20, 37], np.int32)
    table, num = make_table(rng, ctx)
    rv = np.array([1, 2], np.int32)
    bv = np.full(num, -1, np.int32)
    for b, L in enumerate(ctx):
        bv[table[b, :(L + BS - 1) // BS]] = rv[b]
    bv[table[1, 0]] = 5                                  # request 1: block 0 stale
    kd = rand_bf16(rng, (num, hkv, BS, D))
    vd = rand_bf16(rng, (num, hkv, BS, D))
    kc, vc = dense_to_pool(kd, vd)
    x = rand_bf16(rng, (2, H))
    lw = {"W_q": np.zeros((hq * D, H), np.uint16),
          "W_k": rand_bf16(rng, (hkv * D, H), 0.05),
          "W_v": rand_bf16(rng, (hkv * D, H), 0.05),
          "W_o": rand_bf16(rng, (H, hq * D), 0.05)}
    qi = np.arange(3, dtype=np.int32)
    y, st = ochain.layer(x, lw, kc, vc, hq, hkv, D, table, qi, ctx, bv, rv,
                         np.full(2, -1, np.int32), np.zeros(2, np.float32), residual=False)
    # expected: v_new = bf16(x W_v^T) appended at position L-1, then the mean
    # of V over the valid positions, per head
    v_new = oracle.to_bf16(bits_to_f64(x) @ bits_to_f64(lw["W_v"]).T).reshape(2, hkv, D)
    _, vdense = pool_to_dense(kc, vc, num, hkv, D)      # after the chain's append
    for b, L in enumerate(ctx):
        pos = [p for p in range(L) if bv[table[b, p // BS]] == rv[b]]
        assert L - 1 in pos
        slot = vdense[table[b, (L - 1) // BS], :, (L - 1) % BS]
        assert np.array_equal(slot, v_new[b])          # the step's own v was appended
        V = bits_to_f64(vdense[table[b, np.array(pos) // BS], :, np.array(pos) % BS])
        mean = V.mean(axis=0)                           # [hkv, D]
        for h in range(hq):
            np.testing.assert_allclose(st["o"][b].reshape(hq, D)[h], mean[h // (hq // hkv)],
                                       rtol=1e-12, atol=1e-12)
        assert np.allclose(st["lse"][b], math.log(len(pos)), rtol=1e-12)
    o_b = oracle.to_bf16(st["o"])
    np.testing.assert_allclose(st["y"], bits_to_f64(o_b) @ bits_to_f64(lw["W_o"]).T,
                               rtol=1e-12, atol=1e-12)
    assert np.array_equal(y, oracle.to_bf16(st["y"]))
