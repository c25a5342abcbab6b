"""Pins of the oracle's mixed-adapter LoRA projection.

None of these retypes the oracle's loops. They compare it with what the
mathematics of LoRA fixes: the base projection as a library matmul, exact
closed forms for special adapters, and the merged-weight identity
W' = W + s * B_a A_a (the low-rank update can be folded into the base
weight, which is what makes a LoRA adapter a "delta" on a frozen base, §2.2).
"""
import numpy as np
import pytest

import oracle
from tests.pool_helpers import bits_to_f64, f32_to_bf16_bits, rand_bf16


def _setup(rng, T=7, K=64, N=48, n_ad=3, r_max=8, ranks=None):
    x = rand_bf16(rng, (T, K))
    W = rand_bf16(rng, (N, K), 0.02)
    A = rand_bf16(rng, (n_ad, r_max, K), 1 / np.sqrt(r_max))
    B = rand_bf16(rng, (n_ad, N, r_max), 0.05)
    if ranks is None:
        ranks = np.full(n_ad, r_max, dtype=np.int32)
    return x, W, A, B, np.asarray(ranks, dtype=np.int32)


def test_base_matches_numpy_matmul():
    rng = np.random.default_rng(1)
    x, W, *_ = _setup(rng, T=9, K=128, N=40)
    y = oracle.lora_linear(x, W)
    ref = bits_to_f64(x) @ bits_to_f64(W).T
    np.testing.assert_allclose(y, ref, rtol=1e-12, atol=1e-12)


def test_zero_B_is_exactly_base():
    rng = np.random.default_rng(2)
    x, W, A, B, ranks = _setup(rng)
    T = x.shape[0]
    idx = rng.integers(0, 3, size=T).astype(np.int32)
    s = np.full(T, 2.0, np.float32)
    y0 = oracle.lora_linear(x, W)
    y = oracle.lora_linear(x, W, A, np.zeros_like(B), ranks, idx, s)
    assert np.array_equal(y, y0)


def test_no_adapter_and_zero_scale_are_base():
    rng = np.random.default_rng(3)
    x, W, A, B, ranks = _setup(rng)
    T = x.shape[0]
    y0 = oracle.lora_linear(x, W)
    y1 = oracle.lora_linear(x, W, A, B, ranks, np.full(T, -1, np.int32),
                            np.full(T, 2.0, np.float32))
    y2 = oracle.lora_linear(x, W, A, B, ranks, np.zeros(T, np.int32),
                            np.zeros(T, np.float32))
    assert np.array_equal(y1, y0)
    assert np.array_equal(y2, y0)


def test_rank1_one_hot_adapter_closed_form():
    # A[a,0,:] = e_i and B[a,:,0] = e_j make the delta s * x[:, i] in column j
    # only; any transposed or shifted index moves it elsewhere.
    rng = np.random.default_rng(4)
    T, K, N, i, j, a = 5, 64, 32, 37, 11, 1
    x, W, _, _, _ = _setup(rng, T=T, K=K, N=N)
    A = np.zeros((2, 8, K), np.uint16)
    B = np.zeros((2, N, 8), np.uint16)
    one = f32_to_bf16_bits(np.array([1.0], np.float32))[0]
    A[a, 0, i] = one
    B[a, j, 0] = one
    s = np.array([2.0, -0.5, 3.0, 1.0, 0.25], np.float32)
    y = oracle.lora_linear(x, W, A, B, np.array([1, 1], np.int32),
                           np.full(T, a, np.int32), s)
    base = bits_to_f64(x) @ bits_to_f64(W).T
    expect = base.copy()
    expect[:, j] += s.astype(np.float64) * bits_to_f64(x)[:, i]
    np.testing.assert_allclose(y, expect, rtol=1e-12, atol=1e-12)


def test_merged_weight_identity_per_token():
    # Each token equals x_t (W + s_t B_a A_a)^T for its own adapter a.
    rng = np.random.default_rng(5)
    x, W, A, B, ranks = _setup(rng, T=11, K=64, N=40, n_ad=4, r_max=16,
                               ranks=[16, 16, 16, 16])
    T = x.shape[0]
    idx = np.array([0, 3, 1, -1, 2, 2, 0, 3, -1, 1, 0], np.int32)
    s = rng.uniform(0.5, 3.0, size=T).astype(np.float32)
    y = oracle.lora_linear(x, W, A, B, ranks, idx, s)
    xf, Wf, Af, Bf = map(bits_to_f64, (x, W, A, B))
    for t in range(T):
        Wm = Wf.copy()
        if idx[t] >= 0:
            Wm = Wm + float(s[t]) * (Bf[idx[t]] @ Af[idx[t]])
        np.testing.assert_allclose(y[t], xf[t] @ Wm.T, rtol=1e-10, atol=1e-10)


def test_rank_padding_is_ignored():
    # Rows of A / columns of B beyond an adapter's rank never contribute, even
    # when they hold large values.
    rng = np.random.default_rng(6)
    x, W, A, B, _ = _setup(rng, T=6, K=64, N=24, n_ad=2, r_max=16)
    ranks = np.array([3, 9], np.int32)
    A_clean, B_clean = A.copy(), B.copy()
    for a, r in enumerate(ranks):
        A_clean[a, r:] = 0
        B_clean[a, :, r:] = 0
        A[a, r:] = f32_to_bf16_bits(np.full(A[a, r:].shape, 1e3, np.float32))
        B[a, :, r:] = f32_to_bf16_bits(np.full(B[a, :, r:].shape, -7.0, np.float32))
    idx = np.array([0, 1, 1, 0, 1, 0], np.int32)
    s = np.full(6, 2.0, np.float32)
    y = oracle.lora_linear(x, W, A, B, ranks, idx, s)
    y_clean = oracle.lora_linear(x, W, A_clean, B_clean, None, idx, s)
    np.testing.assert_allclose(y, y_clean, rtol=1e-12, atol=1e-12)
    xf, Wf = bits_to_f64(x), bits_to_f64(W)
    for t in range(6):
        a, r = idx[t], ranks[idx[t]]
        Wm = Wf + 2.0 * bits_to_f64(B[a, :, :r]) @ bits_to_f64(A[a, :r])
        np.testing.assert_allclose(y[t], xf[t] @ Wm.T, rtol=1e-10, atol=1e-10)


def test_empty_batch():
    rng = np.random.default_rng(7)
    _, W, A, B, ranks = _setup(rng)
    y = oracle.lora_linear(np.zeros((0, 64), np.uint16), W, A, B, ranks,
                           np.zeros(0, np.int32), np.zeros(0, np.float32))
    assert y.shape == (0, W.shape[0])


def test_residual_is_added_as_given():
    rng = np.random.default_rng(8)
    x, W, A, B, ranks = _setup(rng, T=4, K=64, N=16)
    idx = np.array([0, 1, -1, 2], np.int32)
    s = np.full(4, 2.0, np.float32)
    res = rand_bf16(rng, (4, 16), 3.0)
    y0 = oracle.lora_linear(x, W, A, B, ranks, idx, s)
    y1 = oracle.lora_linear(x, W, A, B, ranks, idx, s, residual=res)
    np.testing.assert_allclose(y1 - y0, bits_to_f64(res), rtol=1e-12, atol=1e-12)


def test_adapter_index_out_of_range_is_base():
    rng = np.random.default_rng(9)
    x, W, A, B, ranks = _setup(rng, T=3, K=64, N=16)
    y = oracle.lora_linear(x, W, A, B, ranks, np.array([3, 7, -1], np.int32),
                           np.full(3, 2.0, np.float32))
    assert np.array_equal(y, oracle.lora_linear(x, W))


def test_rank_outside_range_is_clamped():
    # A negative rank acts as rank 0 (the base projection); a rank above r_max
    # as r_max.
    rng = np.random.default_rng(10)
    x, W, A, B, _ = _setup(rng, T=5, K=64, N=16, n_ad=2, r_max=8)
    idx = np.array([0, 1, 1, 0, 1], np.int32)
    s = np.full(5, 1.5, np.float32)
    y = oracle.lora_linear(x, W, A, B, np.array([-4, 99], np.int32), idx, s)
    base = bits_to_f64(x) @ bits_to_f64(W).T
    full = oracle.lora_linear(x, W, A, B, None, idx, s)
    np.testing.assert_allclose(y[idx == 0], base[idx == 0], rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(y[idx == 1], full[idx == 1], rtol=1e-12, atol=1e-12)
