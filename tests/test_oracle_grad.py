"""Pins of the LoRA-backward oracle against the forward definition: the loss
L = sum(dy * y) is linear in each of A, B and x separately (y is computed by the
forward oracle in float64 from the bf16 inputs, with no intermediate rounding),
so moving one entry between two bf16 values changes L by exactly the gradient
times the step. Plus special cases that reduce to plain products."""
import numpy as np

import oracle
from oracle.grad import lora_grad


def bf(a):
    return oracle.to_bf16(np.asarray(a, dtype=np.float64))


def case(rng, T=12, K=32, N=24, n_ad=3, r_max=8, ranks=(8, 5, 0)):
    x = bf(rng.normal(size=(T, K)))
    dy = bf(rng.normal(size=(T, N)))
    W = bf(rng.normal(size=(N, K)) * 0.1)
    A = bf(rng.normal(size=(n_ad, r_max, K)) * 0.3)
    B = bf(rng.normal(size=(n_ad, N, r_max)) * 0.3)
    idx = rng.integers(-1, n_ad + 1, size=T).astype(np.int32)  # includes -1 and n_ad
    idx[:3] = [0, 1, 0]
    scale = rng.uniform(0.5, 2.0, size=T).astype(np.float32)
    return x, dy, W, A, B, np.asarray(ranks, np.int32), idx, scale


def loss(dy, x, W, A, B, ranks, idx, scale):
    y = oracle.lora_linear(x, W, A, B, ranks, idx, scale)
    return float((oracle.bf16_to_f64(dy) * y).sum())


def bump(arr, pos):
    """arr with entry pos moved to the next bf16 value away from zero, and the step."""
    out = arr.copy()
    v = float(oracle.bf16_to_f64(arr[pos:pos + 1] if np.ndim(pos) == 0 else arr[pos][None])[0])
    out[pos] = arr[pos] + 1 if (arr[pos] & 0x7fff) != 0x7f7f else arr[pos] - 1
    return out, float(oracle.bf16_to_f64(out[pos][None])[0]) - v


def test_gradients_are_the_derivatives_of_the_forward():
    rng = np.random.default_rng(3)
    x, dy, W, A, B, ranks, idx, scale = case(rng)
    dA, dB, dx = lora_grad(x, dy, W, A, B, ranks, idx, scale)
    L0 = loss(dy, x, W, A, B, ranks, idx, scale)
    for _ in range(12):
        a, j, k = rng.integers(0, 3), rng.integers(0, 8), rng.integers(0, 32)
        A1, h = bump(A, (a, j, k))
        d = (loss(dy, x, W, A1, B, ranks, idx, scale) - L0) / h
        assert abs(d - dA[a, j, k]) <= 1e-7 * max(1.0, abs(d)), (a, j, k)
        a, n, j = rng.integers(0, 3), rng.integers(0, 24), rng.integers(0, 8)
        B1, h = bump(B, (a, n, j))
        d = (loss(dy, x, W, A, B1, ranks, idx, scale) - L0) / h
        assert abs(d - dB[a, n, j]) <= 1e-7 * max(1.0, abs(d)), (a, n, j)
        t, k = rng.integers(0, 12), rng.integers(0, 32)
        x1, h = bump(x, (t, k))
        d = (loss(dy, x1, W, A, B, ranks, idx, scale) - L0) / h
        assert abs(d - dx[t, k]) <= 1e-7 * max(1.0, abs(d)), (t, k)


def test_padding_ranks_and_unrouted_tokens():
    rng = np.random.default_rng(4)
    x, dy, W, A, B, ranks, idx, scale = case(rng)
    dA, dB, dx = lora_grad(x, dy, W, A, B, ranks, idx, scale)
    assert dA[0].any() and np.all(dA[1, 5:] == 0) and np.all(dB[1, :, 5:] == 0)
    assert np.all(dA[2] == 0) and np.all(dB[2] == 0)          # rank 0: no gradient
    plain = ~((idx >= 0) & (idx < 2))                          # rank-0 adapter, -1, out of range
    base = oracle.bf16_to_f64(dy) @ oracle.bf16_to_f64(W)
    assert np.allclose(dx[plain], base[plain], rtol=0, atol=1e-12)


def test_one_adapter_reduces_to_plain_products():
    # every token on adapter 0 with scale 1: dB = dy^T (x A^T), dA = (dy B)^T x
    rng = np.random.default_rng(5)
    x, dy, W, A, B, ranks, idx, scale = case(rng, ranks=(8, 8, 8))
    idx[:] = 0
    scale[:] = 1.0
    dA, dB, dx = lora_grad(x, dy, W, A, B, ranks, idx, scale)
    X, DY, Af, Bf = (oracle.bf16_to_f64(v) for v in (x, dy, A[0], B[0]))
    assert np.allclose(dB[0], DY.T @ (X @ Af.T), rtol=1e-12, atol=1e-12)
    assert np.allclose(dA[0], (DY @ Bf).T @ X, rtol=1e-12, atol=1e-12)
    assert not dA[1].any() and not dB[1].any()
