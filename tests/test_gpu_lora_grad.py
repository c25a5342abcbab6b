"""GPU parity of the LoRA backward (local_lora_grad: dA, dB; local_lora_grad_input:
dx) against oracle.grad on the same seeded inputs: ragged token counts, every
rank tile of the kernels, many adapters, unrouted tokens, ranks below r_max
with NaN padding, T = 0, and the full size of a 4096-wide projection."""
import math

import numpy as np
import pytest
import torch

import paper_2608_15241_amd as lk
from oracle.grad import lora_grad
from tests.gpu_helpers import assert_rel, dev, dev_u16, f64, say
from tests.pool_helpers import rand_bf16

pytestmark = pytest.mark.gpu


def _inputs(rng, T, K, N, n_ad, r_max, ranks=None, neg_frac=0.15):
    if ranks is None:
        ranks = [r_max] * n_ad
    x = rand_bf16(rng, (T, K))
    dy = rand_bf16(rng, (T, N))
    W = rand_bf16(rng, (N, K), 0.02)
    A = np.zeros((n_ad, r_max, K), np.uint16)
    B = np.zeros((n_ad, N, r_max), np.uint16)
    for a, r in enumerate(ranks):
        A[a, :r] = rand_bf16(rng, (r, K), 1 / math.sqrt(max(r, 1)))
        B[a, :, :r] = rand_bf16(rng, (N, r), 0.01)
    idx = rng.integers(0, n_ad, size=T).astype(np.int32)
    idx[rng.random(T) < neg_frac] = -1
    scale = rng.uniform(0.5, 2.5, size=T).astype(np.float32)
    return x, dy, W, A, B, np.array(ranks, np.int32), idx, scale


def _grads(x, dy, A, B, rk, idx, scale):
    dA, dB = lk.local_lora_grad(dev_u16(x), dev_u16(dy), dev_u16(A), dev_u16(B), dev(rk),
                                dev(idx), dev(scale, torch.float32))
    torch.cuda.synchronize()
    return dA, dB


def _grad_input(dy, W, A, B, rk, idx, scale):
    Wt = np.ascontiguousarray(W.T)
    dx = lk.local_lora_grad_input(dev_u16(dy), dev_u16(Wt), dev_u16(A), dev_u16(B), dev(rk),
                                  dev(idx), dev(scale, torch.float32))
    torch.cuda.synchronize()
    return dx


CASES = [
    # T, K, N, n_ad, r_max, ranks
    (1, 256, 256, 3, 8, None),
    (63, 512, 256, 2, 16, None),
    (300, 512, 640, 4, 16, [16, 3, 9, 0]),
    (257, 1024, 256, 3, 24, [24, 1, 17]),
    (1000, 256, 512, 5, 32, None),
    (200, 512, 256, 2, 64, [64, 40]),
    (130, 256, 512, 2, 128, [128, 57]),
    (700, 256, 384, 40, 8, None),
    (2000, 256, 256, 256, 8, None),
    (4100, 256, 256, 1, 16, None),     # one adapter, several passes of the bucket sort
]


@pytest.mark.parametrize("case", CASES, ids=lambda c: "T%d_K%d_N%d_ad%d_r%d" % c[:5])
def test_matches_oracle(case):
    T, K, N, n_ad, r_max, ranks = case
    say("lora_grad", case)
    rng = np.random.default_rng(T * 11 + K + N + n_ad + r_max)
    x, dy, W, A, B, rk, idx, scale = _inputs(rng, T, K, N, n_ad, r_max, ranks)
    rA, rB, rdx = lora_grad(x, dy, W, A, B, rk, idx, scale)
    dA, dB = _grads(x, dy, A, B, rk, idx, scale)
    for a in range(n_ad):  # per adapter: each has its own magnitude
        if np.any(idx == a) and rk[a] > 0:
            assert_rel(f64(dA[a]), rA[a], "dA[%d]" % a)
            assert_rel(f64(dB[a]), rB[a], "dB[%d]" % a)
    # past the rank and for adapters without tokens: exact zeros
    hA, hB = f64(dA), f64(dB)
    for a in range(n_ad):
        assert not hA[a, rk[a]:].any() and not hB[a, :, rk[a]:].any(), a
        if not np.any(idx == a):
            assert not hA[a].any() and not hB[a].any(), a
    dx = _grad_input(dy, W, A, B, rk, idx, scale)
    assert_rel(f64(dx), rdx, "dx")


def test_nan_padding_beyond_rank_is_never_used():
    rng = np.random.default_rng(41)
    T, K, N, ranks = 300, 512, 256, [3, 8, 13, 16]
    x, dy, W, A, B, rk, idx, scale = _inputs(rng, T, K, N, 4, 16, ranks)
    nan = np.uint16(0x7FC0)
    for a, r in enumerate(ranks):
        A[a, r:] = nan
        B[a, :, r:] = nan
    clean_A, clean_B = A.copy(), B.copy()
    for a, r in enumerate(ranks):
        clean_A[a, r:] = 0
        clean_B[a, :, r:] = 0
    rA, rB, rdx = lora_grad(x, dy, W, clean_A, clean_B, rk, idx, scale)
    dA, dB = _grads(x, dy, A, B, rk, idx, scale)
    assert torch.isfinite(dA).all() and torch.isfinite(dB).all()
    assert_rel(f64(dA), rA, "dA")
    assert_rel(f64(dB), rB, "dB")
    dx = _grad_input(dy, W, A, B, rk, idx, scale)
    assert_rel(f64(dx), rdx, "dx")


def test_no_tokens_and_no_routed_tokens_give_zero_gradients():
    rng = np.random.default_rng(42)
    K, N = 256, 512
    x, dy, W, A, B, rk, idx, scale = _inputs(rng, 0, K, N, 3, 16)
    dA = torch.full((3, 16, K), 7.0, device="cuda")
    dB = torch.full((3, N, 16), 7.0, device="cuda")
    lk.local_lora_grad(dev_u16(x), dev_u16(dy), dev_u16(A), dev_u16(B), dev(rk), dev(idx),
                       dev(scale, torch.float32), dA=dA, dB=dB)
    torch.cuda.synchronize()
    assert not dA.any() and not dB.any()
    x, dy, W, A, B, rk, idx, scale = _inputs(rng, 150, K, N, 3, 16)
    idx[:] = -1
    idx[::7] = 3  # out of range: unrouted too
    dA, dB = _grads(x, dy, A, B, rk, idx, scale)
    assert not dA.any() and not dB.any()


def test_deterministic_and_workspace_reuse():
    rng = np.random.default_rng(43)
    x, dy, W, A, B, rk, idx, scale = _inputs(rng, 900, 512, 512, 6, 16)
    args = (dev_u16(x), dev_u16(dy), dev_u16(A), dev_u16(B), dev(rk), dev(idx),
            dev(scale, torch.float32))
    ws = lk.Workspace()
    c1 = lk.prepare_lora_grad(*args, workspace=ws)
    dA1, dB1 = (t.clone() for t in c1())
    # another call through the same workspace in between
    x2, dy2, _, A2, B2, rk2, idx2, s2 = _inputs(rng, 300, 256, 256, 2, 8)
    lk.local_lora_grad(dev_u16(x2), dev_u16(dy2), dev_u16(A2), dev_u16(B2), dev(rk2),
                       dev(idx2), dev(s2, torch.float32), workspace=ws)
    dA2, dB2 = c1()
    torch.cuda.synchronize()
    assert torch.equal(dA1, dA2) and torch.equal(dB1, dB2)


def test_full_size_projection():
    # a 4096 x 4096 projection, 2048 tokens over 8 rank-16 adapters
    T, K, N, n_ad, r_max = 2048, 4096, 4096, 8, 16
    say("lora_grad full size", T, K, N, n_ad, r_max)
    rng = np.random.default_rng(44)
    x, dy, W, A, B, rk, idx, scale = _inputs(rng, T, K, N, n_ad, r_max, neg_frac=0.05)
    rA, rB, rdx = lora_grad(x, dy, W, A, B, rk, idx, scale)
    dA, dB = _grads(x, dy, A, B, rk, idx, scale)
    for a in range(n_ad):
        assert_rel(f64(dA[a]), rA[a], "dA[%d]" % a)
        assert_rel(f64(dB[a]), rB[a], "dB[%d]" % a)
    dx = _grad_input(dy, W, A, B, rk, idx, scale)
    assert_rel(f64(dx), rdx, "dx")


@pytest.mark.parametrize("T,Ns,ranks", [
    (300, (512, 128, 128), ([16, 3, 9, 0], [16, 16, 16, 16], None)),
    (1000, (256, 256, 384, 128), ([16, 8, 1, 12], None, [4, 4, 16, 2], [16, 16, 16, 16])),
    (0, (256, 128), (None, None)),
], ids=["qkv", "four", "empty"])
def test_grouped_matches_oracle(T, Ns, ranks):
    # q/k/v-like projections of one x: each projection against the oracle
    say("lora_grad grouped", T, Ns)
    rng = np.random.default_rng(T + sum(Ns))
    K, n_ad, r_max = 512, 4, 16
    x = rand_bf16(rng, (T, K))
    idx = rng.integers(0, n_ad, size=T).astype(np.int32)
    idx[rng.random(T) < 0.15] = -1
    scale = rng.uniform(0.5, 2.5, size=T).astype(np.float32)
    dys, As, Bs, rks, Ws = [], [], [], [], []
    for g, N in enumerate(Ns):
        rk = ranks[g] if ranks[g] is not None else [r_max] * n_ad
        _, dy, W, A, B, r, _, _ = _inputs(rng, T, K, N, n_ad, r_max, rk)
        dys.append(dy), As.append(A), Bs.append(B), rks.append(r), Ws.append(W)
    dev_r = [dev(rks[g]) if ranks[g] is not None else None for g in range(len(Ns))]
    dAs, dBs = lk.local_lora_grad_grouped(dev_u16(x), [dev_u16(d) for d in dys],
                                          [dev_u16(a) for a in As], [dev_u16(b) for b in Bs],
                                          dev_r, dev(idx), dev(scale, torch.float32))
    torch.cuda.synchronize()
    for g in range(len(Ns)):
        rA, rB, _ = lora_grad(x, dys[g], Ws[g], As[g], Bs[g], rks[g], idx, scale)
        for a in range(n_ad):
            if np.any(idx == a) and rks[g][a] > 0:
                assert_rel(f64(dAs[g][a]), rA[a], "dA[%d][%d]" % (g, a))
                assert_rel(f64(dBs[g][a]), rB[a], "dB[%d][%d]" % (g, a))
            else:
                assert not f64(dAs[g][a]).any() and not f64(dBs[g][a]).any(), (g, a)
