"""GPU parity of local_lora_linear against the oracle, plus exact
self-consistency (a zero up-projection changes nothing, bit for bit)."""
import math

import numpy as np
import pytest
import torch

import oracle
import paper_2608_15241_amd as lk
from tests.gpu_helpers import assert_rel, dev, dev_u16, f64, host_u16, say
from tests.pool_helpers import rand_bf16

pytestmark = pytest.mark.gpu


def _inputs(rng, T, K, N, n_ad, r_max, ranks=None, neg_frac=0.15):
    x = rand_bf16(rng, (T, K))
    W = rand_bf16(rng, (N, K), 0.02)
    if n_ad == 0:
        return x, W, None, None, None, None, None
    if ranks is None:
        ranks = [r_max] * n_ad
    A = np.zeros((n_ad, r_max, K), np.uint16)
    B = np.zeros((n_ad, N, r_max), np.uint16)
    for a, r in enumerate(ranks):
        A[a, :r] = rand_bf16(rng, (r, K), 1 / math.sqrt(max(r, 1)))
        B[a, :, :r] = rand_bf16(rng, (N, r), 0.01)
    idx = rng.integers(0, n_ad, size=T).astype(np.int32)
    idx[rng.random(T) < neg_frac] = -1
    scale = np.full(T, 2.0, np.float32)
    return x, W, A, B, np.array(ranks, np.int32), idx, scale


def _run_gpu(x, W, A, B, ranks, idx, scale, residual=None):
    args = [dev_u16(x), dev_u16(W)]
    kw = {}
    if A is not None:
        kw = dict(A=dev_u16(A), B=dev_u16(B), ranks=dev(ranks), adapter_idx=dev(idx),
                  scale=dev(scale, torch.float32))
    if residual is not None:
        kw["residual"] = dev_u16(residual)
    y = lk.local_lora_linear(*args, **kw)
    torch.cuda.synchronize()
    return y


CASES = [
    # T, K, N, n_ad, r_max, ranks
    (1, 256, 256, 3, 8, None),
    (5, 512, 256, 4, 16, None),
    (32, 1024, 512, 8, 16, None),
    (33, 256, 320, 3, 8, None),
    (64, 512, 1024, 16, 64, [8, 16, 32, 64] * 4),
    (100, 256, 512, 3, 8, None),
    (128, 512, 512, 32, 16, None),
    (257, 512, 256, 4, 16, None),
    (300, 512, 640, 4, 16, [16, 3, 9, 16]),
    (1000, 256, 512, 4, 16, None),
    (256, 512, 256, 2, 128, [128, 57]),
    (200, 1024, 256, 5, 32, [32, 1, 17, 32, 24]),
    (40, 4160, 256, 5, 16, None),
    (64, 4096, 512, 16, 64, [8, 16, 32, 64] * 4),
    (24, 2048, 256, 2, 128, [128, 100]),
    (128, 512, 256, 16, 32, [32, 8, 24, 16] * 4),
    (16, 512, 64, 16, 16, None),
    (32, 1024, 4096, 8, 16, None),
    (64, 512, 3072, 16, 32, None),
    (64, 512, 512, 0, 0, None),
    (700, 256, 384, 0, 0, None),
    # long chunks: the shrink's rank tiles (r_max 8 padded to 16, 24, 128),
    # a K of 65 steps (5 slices), many adapters inside one 32-token tile
    (513, 512, 512, 3, 8, None),
    (300, 256, 256, 5, 24, [24, 1, 17, 0, 24]),
    (400, 1024, 256, 2, 128, [128, 57]),
    (600, 4160, 256, 16, 64, [8, 16, 32, 64] * 4),
]


@pytest.mark.parametrize("case", CASES, ids=lambda c: "T%d_K%d_N%d_ad%d_r%d" % c[:5])
def test_matches_oracle(case):
    T, K, N, n_ad, r_max, ranks = case
    say("lora_linear", case)
    rng = np.random.default_rng(T * 7 + K + N + n_ad)
    x, W, A, B, rk, idx, scale = _inputs(rng, T, K, N, n_ad, r_max, ranks)
    y = _run_gpu(x, W, A, B, rk, idx, scale)
    ref = oracle.lora_linear(x, W, A, B, rk, idx, scale)
    assert_rel(f64(y), ref, "y")
    # the adapter delta itself (y - base) must also match where adapters apply
    if n_ad:
        base = oracle.lora_linear(x, W)
        rows = idx >= 0
        if rows.any():
            y0 = _run_gpu(x, W, None, None, None, None, None)
            assert_rel(f64(y)[rows] - f64(y0)[rows], (ref - base)[rows], "delta", tol=5e-2)


def test_random_scales_and_residual():
    rng = np.random.default_rng(9)
    T, K, N = 48, 512, 256
    x, W, A, B, rk, idx, _ = _inputs(rng, T, K, N, 5, 16)
    scale = rng.uniform(-3, 3, size=T).astype(np.float32)
    res = rand_bf16(rng, (T, N), 1.5)
    y = _run_gpu(x, W, A, B, rk, idx, scale, residual=res)
    ref = oracle.lora_linear(x, W, A, B, rk, idx, scale, residual=res)
    assert_rel(f64(y), ref, "y+res")
    # prefill tiling too
    T = 400
    x, W, A, B, rk, idx, _ = _inputs(rng, T, K, N, 5, 16)
    scale = rng.uniform(-3, 3, size=T).astype(np.float32)
    res = rand_bf16(rng, (T, N), 1.5)
    y = _run_gpu(x, W, A, B, rk, idx, scale, residual=res)
    ref = oracle.lora_linear(x, W, A, B, rk, idx, scale, residual=res)
    assert_rel(f64(y), ref, "y+res prefill")


@pytest.mark.parametrize("T", [32, 300])
def test_zero_up_projection_is_bitwise_base(T):
    rng = np.random.default_rng(T)
    K, N = 1024, 512
    x, W, A, B, rk, idx, scale = _inputs(rng, T, K, N, 6, 16, neg_frac=0.0)
    y_zero = _run_gpu(x, W, A, np.zeros_like(B), rk, idx, scale)
    y_none = _run_gpu(x, W, A, B, rk, np.full(T, -1, np.int32), scale)
    y_base = _run_gpu(x, W, None, None, None, None, None)
    assert torch.equal(y_zero.view(torch.int16), y_base.view(torch.int16))
    assert torch.equal(y_none.view(torch.int16), y_base.view(torch.int16))


@pytest.mark.parametrize("T", [80, 300])
def test_padding_beyond_rank_is_never_read(T):
    # NaN beyond each adapter's rank: any read of it would poison the output
    # (T = 300: the long-chunk shrink reads A rows up to r_max, U_s masks them).
    rng = np.random.default_rng(77)
    K, N = 512, 256
    ranks = [3, 8, 13, 16]
    x, W, A, B, rk, idx, scale = _inputs(rng, T, K, N, 4, 16, ranks)
    nan = np.uint16(0x7FC0)
    for a, r in enumerate(ranks):
        A[a, r:] = nan
        B[a, :, r:] = nan
    y = _run_gpu(x, W, A, B, rk, idx, scale)
    ref = oracle.lora_linear(x, W, A, B, rk, idx, scale)
    assert_rel(f64(y), ref, "y")


def test_empty_batch_launches_nothing():
    W = dev_u16(np.zeros((64, 64), np.uint16))
    x = dev_u16(np.zeros((0, 64), np.uint16))
    y = lk.local_lora_linear(x, W)
    torch.cuda.synchronize()
    assert y.shape == (0, 64)


@pytest.mark.parametrize("T", [16, 256, 257])
def test_one_adapter_for_every_token(T):
    # All tokens on one adapter: the shrink's token groups for that adapter
    # span many MFMA column tiles, the others get no tokens.
    say("lora_linear one adapter", T)
    rng = np.random.default_rng(500 + T)
    K, N = 512, 256
    x, W, A, B, rk, _, scale = _inputs(rng, T, K, N, 3, 16)
    idx = np.full(T, 1, np.int32)
    scale = rng.uniform(-2, 2, size=T).astype(np.float32)
    y = _run_gpu(x, W, A, B, rk, idx, scale)
    ref = oracle.lora_linear(x, W, A, B, rk, idx, scale)
    assert_rel(f64(y), ref, "y")


def test_out_of_range_adapter_and_rank():
    # Adapter indices outside [0, n_adapters) mean no adapter; ranks outside
    # [0, r_max] are clamped.
    say("lora_linear out of range")
    rng = np.random.default_rng(606)
    for T in (40, 300):
        K, N = 512, 256
        x, W, A, B, _, _, scale = _inputs(rng, T, K, N, 4, 16)
        rk = np.array([-3, 40, 16, 7], np.int32)
        idx = rng.integers(-5, 9, size=T).astype(np.int32)
        y = _run_gpu(x, W, A, B, rk, idx, scale)
        ref = oracle.lora_linear(x, W, A, B, rk, idx, scale)
        assert_rel(f64(y), ref, "y T=%d" % T)


def _grouped_gpu(x, Ws, As, Bs, ranks, idx, scale):
    kw = {}
    if As is not None:
        kw = dict(As=[dev_u16(a) for a in As], Bs=[dev_u16(b) for b in Bs],
                  ranks=[dev(r) for r in ranks], adapter_idx=dev(idx),
                  scale=dev(scale, torch.float32))
    ys = lk.local_lora_linear_grouped(dev_u16(x), [dev_u16(w) for w in Ws], **kw)
    torch.cuda.synchronize()
    return ys


GROUPED = [
    # T, K, N per projection, n_ad, r_max, ranks
    (32, 1024, (1024, 256, 256), 8, 16, None),
    (64, 512, (2048, 512, 512), 16, 64, [8, 16, 32, 64] * 4),
    (128, 512, (1024, 256, 256), 32, 16, None),
    (4, 256, (256, 256), 3, 8, None),
    (300, 512, (512, 256), 4, 16, None),       # long chunk: one launch over both
    (520, 512, (256, 768, 512), 5, 16, [16, 3, 9, 16, 0]),  # long chunk, three projections
    (300, 256, (320, 256), 3, 8, None),        # long chunk, N % 256 != 0: one at a time
    (16, 512, (64, 64), 16, 16, None),          # shrink too wide to fuse: grouped SGMV
    (64, 1024, (512, 128, 128), 16, 64, [8, 16, 32, 64] * 4),  # padded ranks: grouped SGMV
    (32, 512, (512, 512, 512), 0, 0, None),
    (200, 256, (256, 256, 512, 256), 5, 32, [32, 1, 17, 32, 24]),
]


@pytest.mark.parametrize("case", GROUPED, ids=lambda c: "T%d_K%d_G%d_ad%d" % (c[0], c[1], len(c[2]), c[3]))
def test_grouped_matches_oracle(case):
    T, K, Ns, n_ad, r_max, ranks = case
    say("lora_linear_grouped", case)
    rng = np.random.default_rng(T + K + sum(Ns) + n_ad)
    x = rand_bf16(rng, (T, K))
    Ws, As, Bs, Rs = [], [], [], []
    idx = scale = None
    for N in Ns:
        _, W, A, B, rk, idx_g, scale_g = _inputs(rng, T, K, N, n_ad, r_max, ranks)
        Ws.append(W)
        As.append(A)
        Bs.append(B)
        Rs.append(rk)
        if idx is None:
            idx, scale = idx_g, scale_g
    if n_ad:
        scale = rng.uniform(-2, 2, size=T).astype(np.float32)
    ys = _grouped_gpu(x, Ws, As if n_ad else None, Bs, Rs, idx, scale)
    for g, (W, A, B, rk) in enumerate(zip(Ws, As, Bs, Rs)):
        ref = oracle.lora_linear(x, W, A, B, rk, idx, scale) if n_ad else \
            oracle.lora_linear(x, W)
        assert_rel(f64(ys[g]), ref, "y[%d]" % g)


def test_grouped_zero_up_projection_is_bitwise_base():
    rng = np.random.default_rng(808)
    T, K, Ns = 32, 1024, (1024, 256, 256)
    x = rand_bf16(rng, (T, K))
    parts = [_inputs(rng, T, K, N, 6, 16, neg_frac=0.0) for N in Ns]
    Ws = [p[1] for p in parts]
    As = [p[2] for p in parts]
    Bz = [np.zeros_like(p[3]) for p in parts]
    Rs = [p[4] for p in parts]
    idx, scale = parts[0][5], parts[0][6]
    y_zero = _grouped_gpu(x, Ws, As, Bz, Rs, idx, scale)
    y_base = _grouped_gpu(x, Ws, None, None, None, None, None)
    for a, b in zip(y_zero, y_base):
        assert torch.equal(a.view(torch.int16), b.view(torch.int16))


@pytest.mark.parametrize("Ns", [(4096, 4096, 4096), (4096, 1024, 1024)],
                         ids=["mha_qkv", "gqa_qkv"])
def test_grouped_long_chunk_at_full_size(Ns):
    # The grouped call as the prefill step issues it: q, k, v of one 2048 x
    # 4096 activation over 4 rank-16 adapters (and unrouted tokens), one
    # shrink pass and one product over every projection's tiles. Checked on
    # sampled rows: each 128-token tile's first and last rows, the chunk
    # boundaries, and random rows.
    T, K, n_ad, r_max = 2048, 4096, 4, 16
    say("lora_linear_grouped full size", Ns)
    rng = np.random.default_rng(sum(Ns))
    x = rand_bf16(rng, (T, K))
    Ws = [rand_bf16(rng, (N, K), 0.02) for N in Ns]
    As = [rand_bf16(rng, (n_ad, r_max, K), 1 / math.sqrt(r_max)) for _ in Ns]
    Bs = [rand_bf16(rng, (n_ad, N, r_max), 0.01) for N in Ns]
    Rs = [np.full(n_ad, r_max, np.int32) for _ in Ns]
    idx = np.repeat(rng.integers(0, n_ad, size=T // 512), 512).astype(np.int32)
    idx[rng.random(T) < 0.05] = -1
    scale = rng.uniform(-2, 2, size=T).astype(np.float32)
    ys = _grouped_gpu(x, Ws, As, Bs, Rs, idx, scale)
    y0s = _grouped_gpu(x, Ws, None, None, None, None, None)
    rows = np.unique(np.concatenate([np.arange(0, T, 128), np.arange(127, T, 128),
                                     rng.choice(T, size=24, replace=False)]))
    sel = idx[rows] >= 0
    for g, (W, A, B, rk) in enumerate(zip(Ws, As, Bs, Rs)):
        ref = oracle.lora_linear(x[rows], W, A, B, rk, idx[rows], scale[rows])
        assert_rel(f64(ys[g])[rows], ref, "y[%d]" % g)
        # the adapter delta alone, against the oracle's (y - base)
        base = oracle.lora_linear(x[rows], W)
        assert_rel(f64(ys[g])[rows][sel] - f64(y0s[g])[rows][sel], (ref - base)[sel],
                   "delta[%d]" % g, tol=5e-2)
