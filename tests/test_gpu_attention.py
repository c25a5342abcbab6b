"""GPU parity of local_paged_attn_decode / local_paged_attn_prefill against the
oracle, including the in-kernel version mask, the KV append (bit-exact pool
contents) and the degenerate cases (one key, no valid key, ragged tails)."""
import math

import numpy as np
import pytest
import torch

import oracle
import paper_2608_15241_amd as lk
from tests.gpu_helpers import assert_attn, assert_lse, assert_rel, dev, dev_u16, f64, host_u16, say
from tests.pool_helpers import make_table, rand_bf16

pytestmark = pytest.mark.gpu


def _pool(rng, num, hkv, D):
    return rand_bf16(rng, (num * hkv * 16 * D,)), rand_bf16(rng, (num * hkv * 16 * D,))


def _tags(rng, table, ctx, rv, num, stale_frac, stale_last=True):
    bv = np.full(num, -7, np.int32)
    for b, L in enumerate(ctx):
        nb = (int(L) + 15) // 16
        tags = np.full(nb, rv[b], np.int32)
        pick = rng.random(nb) < stale_frac
        if not stale_last and nb:
            pick[nb - 1] = False
        tags[pick] = rv[b] + rng.choice([-1, 1, 5000], size=int(pick.sum()))
        bv[table[b, :nb]] = tags
    return bv


def _decode_case(rng, ctx, Hq, Hkv, D, stale_frac, append=True, max_blocks=None):
    ctx = np.asarray(ctx, np.int32)
    B = len(ctx)
    table, num = make_table(rng, ctx, extra_blocks=3, max_blocks=max_blocks)
    rv = (rng.integers(1, 9, size=B) * 1000).astype(np.int32)
    bv = _tags(rng, table, ctx, rv, num, stale_frac)
    kc, vc = _pool(rng, num, Hkv, D)
    q = rand_bf16(rng, (B, Hq, D))
    kn = rand_bf16(rng, (B, Hkv, D)) if append else None
    vn = rand_bf16(rng, (B, Hkv, D)) if append else None
    return dict(ctx=ctx, table=table, rv=rv, bv=bv, kc=kc, vc=vc, q=q, kn=kn, vn=vn,
                Hq=Hq, Hkv=Hkv, D=D, B=B)


def _run_decode(c):
    kc_d, vc_d = dev_u16(c["kc"]), dev_u16(c["vc"])
    out, lse = lk.local_paged_attn_decode(
        dev_u16(c["q"]), kc_d, vc_d, dev(c["table"]), dev(c["ctx"]), dev(c["bv"]),
        dev(c["rv"]), 1.0 / math.sqrt(c["D"]),
        k_new=None if c["kn"] is None else dev_u16(c["kn"]),
        v_new=None if c["vn"] is None else dev_u16(c["vn"]), Hkv=c["Hkv"])
    torch.cuda.synchronize()
    return out, lse, kc_d, vc_d


def _oracle_decode(c):
    kc, vc = c["kc"].copy(), c["vc"].copy()
    qi = np.arange(c["B"] + 1, dtype=np.int32)
    if c["kn"] is not None:
        oracle.kv_append(kc, vc, c["Hkv"], c["D"], c["table"], qi, c["ctx"], c["kn"], c["vn"])
    out, lse = oracle.paged_attn(c["q"], qi, c["Hq"], c["Hkv"], c["D"], kc, vc, c["table"],
                                 c["ctx"], c["bv"], c["rv"], 1.0 / math.sqrt(c["D"]))
    return out, lse, kc, vc


CTX = [1, 15, 16, 17, 31, 100, 511, 512, 513, 1025, 2000, 3333]


@pytest.mark.parametrize("Hq,Hkv,D", [(4, 4, 64), (32, 32, 128), (32, 8, 128), (8, 1, 128),
                                      (16, 16, 64), (12, 4, 64)])
def test_decode_matches_oracle(Hq, Hkv, D):
    say("decode", Hq, Hkv, D)
    rng = np.random.default_rng(Hq * 31 + Hkv * 7 + D)
    c = _decode_case(rng, CTX, Hq, Hkv, D, stale_frac=0.2)
    out, lse, kc_d, vc_d = _run_decode(c)
    ro, rl, rkc, rvc = _oracle_decode(c)
    assert_attn(f64(out), ro, "out", D)
    assert_lse(lse.cpu().numpy(), rl, "lse")
    assert np.array_equal(host_u16(kc_d), rkc), "appended K pool differs"
    assert np.array_equal(host_u16(vc_d), rvc), "appended V pool differs"


def test_decode_without_append_and_long_contexts():
    rng = np.random.default_rng(3)
    c = _decode_case(rng, [16384, 9000, 4097, 1], 32, 8, 128, stale_frac=0.1, append=False)
    out, lse, kc_d, _ = _run_decode(c)
    ro, rl, rkc, _ = _oracle_decode(c)
    assert_attn(f64(out), ro, "out", c["D"])
    assert_lse(lse.cpu().numpy(), rl, "lse")
    assert np.array_equal(host_u16(kc_d), rkc)


def test_decode_degenerate_cases():
    # request 0: every block stale; request 1: one valid key (position 0 of a
    # fully stale tail); request 2: context 1 (only the appended token).
    rng = np.random.default_rng(4)
    Hq = Hkv = 4
    D = 128
    ctx = np.array([70, 40, 1], np.int32)
    table, num = make_table(rng, ctx)
    rv = np.array([10, 20, 30], np.int32)
    bv = np.full(num, 0, np.int32)
    bv[table[1, 0]] = 20                       # tokens 0..15 valid
    bv[table[2, 0]] = 30
    kc, vc = _pool(rng, num, Hkv, D)
    q = rand_bf16(rng, (3, Hq, D))
    kn, vn = rand_bf16(rng, (3, Hkv, D)), rand_bf16(rng, (3, Hkv, D))
    c = dict(ctx=ctx, table=table, rv=rv, bv=bv, kc=kc, vc=vc, q=q, kn=kn, vn=vn,
             Hq=Hq, Hkv=Hkv, D=D, B=3)
    out, lse, _, _ = _run_decode(c)
    ro, rl, _, _ = _oracle_decode(c)
    o = f64(out)
    assert np.all(o[0] == 0.0) and np.all(np.isneginf(lse[0].cpu().numpy()))
    assert_attn(o[1:], ro[1:], "out", D)
    assert_lse(lse.cpu().numpy(), rl, "lse")
    # context 1: the output is exactly the appended V row (rounded once)
    assert np.array_equal(host_u16(out)[2], vn[2].reshape(Hkv, D))


@pytest.mark.parametrize("max_blocks", [4, 80])
def test_decode_empty_context(max_blocks):
    # An empty context has no key: zero output and lse = -inf, also when the
    # table is narrow enough for a single partition (no merge pass), and no
    # append (the token position L-1 does not exist).
    say("decode empty context", max_blocks)
    rng = np.random.default_rng(40 + max_blocks)
    c = _decode_case(rng, [0, 33, 0, 50], 8, 2, 128, stale_frac=0.0,
                     max_blocks=max_blocks)
    out, lse, kc_d, vc_d = _run_decode(c)
    ro, rl, rkc, rvc = _oracle_decode(c)
    o, l = f64(out), lse.cpu().numpy()
    for b in (0, 2):
        assert np.all(o[b] == 0.0) and np.all(np.isneginf(l[b]))
    assert_attn(o, ro, "out", 128)
    assert_lse(l, rl, "lse")
    assert np.array_equal(host_u16(kc_d), rkc) and np.array_equal(host_u16(vc_d), rvc)


def test_decode_wide_block_table_and_batch():
    rng = np.random.default_rng(8)
    ctx = rng.integers(1, 700, size=97)
    c = _decode_case(rng, ctx, 16, 2, 128, stale_frac=0.3, max_blocks=200)
    out, lse, _, _ = _run_decode(c)
    ro, rl, _, _ = _oracle_decode(c)
    assert_attn(f64(out), ro, "out", c["D"])
    assert_lse(lse.cpu().numpy(), rl, "lse")


@pytest.mark.parametrize("B", [600, 1100])
def test_decode_batch_beyond_ranked_dispatch(B):
    # More requests than the longest-first ranking of the grid covers (512):
    # the grid is walked in partition-row order instead. Mixed contexts from
    # 1 token to several partitions, stale blocks, GQA, with the append.
    say("decode large batch", B)
    rng = np.random.default_rng(B)
    ctx = np.rint(np.exp(rng.uniform(0.0, np.log(3000.0), size=B))).astype(np.int32)
    ctx[::97] = 1
    ctx[5] = 2049
    c = _decode_case(rng, ctx, 8, 2, 128, stale_frac=0.15)
    out, lse, kc_d, vc_d = _run_decode(c)
    ro, rl, rkc, rvc = _oracle_decode(c)
    assert_attn(f64(out), ro, "out", 128)
    assert_lse(lse.cpu().numpy(), rl, "lse")
    assert np.array_equal(host_u16(kc_d), rkc), "appended K pool differs"
    assert np.array_equal(host_u16(vc_d), rvc), "appended V pool differs"


# ------------------------------------------------------------------ prefill

def _prefill_case(rng, prefix, chunk, Hq, Hkv, D, stale_frac):
    prefix = np.asarray(prefix, np.int32)
    chunk = np.asarray(chunk, np.int32)
    ctx = prefix + chunk
    B = len(ctx)
    table, num = make_table(rng, ctx, extra_blocks=2)
    rv = (rng.integers(1, 9, size=B) * 1000).astype(np.int32)
    bv = _tags(rng, table, ctx, rv, num, stale_frac)
    kc, vc = _pool(rng, num, Hkv, D)
    qi = np.concatenate([[0], np.cumsum(chunk)]).astype(np.int32)
    T = int(qi[-1])
    return dict(ctx=ctx, table=table, rv=rv, bv=bv, kc=kc, vc=vc, qi=qi, T=T,
                q=rand_bf16(rng, (T, Hq, D)), kn=rand_bf16(rng, (T, Hkv, D)),
                vn=rand_bf16(rng, (T, Hkv, D)), Hq=Hq, Hkv=Hkv, D=D)


@pytest.mark.parametrize("Hq,Hkv,D", [(4, 4, 64), (8, 2, 128), (32, 32, 128)])
def test_prefill_matches_oracle(Hq, Hkv, D):
    say("prefill", Hq, Hkv, D)
    rng = np.random.default_rng(Hq + 100 * Hkv + D)
    c = _prefill_case(rng, [0, 5, 16, 100, 700, 33], [1, 17, 64, 130, 200, 0], Hq, Hkv, D, 0.2)
    kc_d, vc_d = dev_u16(c["kc"]), dev_u16(c["vc"])
    out, lse = lk.local_paged_attn_prefill(
        dev_u16(c["q"]), dev(c["qi"]), kc_d, vc_d, dev(c["table"]), dev(c["ctx"]),
        dev(c["bv"]), dev(c["rv"]), 1.0 / math.sqrt(D), k_new=dev_u16(c["kn"]),
        v_new=dev_u16(c["vn"]), Hkv=Hkv)
    torch.cuda.synchronize()
    kc, vc = c["kc"].copy(), c["vc"].copy()
    oracle.kv_append(kc, vc, Hkv, D, c["table"], c["qi"], c["ctx"], c["kn"], c["vn"])
    ro, rl = oracle.paged_attn(c["q"], c["qi"], Hq, Hkv, D, kc, vc, c["table"], c["ctx"],
                               c["bv"], c["rv"], 1.0 / math.sqrt(D))
    assert np.array_equal(host_u16(kc_d), kc), "appended K pool differs"
    assert np.array_equal(host_u16(vc_d), vc), "appended V pool differs"
    assert_attn(f64(out), ro, "out", D)
    assert_lse(lse.cpu().numpy(), rl, "lse")


@pytest.mark.parametrize("B,append", [(65, True), (130, True), (300, True), (300, False)])
def test_prefill_many_requests(B, append):
    # more requests than a wavefront scans at once, and (300) than the unit
    # planner's workgroup lists in one pass: the device-side mapping of the
    # grid onto (request, tile) and (request, block) takes several passes;
    # empty chunks, chunks starting and ending inside a block, long chunks;
    # without an append the planner runs as a launch of its own
    say("prefill many requests", B, append)
    rng = np.random.default_rng(B + (0 if append else 1))
    Hq, Hkv, D = 8, 2, 64
    prefix = rng.integers(0, 300, size=B)
    chunk = rng.integers(0, 150, size=B)
    chunk[::7] = 0
    chunk[3] = 300
    c = _prefill_case(rng, prefix, chunk, Hq, Hkv, D, 0.1)
    kc_d, vc_d = dev_u16(c["kc"]), dev_u16(c["vc"])
    kw = dict(k_new=dev_u16(c["kn"]), v_new=dev_u16(c["vn"])) if append else {}
    out, lse = lk.local_paged_attn_prefill(
        dev_u16(c["q"]), dev(c["qi"]), kc_d, vc_d, dev(c["table"]), dev(c["ctx"]),
        dev(c["bv"]), dev(c["rv"]), 1.0 / math.sqrt(D), Hkv=Hkv, **kw)
    torch.cuda.synchronize()
    kc, vc = c["kc"].copy(), c["vc"].copy()
    if append:
        oracle.kv_append(kc, vc, Hkv, D, c["table"], c["qi"], c["ctx"], c["kn"], c["vn"])
    ro, rl = oracle.paged_attn(c["q"], c["qi"], Hq, Hkv, D, kc, vc, c["table"], c["ctx"],
                               c["bv"], c["rv"], 1.0 / math.sqrt(D))
    assert np.array_equal(host_u16(kc_d), kc), "appended K pool differs"
    assert np.array_equal(host_u16(vc_d), vc), "appended V pool differs"
    assert_attn(f64(out), ro, "out", D)
    assert_lse(lse.cpu().numpy(), rl, "lse")


def test_prefill_one_token_chunk_equals_decode():
    rng = np.random.default_rng(21)
    Hq, Hkv, D = 8, 2, 128
    c = _decode_case(rng, [40, 1000, 17], Hq, Hkv, D, stale_frac=0.25)
    out_d, lse_d, _, _ = _run_decode(c)
    qi = np.arange(4, dtype=np.int32)
    out_p, lse_p = lk.local_paged_attn_prefill(
        dev_u16(c["q"]), dev(qi), dev_u16(c["kc"]), dev_u16(c["vc"]), dev(c["table"]),
        dev(c["ctx"]), dev(c["bv"]), dev(c["rv"]), 1.0 / math.sqrt(D),
        k_new=dev_u16(c["kn"]), v_new=dev_u16(c["vn"]), Hkv=Hkv)
    torch.cuda.synchronize()
    assert_attn(f64(out_p), f64(out_d), "prefill vs decode", D, tol=1e-2)
    assert_lse(lse_p.cpu().numpy(), lse_d.cpu().numpy(), "lse")


@pytest.mark.parametrize("sm_scale", [-0.09, 0.0, 0.3])
def test_prefill_any_sign_of_the_scale(sm_scale):
    # any sign of the softmax scale: a negative one reverses the ranking of the
    # keys, a zero one gives the mean of the visible values (masked positions
    # and stale blocks stay out)
    say("prefill scale", sm_scale)
    rng = np.random.default_rng(int(1000 * abs(sm_scale)) + (7 if sm_scale < 0 else 5))
    Hq, Hkv, D = 8, 2, 128
    c = _prefill_case(rng, [0, 40, 300], [37, 130, 64], Hq, Hkv, D, 0.2)
    kc_d, vc_d = dev_u16(c["kc"]), dev_u16(c["vc"])
    out, lse = lk.local_paged_attn_prefill(
        dev_u16(c["q"]), dev(c["qi"]), kc_d, vc_d, dev(c["table"]), dev(c["ctx"]),
        dev(c["bv"]), dev(c["rv"]), sm_scale, k_new=dev_u16(c["kn"]),
        v_new=dev_u16(c["vn"]), Hkv=Hkv)
    torch.cuda.synchronize()
    kc, vc = c["kc"].copy(), c["vc"].copy()
    oracle.kv_append(kc, vc, Hkv, D, c["table"], c["qi"], c["ctx"], c["kn"], c["vn"])
    ro, rl = oracle.paged_attn(c["q"], c["qi"], Hq, Hkv, D, kc, vc, c["table"], c["ctx"],
                               c["bv"], c["rv"], sm_scale)
    assert_attn(f64(out), ro, "out", D)
    assert_lse(lse.cpu().numpy(), rl, "lse")


def test_prefill_request_with_bad_row_range_is_skipped():
    # Requests 1 and 2 have row ranges that are not ranges of q (past T,
    # reversed): they must get no work at all (no append into their blocks,
    # no rows), and the valid requests 0 and 3 must be exactly as if the bad
    # ones were absent.
    say("prefill bad row range")
    rng = np.random.default_rng(1234)
    Hq, Hkv, D = 8, 2, 128
    ctx = np.array([21, 50, 80, 94], np.int32)
    qi = np.array([0, 16, 60, 16, 40], np.int32)
    T = 40
    table, num = make_table(rng, ctx, extra_blocks=2)
    rv = np.array([1000, 2000, 3000, 4000], np.int32)
    bv = _tags(rng, table, ctx, rv, num, 0.1, stale_last=False)
    kc, vc = _pool(rng, num, Hkv, D)
    q = rand_bf16(rng, (T, Hq, D))
    kn, vn = rand_bf16(rng, (T, Hkv, D)), rand_bf16(rng, (T, Hkv, D))
    kc_d, vc_d = dev_u16(kc), dev_u16(vc)
    out, lse = lk.local_paged_attn_prefill(
        dev_u16(q), dev(qi), kc_d, vc_d, dev(table), dev(ctx), dev(bv), dev(rv),
        1.0 / math.sqrt(D), k_new=dev_u16(kn), v_new=dev_u16(vn), Hkv=Hkv)
    torch.cuda.synchronize()
    keep = [0, 3]
    sub_qi = np.array([0, 16, 40], np.int32)
    rk, rvv = kc.copy(), vc.copy()
    oracle.kv_append(rk, rvv, Hkv, D, table[keep], sub_qi, ctx[keep], kn, vn)
    ro, rl = oracle.paged_attn(q, sub_qi, Hq, Hkv, D, rk, rvv, table[keep], ctx[keep], bv,
                               rv[keep], 1.0 / math.sqrt(D))
    assert np.array_equal(host_u16(kc_d), rk), "K pool: a skipped request appended"
    assert np.array_equal(host_u16(vc_d), rvv), "V pool: a skipped request appended"
    assert_attn(f64(out), ro, "out", D)
    assert_lse(lse.cpu().numpy(), rl, "lse")


def test_binding_rejects_wrong_output_and_tag_shapes():
    # The binding checks what the kernels would otherwise write or read out
    # of bounds: the output and lse shapes and one tag per pool block.
    rng = np.random.default_rng(55)
    c = _decode_case(rng, [40, 17], 8, 2, 64, stale_frac=0.0)
    args = (dev_u16(c["q"]), dev_u16(c["kc"]), dev_u16(c["vc"]), dev(c["table"]),
            dev(c["ctx"]), dev(c["bv"]), dev(c["rv"]), 0.125)
    with pytest.raises(ValueError):
        lk.prepare_paged_attn_decode(*args, Hkv=2, out=torch.empty(
            (2, 8, 32), dtype=torch.bfloat16, device="cuda"))
    with pytest.raises(ValueError):
        lk.prepare_paged_attn_decode(*args, Hkv=2, lse=torch.empty(
            (1, 8), dtype=torch.float32, device="cuda"))
    short = dev(c["bv"][:-1])
    with pytest.raises(ValueError):
        lk.prepare_paged_attn_decode(args[0], args[1], args[2], args[3], args[4], short,
                                     args[6], 0.125, Hkv=2)
    qi = np.array([0, 1, 2], np.int32)
    with pytest.raises(ValueError):
        lk.prepare_paged_attn_prefill(args[0], dev(qi), args[1], args[2], args[3], args[4],
                                      args[5], args[6], 0.125, Hkv=2, out=torch.empty(
                                          (3, 8, 64), dtype=torch.bfloat16, device="cuda"))


@pytest.mark.parametrize("D", [64, 128])
def test_prefill_long_prefixes_split_key_ranges(D):
    # Tiles whose causal range is long are split into 2 to 4 key ranges run
    # by different workgroups and merged: long prefixes, chunks ending inside
    # a tile, a request whose whole first key range is stale (a split with no
    # valid key), a one-token chunk on a long prefix, and a negative scale
    # for one of the two head dims.
    say("prefill split key ranges", D)
    rng = np.random.default_rng(900 + D)
    Hq, Hkv = 8, 2
    c = _prefill_case(rng, [3000, 1500, 800, 0, 5000, 2047], [130, 300, 17, 256, 1, 200],
                      Hq, Hkv, D, 0.1)
    # request 0: its first 70 blocks stale, so its tiles' first key range is empty
    c["bv"][c["table"][0, :70]] = c["rv"][0] - 1
    scale = -1.0 / math.sqrt(D) if D == 64 else 1.0 / math.sqrt(D)
    kc_d, vc_d = dev_u16(c["kc"]), dev_u16(c["vc"])
    out, lse = lk.local_paged_attn_prefill(
        dev_u16(c["q"]), dev(c["qi"]), kc_d, vc_d, dev(c["table"]), dev(c["ctx"]),
        dev(c["bv"]), dev(c["rv"]), scale, k_new=dev_u16(c["kn"]), v_new=dev_u16(c["vn"]),
        Hkv=Hkv)
    torch.cuda.synchronize()
    kc, vc = c["kc"].copy(), c["vc"].copy()
    oracle.kv_append(kc, vc, Hkv, D, c["table"], c["qi"], c["ctx"], c["kn"], c["vn"])
    ro, rl = oracle.paged_attn(c["q"], c["qi"], Hq, Hkv, D, kc, vc, c["table"], c["ctx"],
                               c["bv"], c["rv"], scale)
    assert np.array_equal(host_u16(kc_d), kc), "appended K pool differs"
    assert np.array_equal(host_u16(vc_d), vc), "appended V pool differs"
    assert_attn(f64(out), ro, "out", D)
    assert_lse(lse.cpu().numpy(), rl, "lse")


@pytest.mark.parametrize("B,max_blocks,cap", [(40, None, None), (600, None, 50), (7, 300, 0),
                                              (129, 64, None), (9, 700, None)])
def test_decode_checked_equals_attention_and_version_check(B, max_blocks, cap):
    # The attention call that also reports the version check: its attention
    # results are the plain call's bit for bit, and its stale list, count and
    # valid tokens are the separate version check's (and the oracle's) bit
    # for bit, also truncated at cap, with empty contexts and a table wider
    # than the contexts.
    say("decode checked", B, max_blocks, cap)
    rng = np.random.default_rng(3000 + B)
    ctx = rng.integers(0, 3000, size=B).astype(np.int32)
    if max_blocks is not None:
        ctx = np.minimum(ctx, 16 * max_blocks)
    ctx[::11] = 0
    c = _decode_case(rng, ctx, 8, 2, 128, stale_frac=0.3, max_blocks=max_blocks)
    ctx_d, tab, bv, rv = dev(c["ctx"]), dev(c["table"]), dev(c["bv"]), dev(c["rv"])
    res = []
    for fn in (lk.local_paged_attn_decode, lk.local_paged_attn_decode_checked):
        kc, vc = dev_u16(c["kc"]), dev_u16(c["vc"])
        kw = {} if fn is lk.local_paged_attn_decode else {"cap": cap}
        r = fn(dev_u16(c["q"]), kc, vc, tab, ctx_d, bv, rv, 1.0 / math.sqrt(128),
               k_new=dev_u16(c["kn"]), v_new=dev_u16(c["vn"]), Hkv=2, **kw)
        torch.cuda.synchronize()
        res.append((r, kc, vc))
    (o1, l1), k1, v1 = res[0]
    (o2, l2, pairs, n, valid), k2, v2 = res[1]
    assert torch.equal(o1.view(torch.int16), o2.view(torch.int16))
    assert torch.equal(l1.view(torch.int32), l2.view(torch.int32))
    assert torch.equal(k1.view(torch.int16), k2.view(torch.int16))
    assert torch.equal(v1.view(torch.int16), v2.view(torch.int16))
    cap_ = c["table"].size if cap is None else cap
    p_ref, n_ref, v_ref = lk.local_block_version_check(tab, ctx_d, bv, rv, cap=cap_)
    torch.cuda.synchronize()
    ep, en, ev = oracle.block_version_check(c["table"], c["ctx"], c["bv"], c["rv"], cap=cap_)
    assert int(n.item()) == en == int(n_ref.item())
    assert np.array_equal(valid.cpu().numpy(), ev)
    k = min(en, cap_)
    assert np.array_equal(pairs[:k].cpu().numpy(), ep)
    assert np.array_equal(p_ref[:k].cpu().numpy(), ep)
