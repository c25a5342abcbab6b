"""local_paged_attn_decode_noalloc (the decode entry point that takes no
workspace and allocates nothing) against local_paged_attn_decode and the
oracle: two calls in a row through the C ABI, the second with a smaller
input, so the second runs on scratch the first left behind."""
import math

import numpy as np
import pytest
import torch

import oracle
import paper_2608_15241_amd as lk
from tests.gpu_helpers import assert_attn, assert_lse, dev, dev_u16, f64, host_u16, say
from tests.pool_helpers import make_table, rand_bf16

pytestmark = pytest.mark.gpu


def _case(rng, ctx, Hq, Hkv, D, max_blocks=None):
    ctx = np.asarray(ctx, np.int32)
    B = len(ctx)
    table, num = make_table(rng, ctx, extra_blocks=2, max_blocks=max_blocks)
    rv = (rng.integers(1, 9, size=B) * 1000).astype(np.int32)
    bv = np.zeros(num, np.int32)
    for b, L in enumerate(ctx):
        nb = (int(L) + 15) // 16
        tags = np.full(nb, rv[b], np.int32)
        stale = rng.random(nb) < 0.15
        stale[nb - 1:] = False
        tags[stale] = rv[b] - 1
        bv[table[b, :nb]] = tags
    n = num * Hkv * 16 * D
    return dict(ctx=ctx, table=table, rv=rv, bv=bv, kc=rand_bf16(rng, (n,)),
                vc=rand_bf16(rng, (n,)), q=rand_bf16(rng, (B, Hq, D)),
                kn=rand_bf16(rng, (B, Hkv, D)), vn=rand_bf16(rng, (B, Hkv, D)),
                Hq=Hq, Hkv=Hkv, D=D, B=B)


def _both(c):
    """(out, lse, K pool, V pool) of each entry point, each on its own pool copy."""
    res = []
    for fn in (lk.local_paged_attn_decode, lk.local_paged_attn_decode_noalloc):
        kc, vc = dev_u16(c["kc"]), dev_u16(c["vc"])
        out, lse = fn(dev_u16(c["q"]), kc, vc, dev(c["table"]), dev(c["ctx"]), dev(c["bv"]),
                      dev(c["rv"]), 1.0 / math.sqrt(c["D"]), k_new=dev_u16(c["kn"]),
                      v_new=dev_u16(c["vn"]), Hkv=c["Hkv"])
        torch.cuda.synchronize()
        res.append((out, lse, kc, vc))
    return res


def _check(c, res):
    (o1, l1, k1, v1), (o2, l2, k2, v2) = res
    # the same kernels on the same inputs: bit for bit
    assert torch.equal(o1.view(torch.int16), o2.view(torch.int16))
    assert torch.equal(l1.view(torch.int32), l2.view(torch.int32))
    assert torch.equal(k1.view(torch.int16), k2.view(torch.int16))
    assert torch.equal(v1.view(torch.int16), v2.view(torch.int16))
    kc, vc = c["kc"].copy(), c["vc"].copy()
    qi = np.arange(c["B"] + 1, dtype=np.int32)
    oracle.kv_append(kc, vc, c["Hkv"], c["D"], c["table"], qi, c["ctx"], c["kn"], c["vn"])
    ro, rl = oracle.paged_attn(c["q"], qi, c["Hq"], c["Hkv"], c["D"], kc, vc, c["table"],
                               c["ctx"], c["bv"], c["rv"], 1.0 / math.sqrt(c["D"]))
    assert_attn(f64(o2), ro, "noalloc out", c["D"])
    assert_lse(l2.cpu().numpy(), rl, "noalloc lse")
    assert np.array_equal(host_u16(k2), kc) and np.array_equal(host_u16(v2), vc)


def test_noalloc_matches_workspace_entry_point_twice():
    rng = np.random.default_rng(77)
    # first call: long contexts, many partitions per request (the scratch in use)
    say("noalloc call 1")
    c1 = _case(rng, rng.integers(1, 6000, size=48), 32, 8, 128)
    _check(c1, _both(c1))
    # second call, smaller: fewer requests, shorter table, D = 64; it reads
    # only partials it wrote itself, whatever the first call left
    say("noalloc call 2")
    c2 = _case(rng, rng.integers(1, 1500, size=9), 8, 8, 64)
    _check(c2, _both(c2))


def test_noalloc_at_its_size_limit_and_beyond():
    # 256 requests x 32 heads with a 1024-block table (16 partitions of 64
    # blocks) need exactly the library's scratch; one request more is refused
    # before any launch.
    rng = np.random.default_rng(78)
    say("noalloc at the limit")
    c = _case(rng, rng.integers(1, 1100, size=256), 32, 8, 128, max_blocks=1024)
    _check(c, _both(c))
    big = _case(rng, rng.integers(1, 40, size=257), 32, 8, 128, max_blocks=1024)
    with pytest.raises(lk.LocalError, match="scratch"):
        lk.local_paged_attn_decode_noalloc(
            dev_u16(big["q"]), dev_u16(big["kc"]), dev_u16(big["vc"]), dev(big["table"]),
            dev(big["ctx"]), dev(big["bv"]), dev(big["rv"]), 0.088, Hkv=8)
