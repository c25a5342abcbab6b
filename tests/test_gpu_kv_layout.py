"""Pool layout conversion (local_kv_pool_import / local_kv_pool_export) on the
GPU, bit for bit against numpy reshapes of the same pools (tests/pool_helpers:
dense_to_pool, pool_to_dense), including a pool of more tiles than the launch
has workgroups (the grid-stride loop) and an attention call on an imported
pool."""
import math

import numpy as np
import pytest
import torch

import oracle
import paper_2608_15241_amd as lk
from tests.gpu_helpers import assert_attn, assert_lse, dev, dev_u16, f64, host_u16, say
from tests.pool_helpers import dense_to_pool, make_table, pool_to_dense, rand_bf16

pytestmark = pytest.mark.gpu


def _bits(rng, shape):
    # every 16-bit pattern (NaNs, infinities and signed zeros included): a
    # permutation carries each unchanged
    return rng.integers(0, 1 << 16, size=shape, dtype=np.uint32).astype(np.uint16)


@pytest.mark.parametrize("nb,hkv,D", [(1, 1, 64), (37, 3, 128), (5, 8, 64), (19, 32, 128),
                                      (66000, 1, 64)])
def test_import_export_bitwise(nb, hkv, D):
    say("kv_pool import/export nb=%d hkv=%d D=%d" % (nb, hkv, D))
    rng = np.random.default_rng(nb * 131 + hkv * 7 + D)
    kd = _bits(rng, (nb, hkv, 16, D))
    vd = _bits(rng, (nb, hkv, 16, D))
    k_tok, v_tok = dev_u16(kd).view(nb, hkv, 16, D), dev_u16(vd).view(nb, hkv, 16, D)
    kc, vc = lk.local_kv_pool_import(k_tok, v_tok)
    torch.cuda.synchronize()
    ek, ev = dense_to_pool(kd, vd)
    assert np.array_equal(host_u16(kc).reshape(-1), ek)
    assert np.array_equal(host_u16(vc).reshape(-1), ev)
    # export of the imported pools gives the input back
    k2, v2 = lk.local_kv_pool_export(kc, vc, D)
    torch.cuda.synchronize()
    assert np.array_equal(host_u16(k2), kd)
    assert np.array_equal(host_u16(v2), vd)
    # export of independent library pools against the numpy inverse
    kl = _bits(rng, (nb, hkv, 16 * D))
    vl = _bits(rng, (nb, hkv, 16 * D))
    k3, v3 = lk.local_kv_pool_export(dev_u16(kl).view(nb, hkv, 16 * D),
                                     dev_u16(vl).view(nb, hkv, 16 * D), D)
    torch.cuda.synchronize()
    rk, rv = pool_to_dense(kl.reshape(-1), vl.reshape(-1), nb, hkv, D)
    assert np.array_equal(host_u16(k3), rk)
    assert np.array_equal(host_u16(v3), rv)


def test_import_empty_and_errors():
    z = torch.empty((0, 2, 16, 64), dtype=torch.bfloat16, device="cuda")
    kc, vc = lk.local_kv_pool_import(z, z.clone())
    assert kc.shape == (0, 2, 1024)
    x = torch.zeros((4, 2, 16, 64), dtype=torch.bfloat16, device="cuda")
    with pytest.raises(lk.LocalError):  # destination overlaps the source
        lk.local_kv_pool_import(x, x.clone(), k_cache=x.view(4, 2, 1024))


def test_decode_on_imported_pool_matches_oracle():
    """A token-major pool imported once, then decode attention on it, against
    the oracle on the numpy conversion of the same pool."""
    rng = np.random.default_rng(4242)
    hq, hkv, D = 8, 2, 128
    ctx = np.array([1, 17, 300, 513], dtype=np.int32)
    table, nb = make_table(rng, ctx, extra_blocks=3)
    B = len(ctx)
    kd = rand_bf16(rng, (nb, hkv, 16, D))
    vd = rand_bf16(rng, (nb, hkv, 16, D))
    tags = np.zeros(nb, dtype=np.int32)
    rv = np.zeros(B, dtype=np.int32)
    q = rand_bf16(rng, (B, hq, D))
    kc, vc = lk.local_kv_pool_import(dev_u16(kd).view(nb, hkv, 16, D),
                                     dev_u16(vd).view(nb, hkv, 16, D))
    sm = 1.0 / math.sqrt(D)
    out, lse = lk.local_paged_attn_decode(dev_u16(q).view(B, hq, D), kc, vc, dev(table),
                                          dev(ctx), dev(tags), dev(rv), sm, Hkv=hkv)
    torch.cuda.synchronize()
    ek, ev = dense_to_pool(kd, vd)
    qi = np.arange(B + 1, dtype=np.int32)
    ref, ref_lse = oracle.paged_attn(q, qi, hq, hkv, D, ek, ev, table, ctx, tags, rv, sm)
    assert_attn(f64(out), ref, "decode on imported pool", D)
    assert_lse(lse.cpu().numpy(), ref_lse, "decode on imported pool")
