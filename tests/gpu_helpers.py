"""Helpers of the GPU parity tests (test infrastructure).

Inputs come from `workloads` (seeded); the expected values come from `oracle`
on host copies of exactly those inputs. Nothing here computes any part of the
method.
"""
from __future__ import annotations

import sys

import numpy as np
import torch

import oracle

TOL = 2e-2  # max |gpu - ref| <= TOL * max |ref|, per output tensor
LSE_ABS = 1e-3  # |gpu lse - ref lse| in nats, every finite entry


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def dev(a, dtype=torch.int32):
    return torch.from_numpy(np.ascontiguousarray(a)).to(device="cuda", dtype=dtype)


def dev_u16(a):
    """uint16 bf16 bits (numpy) -> bf16 device tensor."""
    a = np.ascontiguousarray(a, dtype=np.uint16)
    return torch.from_numpy(a.view(np.int16)).to("cuda").view(torch.bfloat16)


def host_u16(t) -> np.ndarray:
    return t.detach().contiguous().view(torch.int16).cpu().numpy().view(np.uint16)


def f64(t) -> np.ndarray:
    if isinstance(t, np.ndarray):
        return oracle.bf16_to_f64(t)
    if t.dtype == torch.bfloat16:
        return oracle.bf16_to_f64(host_u16(t))
    return t.detach().cpu().numpy().astype(np.float64)


def assert_rel(gpu, ref, name, tol=TOL):
    gpu = np.asarray(gpu, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    assert gpu.shape == ref.shape, (name, gpu.shape, ref.shape)
    if ref.size == 0:
        return 0.0
    assert np.all(np.isfinite(gpu)), "%s: non-finite GPU values" % name
    scale = np.abs(ref).max()
    err = np.abs(gpu - ref).max()
    assert err <= tol * scale, "%s: max|d|=%.4g > %.3g*max|ref|=%.4g" % (
        name, err, tol, tol * scale)
    return err / scale if scale > 0 else err


def assert_attn(gpu, ref, name, row_len, tol=TOL):
    """Attention outputs: the tolerance rule per output tensor and also per
    row of `row_len` values (one token and query head), so that a row whose
    values are small next to the tensor's largest (a long context averages
    its values down) is held to its own scale. A row whose reference is all
    zero (no valid key) must be exactly zero."""
    err = assert_rel(gpu, ref, name, tol)
    g = np.asarray(gpu, np.float64).reshape(-1, row_len)
    r = np.asarray(ref, np.float64).reshape(-1, row_len)
    scale = np.abs(r).max(axis=1)
    d = np.abs(g - r).max(axis=1)
    bad = np.nonzero(d > tol * scale)[0]
    assert bad.size == 0, "%s: %d rows off, first row %d: max|d|=%.4g > %.3g*max|ref row|=%.4g" % (
        name, bad.size, bad[0], d[bad[0]], tol, tol * scale[bad[0]])
    return err


def assert_lse(gpu_lse, ref_lse, name, atol=LSE_ABS):
    """lse: the same -inf entries (no valid key), and every finite entry within
    `atol` nats (a float32 log-sum-exp is good to about 1e-5 here)."""
    g = np.asarray(gpu_lse, np.float64)
    r = np.asarray(ref_lse, np.float64)
    inf_r = np.isneginf(r)
    assert np.array_equal(np.isneginf(g), inf_r), "%s: -inf pattern differs" % name
    if (~inf_r).any():
        assert np.all(np.isfinite(g[~inf_r])), "%s: non-finite GPU values" % name
        d = np.abs(g[~inf_r] - r[~inf_r])
        assert d.max() <= atol, "%s: max|d|=%.3g nats > %.3g" % (name, d.max(), atol)


def gather_requests(k_pool, v_pool, hkv, D, block_table, ctx_lens, block_version, reqs):
    """Host copies of just the blocks of `reqs` (device pools of one layer).

    Returns (k_host, v_host, table, block_version) with block ids renumbered
    0..n-1 in the order the requests own them.
    """
    nb = [(int(ctx_lens[b]) + 15) // 16 for b in reqs]
    mb = max(nb) if nb else 1
    ids = np.concatenate([block_table[b, :n] for b, n in zip(reqs, nb)]).astype(np.int64)
    idx = torch.from_numpy(ids).to("cuda")
    per = hkv * 16 * D
    kh = host_u16(k_pool.view(-1, per).index_select(0, idx)).reshape(-1)
    vh = host_u16(v_pool.view(-1, per).index_select(0, idx)).reshape(-1)
    table = np.zeros((len(reqs), mb), np.int32)
    off = 0
    for i, n in enumerate(nb):
        table[i, :n] = np.arange(off, off + n)
        off += n
    bv = block_version[ids].astype(np.int32)
    return kh, vh, table, bv
