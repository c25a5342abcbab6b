"""The host-side KV manager of local_kv.h (C++, in liblocal.so) against its
oracle (oracle/kvm.py), call by call, on seeded random operation sequences;
plus the error behaviour of the C ABI. CPU only."""
import numpy as np
import pytest

import paper_2608_15241_amd as lk
from oracle.kvm import BS, KVMOracle

pytestmark = pytest.mark.filterwarnings("ignore::DeprecationWarning")


def _paths(rng, n_paths, vocab, max_blocks):
    """Token paths sharing prefixes: each extends a random earlier one."""
    paths = []
    for _ in range(n_paths):
        if paths and rng.random() < 0.7:
            base = paths[rng.integers(len(paths))]
            keep = int(rng.integers(0, len(base) // BS + 1)) * BS
            base = base[:keep]
        else:
            base = []
        extra = int(rng.integers(1, max_blocks + 1)) * BS + int(rng.integers(0, BS))
        paths.append(base + [int(v) for v in rng.integers(0, vocab, size=extra)])
    return paths


def _close(a, b):
    return a == b or abs(a - b) <= 1e-12 * max(abs(a), abs(b))


@pytest.mark.parametrize("seed", range(6))
def test_random_sequences_match_the_oracle(seed):
    rng = np.random.default_rng(1000 + seed)
    nb = int(rng.integers(24, 96))
    params = dict(lambda_p=float(rng.uniform(0.5, 0.95)), lambda_a=float(rng.uniform(0.5, 0.95)),
                  beta=0.3, chi=0.7, eta=0.2, zeta=1.5, alpha_l=0.5, l_max=64.0,
                  c_tok=1.0, c_ctx=0.01, block_bytes=2.0)
    m = lk.KVManager(nb, params)
    o = KVMOracle(nb, params)
    adapters = {0: 1000, 1: 2000, 2: 3000}
    for a, v in adapters.items():
        m.set_committed(a, v)
        o.set_committed(a, v)
    paths = _paths(rng, 14, vocab=3, max_blocks=6)
    next_version = {a: v + 1 for a, v in adapters.items()}
    held = []  # block lists pinned by "active requests"
    for step in range(300):
        op = rng.choice(["lookup", "lookup", "fill", "stage", "publish", "discard", "evict",
                         "plan", "unpin"])
        a = int(rng.integers(0, 3))
        ns = int(rng.integers(0, 2))
        path = paths[int(rng.integers(len(paths)))]
        committed, staged = m.versions(a)
        assert (committed, staged) == (o.committed[a], o.staged.get(a, 0))
        if op == "lookup":
            v = staged if (staged and rng.random() < 0.3) else committed
            d, s_, da = (float(x) for x in rng.uniform(0, 2, size=3))
            got = m.lookup(ns, a, v, path, d, s_, da)
            assert list(got) == o.lookup(ns, a, v, path, d, s_, da), step
            if len(got) and rng.random() < 0.4:  # the request runs: it holds its blocks
                m.pin(got)
                o.pin(list(got))
                held.append(list(got))
        elif op == "unpin" and held:
            blocks = held.pop(int(rng.integers(len(held))))
            m.unpin(blocks)
            o.unpin(blocks)
        elif op == "fill":
            # prefill what the lookup did not match, under the bound version
            v = staged if (staged and rng.random() < 0.5) else committed
            matched = o.lookup(ns, a, v, path)
            assert list(m.lookup(ns, a, v, path)) == matched
            need = len(path) // BS - len(matched)
            if need > sum(st == "free" for st in o.state):
                continue
            blocks = m.alloc(need, v)
            assert list(blocks) == o.alloc(need, v)
            rec = m.insert(ns, a, v, path, blocks, first=len(matched))
            assert list(rec) == o.insert(ns, a, v, path, list(blocks), first=len(matched))
        elif op == "stage" and not staged:
            v = next_version[a]
            next_version[a] += 1
            m.stage(a, v)
            o.stage(a, v)
        elif op == "publish" and staged:
            assert m.publish(a) == o.publish(a)
        elif op == "discard" and staged:
            pinned = any(o.pins.get(b, 0) for k, b in o.records.items()
                         if k[2] == a and k[3] == staged)
            if pinned:  # refused while an active request holds its KV
                with pytest.raises(lk.LocalError):
                    m.discard_staged(a)
            else:
                assert m.discard_staged(a) == o.discard_staged(a)
        elif op == "evict":
            target = int(rng.integers(0, nb + 1))
            freed = m.evict(target)
            assert list(freed) == o.evict(target), step
            assert not set(freed) & {b for h in held for b in h}, step
        elif op == "plan" and staged:
            plan = m.plan_stale_prefill(a, 4)
            assert plan == o.plan_stale_prefill(a, 4), step
            for node, cov, tot in plan:
                ns_, toks = m.path(node)
                assert (ns_, list(toks)) == o.path(node)
        assert np.array_equal(m.tags(), np.array(o.tags, dtype=np.int32)), step
        assert m.stats() == o.stats(), step
    # every score agrees at the end
    for node in range(m.stats()[2]):
        for a in adapters:
            for v in range(adapters[a], next_version[a]):
                hp, ha, hkv, keep = m.scores(node, a, v)
                assert _close(hp, o.h_p(node)) and _close(ha, o.h_a(a, v))
                assert _close(hkv, o.h_kv(node, a, v)) and _close(keep, o.keep(node, a, v))


def test_staged_coverage_is_private_until_published():
    m = lk.KVManager(64)
    m.set_committed(0, 1000)
    toks = np.arange(200, dtype=np.int32)
    old = m.alloc(12, 1000)
    m.insert(7, 0, 1000, toks, old)
    m.stage(0, 1001)
    (node, cov, tot), = m.plan_stale_prefill(0, 8)
    assert (cov, tot) == (0, 12)
    new = m.alloc(12, 1001)
    m.insert(7, 0, 1001, toks, new)
    tags = m.tags()
    assert np.all(tags[old] == 1000) and np.all(tags[new] == 1001)
    assert np.array_equal(m.lookup(7, 0, 1000, toks), old)   # foreground before publish
    assert m.publish(0) == 1000
    assert np.array_equal(m.lookup(7, 0, 1001, toks), new)   # after publish
    assert m.versions(0) == (1001, 0)
    # the superseded coverage is the coldest: it goes first
    freed = m.evict(64 - 24 + 12)
    assert sorted(freed) == sorted(old)
    assert np.all(m.tags()[old] == 0)


def test_errors_leave_the_manager_unchanged():
    m = lk.KVManager(8)
    with pytest.raises(lk.LocalError):
        m.stage(0, 5)                          # adapter not registered
    m.set_committed(0, 10)
    with pytest.raises(lk.LocalError):
        m.stage(0, 10)                         # not a new version
    with pytest.raises(lk.LocalError):
        m.publish(0)                           # nothing staged
    with pytest.raises(lk.LocalError):
        m.alloc(9, 10)                         # more than the pool
    b = m.alloc(2, 10)
    with pytest.raises(lk.LocalError):
        m.insert(0, 0, 11, np.arange(32), b)   # blocks tagged 10, not 11
    with pytest.raises(lk.LocalError):
        m.insert(0, 0, 10, np.arange(32), b, first=1)  # block 0 not recorded
    with pytest.raises(lk.LocalError):
        m.insert(0, 0, 10, np.arange(20), b)   # 2 blocks need 32 tokens
    with pytest.raises(lk.LocalError):
        m.release([b[0], b[0]])                # repeated id
    assert m.stats() == (6, 0, 0)              # no node was made
    assert list(m.insert(0, 0, 10, np.arange(32), b)) == [1, 1]
    with pytest.raises(lk.LocalError):
        m.release(b)                           # recorded, not allocated
    with pytest.raises(lk.LocalError):
        lk.KVManager(4, dict(lambda_p=1.0))    # decay must be < 1
    assert m.stats() == (6, 2, 3)


def test_a_pinned_block_survives_eviction_and_is_not_reallocated():
    # §5.4: the KV an active request holds is not an offload candidate.
    m = lk.KVManager(16)
    m.set_committed(0, 1000)
    hot, cold = np.arange(64, dtype=np.int32), np.arange(100, 148, dtype=np.int32)
    bh = m.alloc(4, 1000)
    m.insert(0, 0, 1000, hot, bh)
    bc = m.alloc(3, 1000)
    m.insert(0, 0, 1000, cold, bc)
    held = m.lookup(0, 0, 1000, hot)
    assert np.array_equal(held, bh)
    m.pin(held)
    freed = m.evict(16)                       # ask for everything
    assert sorted(freed) == sorted(bc)        # only the unpinned path goes
    assert np.all(m.tags()[bh] == 1000)
    fresh = m.alloc(12, 1000)                 # every free block, none of the held ones
    assert not set(fresh) & set(bh)
    with pytest.raises(lk.LocalError):
        m.alloc(1, 1000)                      # the pool is exhausted, the pins stand
    m.release(fresh)
    m.unpin(held)
    assert sorted(m.evict(16)) == sorted(bh)
    with pytest.raises(lk.LocalError):
        m.unpin(held)                         # no pins left
    with pytest.raises(lk.LocalError):
        m.pin(bh)                             # freed blocks cannot be pinned


def test_a_version_belongs_to_one_adapter():
    # one tag must tell adapters apart: a version another adapter has used is
    # refused, committed or staged, and nothing changes
    m = lk.KVManager(8)
    m.set_committed(0, 1000)
    with pytest.raises(lk.LocalError):
        m.set_committed(1, 1000)
    m.set_committed(1, 2000)
    with pytest.raises(lk.LocalError):
        m.stage(1, 1000)
    m.stage(0, 1001)
    with pytest.raises(lk.LocalError):
        m.set_committed(2, 1001)
    assert m.versions(1) == (2000, 0) and m.versions(0) == (1000, 1001)
    m.set_committed(1, 2000)                  # its own version again is fine


def test_discard_waits_for_pinned_staged_records():
    m = lk.KVManager(8)
    m.set_committed(0, 1000)
    m.stage(0, 1001)
    b = m.alloc(2, 1001)
    m.insert(0, 0, 1001, np.arange(32, dtype=np.int32), b)
    m.pin(b[:1])
    with pytest.raises(lk.LocalError):
        m.discard_staged(0)
    assert m.versions(0) == (1000, 1001) and m.stats()[1] == 2
    m.unpin(b[:1])
    assert m.discard_staged(0) == 2
