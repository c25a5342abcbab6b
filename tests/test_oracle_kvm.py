"""Pins of the KV-manager oracle against what §5 fixes independently of it:
closed forms of the decayed heat, hand-evaluated H_KV and Pi_keep, and the
validity-key, publication and eviction semantics on worked examples."""
import math

import pytest

from oracle.kvm import BS, KVMOracle

A, V, V2 = 3, 1000, 1001


def toks(n, base=0):
    return list(range(base, base + n))


def test_prefix_heat_is_a_geometric_series():
    # k requests over one path with signal u = 1 (+ beta d + chi s):
    # H_P = (1 + beta d + chi s)(1 - lambda^k)  (the §5.2 recursion from 0)
    o = KVMOracle(8)
    o.set_committed(A, V)
    o.insert(0, A, V, toks(32), o.alloc(2, V))
    for k in range(1, 6):
        o.lookup(0, A, V, toks(32), d_prefix=2.0, s_prefix=1.0)
        want = (1 + 0.5 * 2.0 + 0.5 * 1.0) * (1 - 0.9 ** k)
        for node in (1, 2):
            assert math.isclose(o.h_p(node), want, rel_tol=1e-12)


def test_untouched_heat_decays_by_lambda_per_request():
    o = KVMOracle(8)
    o.set_committed(A, V)
    o.set_committed(7, 5)
    o.insert(0, A, V, toks(16), o.alloc(1, V))
    o.insert(0, 7, 5, toks(16, 100), o.alloc(1, 5))
    o.lookup(0, A, V, toks(16))
    h0 = o.h_p(1)
    for m in range(1, 5):
        o.lookup(0, 7, 5, toks(16, 100))  # another path: node 1 is not refreshed
        assert math.isclose(o.h_p(1), h0 * 0.9 ** m, rel_tol=1e-12)
        assert math.isclose(o.h_a(A, V), 0.1 * 0.9 ** m, rel_tol=1e-12)


def test_hkv_and_keep_by_hand():
    # two requests: H_P = 1 - 0.9^2 = 0.19 on both nodes; H_A(A, V) = 0.1 from
    # the first, decayed once (the second was for another version): 0.09.
    o = KVMOracle(8)
    o.set_committed(A, V)
    o.insert(0, A, V, toks(32), o.alloc(2, V))
    o.lookup(0, A, V, toks(32))
    o.lookup(0, A, V2, toks(32))
    assert math.isclose(o.h_p(2), 0.19, rel_tol=1e-12)
    assert math.isclose(o.h_a(A, V), 0.09, rel_tol=1e-12)
    hkv = (0.01 + 0.19) * (0.01 + 0.09) * (1 + 1.0 * 32 / 4096)
    assert math.isclose(o.h_kv(2, A, V), hkv, rel_tol=1e-12)
    assert math.isclose(o.keep(2, A, V), hkv * 16 * (1 + 32 / 4096), rel_tol=1e-12)
    # the length term saturates at L_max
    o2 = KVMOracle(8, dict(l_max=16.0, alpha_l=2.0))
    o2.set_committed(A, V)
    o2.insert(0, A, V, toks(32), o2.alloc(2, V))
    assert math.isclose(o2.h_kv(2, A, V), 0.01 * 0.01 * 3.0, rel_tol=1e-12)
    assert math.isclose(o2.h_kv(1, A, V), 0.01 * 0.01 * 3.0, rel_tol=1e-12)


def test_validity_key_every_component_must_match():
    o = KVMOracle(16)
    o.set_committed(A, V)
    o.set_committed(4, V + 7)  # versions identify one adapter each
    blocks = o.alloc(3, V)
    o.insert(0, A, V, toks(48), blocks)
    assert o.lookup(0, A, V, toks(48)) == blocks           # full match
    assert o.lookup(0, A, V, toks(40)) == blocks[:2]       # whole blocks only
    assert o.lookup(0, A, V, toks(15)) == []
    assert o.lookup(1, A, V, toks(48)) == []               # other namespace
    assert o.lookup(0, 4, V, toks(48)) == []               # other adapter
    assert o.lookup(0, A, V2, toks(48)) == []              # other version
    t = toks(48)
    t[20] = -1                                             # differs in block 1
    assert o.lookup(0, A, V, t) == blocks[:1]
    assert o.lookup(0, A, V, toks(48), max_blocks=2) == blocks[:2]


def test_stage_publish_and_discard():
    o = KVMOracle(32)
    o.set_committed(A, V)
    o.set_committed(4, 7)
    old = o.alloc(2, V)
    o.insert(0, A, V, toks(32), old)
    other = o.alloc(2, 7)
    o.insert(0, 4, 7, toks(32), other)
    o.stage(A, V2)
    (node, cov, tot), = o.plan_stale_prefill(A)
    assert (cov, tot) == (0, 2) and o.path(node) == (0, toks(32))
    new = o.alloc(2, V2)
    assert o.insert(0, A, V2, toks(32), new) == [1, 1]
    assert o.plan_stale_prefill(A) == []                   # fully warmed
    assert o.lookup(0, A, V, toks(32)) == old              # foreground: committed
    assert o.publish(A) == V
    assert o.lookup(0, A, V2, toks(32)) == new             # published coverage
    assert o.lookup(0, 4, 7, toks(32)) == other            # other adapters untouched
    # a failed staged version leaves nothing behind
    o.stage(A, 1002)
    o.insert(0, A, 1002, toks(32), o.alloc(2, 1002))
    assert o.discard_staged(A) == 2
    assert o.lookup(0, A, 1002, toks(32)) == []
    with pytest.raises(AssertionError):
        o.stage(A, V)                                      # versions are never reused


def test_eviction_takes_cold_leaves_first():
    o = KVMOracle(6)
    o.set_committed(A, V)
    hot = o.alloc(3, V)
    o.insert(0, A, V, toks(48), hot)
    cold = o.alloc(2, V)
    o.insert(0, A, V, toks(32, 500), cold)
    for _ in range(3):
        o.lookup(0, A, V, toks(48))
    # one block is free. Leaves first: the never-requested path's deepest
    # record, then its parent (now a leaf, still colder than the hot leaf),
    # then the hot path from its end
    assert o.evict(3) == [cold[1], cold[0]]
    assert o.evict(3) == []
    assert o.evict(5) == [hot[2], hot[1]]
    assert o.lookup(0, A, V, toks(48)) == hot[:1]
    assert o.stats() == (5, 1, 6)


def test_versions_identify_one_adapter():
    # One int32 tag carries both the adapter and the version of the validity
    # key only while no version number is used by two adapters: the oracle
    # refuses a version another adapter has had, committed or staged.
    o = KVMOracle(8)
    o.set_committed(A, V)
    with pytest.raises(AssertionError):
        o.set_committed(4, V)
    o.set_committed(4, 7)
    with pytest.raises(AssertionError):
        o.stage(4, V)
    o.stage(A, V2)
    with pytest.raises(AssertionError):
        o.set_committed(5, V2)
    assert o.version_owner == {V: A, 7: 4, V2: A}


def _two_paths_recorded(o):
    """Adapter A at version V: path P (3 blocks) and path Q (2 blocks); P is
    made hot by lookups, Q stays cold."""
    o.set_committed(A, V)
    P, Q = toks(48), [t + 1000 for t in toks(32)]
    bp = o.alloc(3, V)
    o.insert(0, A, V, P, bp)
    bq = o.alloc(2, V)
    o.insert(0, A, V, Q, bq)
    for _ in range(5):
        o.lookup(0, A, V, P)
    return P, Q, bp, bq


def test_offload_order_is_coldest_first_and_shortest_prefix():
    # §5.4: ascending Pi_keep; leaves before their parents (a record past a
    # missing one is never matched); the release stops at the first prefix of
    # that order that reaches the target.
    o = KVMOracle(8)
    P, Q, bp, bq = _two_paths_recorded(o)
    free0 = sum(st == "free" for st in o.state)
    assert free0 == 3
    keep_q = o.keep(o.node_ids[(0, tuple(Q))], A, V)
    keep_p = o.keep(o.node_ids[(0, tuple(P))], A, V)
    assert keep_q < keep_p                          # the cold path ranks first
    assert o.evict(free0 + 1) == [bq[1]]            # exactly one block: the cold leaf
    assert o.evict(free0 + 2) == [bq[0]]            # then its parent
    assert o.evict(free0 + 3) == [bp[2]]            # then the hot path's leaf
    assert o.evict(free0 + 3) == []                 # target reached: nothing more


def test_pinned_records_are_not_eligible():
    # §5.4: the active request's KV is not an offload candidate. A request
    # holding the hot path's blocks keeps them (and, the leaf being pinned,
    # its parents are never leaves either); the rest is released, and the
    # pinned blocks are never handed out again while pinned.
    o = KVMOracle(8)
    P, Q, bp, bq = _two_paths_recorded(o)
    held = o.lookup(0, A, V, P)
    assert held == bp
    o.pin(held)
    freed = o.evict(8)
    assert sorted(freed) == sorted(bq)               # everything but the pinned path
    assert all(o.state[b] == "recorded" for b in bp)
    assert not set(o.alloc(5, V)) & set(bp)          # never reallocated
    o.release([b for b in range(8) if o.state[b] == "allocated"])
    o.pin([bp[0]])                                   # a second request shares block 0
    o.unpin(held)
    assert o.evict(8) == [bp[2], bp[1]]              # block 0 still held
    o.unpin([bp[0]])
    assert o.evict(8) == [bp[0]]
    with pytest.raises(AssertionError):
        o.unpin([bp[0]])                             # not pinned any more
    with pytest.raises(AssertionError):
        o.pin([bp[0]])                               # not a recorded block


def test_discarding_a_staged_version_waits_for_its_pins():
    o = KVMOracle(8)
    o.set_committed(A, V)
    o.stage(A, V2)
    b = o.alloc(2, V2)
    o.insert(0, A, V2, toks(32), b)
    o.pin(b[:1])                                     # a re-prefill chunk still running
    with pytest.raises(AssertionError):
        o.discard_staged(A)
    assert o.staged == {A: V2}                       # unchanged
    o.unpin(b[:1])
    assert o.discard_staged(A) == 2
