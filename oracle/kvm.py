"""Oracle of the host-side KV manager (test infrastructure only).

A deliberately plain model of the version-aware KV management of §5, to be
compared call by call with the manager of local_kv.h. It keeps flat
dictionaries keyed by whole token paths and recomputes every ranking by
scanning them: no trie, no heaps, no incremental bookkeeping.

  §5.1  a record (namespace, token path, adapter, version) -> KV block is
        reusable only by a request whose validity key matches in every
        component; matching is by whole 16-token blocks, longest prefix first.
  §5.2  prefix heat H_P per path, adapter heat H_A per (adapter, version),
        H <- lambda H + (1 - lambda) * signal per request;
        H_KV = (eps + H_P)(eps + H_A)(1 + alpha_L min(L, L_max) / L_max);
        Pi_keep = H_KV * C_recompute / max(1, B); lower Pi_keep is evicted first.
  §5.3  a trained version is staged (foreground keeps binding the committed
        one), hot prefixes are re-prefilled under it, publication commits it.
  §5.4  offload: the KV an active request holds is not eligible; eligible
        records are ordered by (Pi_keep ascending, larger footprint B first)
        and the shortest prefix of that order whose footprint reaches the
        target is released.
  §4.3  a discarded staged version leaves no coverage.

Readings where the paper is silent (they are the manager's documented
behaviour, not taken from its code): one request = one tick of the heat
clock, decay applied lazily as lambda ** (ticks elapsed); every trie node on
the request's token path gets the use signal (prefix heat is
adapter-independent); the staged version of an adapter receives the urgency
signal zeta at staging and at each request routed to that adapter; the
recompute cost of one block at covered length L is 16 (c_tok + c_ctx L);
ties in a ranking go to the smaller node or block id; node ids count trie
nodes in creation order, a namespace's root first; a record becomes an
offload candidate only once no record of the same adapter state lies below
it (a record past a missing one could never be matched), so the order is
re-evaluated after each release; an active request marks the blocks it holds
by pinning them (a count per block); version numbers identify one adapter
each (a version used by one adapter is refused for every other), so a block's
tag alone tells the adapter and the version apart.
"""
from __future__ import annotations

from typing import Dict, List, Optional, Tuple

BS = 16

DEFAULTS = dict(lambda_p=0.9, lambda_a=0.9, beta=0.5, chi=0.5, eta=0.5, zeta=1.0,
                eps=0.01, alpha_l=1.0, l_max=4096.0, c_tok=1.0, c_ctx=1.0 / 4096.0,
                block_bytes=1.0)


class KVMOracle:
    def __init__(self, num_blocks: int, params: Optional[dict] = None):
        self.p = dict(DEFAULTS)
        self.p.update(params or {})
        self.num_blocks = num_blocks
        self.tags = [0] * num_blocks
        self.state = ["free"] * num_blocks
        self.node_ids: Dict[Tuple[int, tuple], int] = {}   # (ns, path) -> id
        self.node_of: List[Tuple[int, tuple]] = []
        self.records: Dict[Tuple[int, tuple, int, int], int] = {}  # -> block
        self.hp: Dict[int, Tuple[float, int]] = {}          # node -> (h, tick)
        self.ha: Dict[Tuple[int, int], Tuple[float, int]] = {}
        self.committed: Dict[int, int] = {}
        self.staged: Dict[int, int] = {}
        self.seen: Dict[int, set] = {}
        self.version_owner: Dict[int, int] = {}  # version -> the adapter that has used it
        self.pins: Dict[int, int] = {}           # block -> active requests holding it
        self.now = 0

    # ---- heat (§5.2) ----
    def _decayed(self, table, key, lam):
        if key not in table:
            return 0.0
        h, t = table[key]
        return h if t == self.now else h * lam ** (self.now - t)

    def _bump(self, table, key, lam, signal):
        table[key] = (self._decayed(table, key, lam) + (1.0 - lam) * signal, self.now)

    def h_p(self, node):
        return self._decayed(self.hp, node, self.p["lambda_p"])

    def h_a(self, adapter, version):
        return self._decayed(self.ha, (adapter, version), self.p["lambda_a"])

    def h_kv(self, node, adapter, version):
        p = self.p
        L = float(len(self.node_of[node][1]))
        return ((p["eps"] + self.h_p(node)) * (p["eps"] + self.h_a(adapter, version)) *
                (1.0 + p["alpha_l"] * min(L, p["l_max"]) / p["l_max"]))

    def keep(self, node, adapter, version):
        p = self.p
        L = float(len(self.node_of[node][1]))
        cost = BS * (p["c_tok"] + p["c_ctx"] * L)
        return self.h_kv(node, adapter, version) * cost / max(1.0, p["block_bytes"])

    # ---- trie nodes (ids in creation order) ----
    def _node(self, ns, path, create):
        key = (ns, tuple(path))
        if key not in self.node_ids:
            if not create:
                return None
            self.node_ids[key] = len(self.node_of)
            self.node_of.append(key)
        return self.node_ids[key]

    # ---- adapters ----
    def set_committed(self, a, v):
        assert a not in self.staged and self.version_owner.get(v, a) == a
        self.committed[a] = v
        self.seen.setdefault(a, set()).add(v)
        self.version_owner[v] = a

    def stage(self, a, v):
        assert a in self.committed and a not in self.staged and v not in self.seen[a]
        assert self.version_owner.get(v, a) == a
        self.staged[a] = v
        self.seen[a].add(v)
        self.version_owner[v] = a
        self._bump(self.ha, (a, v), self.p["lambda_a"], self.p["zeta"])

    def publish(self, a):
        old = self.committed[a]
        self.committed[a] = self.staged.pop(a)
        return old

    def discard_staged(self, a):
        v = self.staged[a]
        gone = [k for k in self.records if k[2] == a and k[3] == v]
        assert not any(self.pins.get(self.records[k], 0) for k in gone)
        del self.staged[a]
        for k in gone:
            self._free(self.records.pop(k))
        return len(gone)

    # ---- blocks ----
    def _free(self, b):
        self.state[b] = "free"
        self.tags[b] = 0

    def alloc(self, n, version):
        free = [b for b in range(self.num_blocks) if self.state[b] == "free"]
        assert len(free) >= n
        for b in free[:n]:
            self.state[b] = "allocated"
            self.tags[b] = version
        return free[:n]

    def release(self, blocks):
        for b in blocks:
            assert self.state[b] == "allocated"
            self._free(b)

    def pin(self, blocks):
        assert all(self.state[b] == "recorded" for b in blocks)
        for b in blocks:
            self.pins[b] = self.pins.get(b, 0) + 1

    def unpin(self, blocks):
        need = {}
        for b in blocks:
            need[b] = need.get(b, 0) + 1
        assert all(self.pins.get(b, 0) >= n for b, n in need.items())
        for b in blocks:
            self.pins[b] -= 1
            if not self.pins[b]:
                del self.pins[b]

    # ---- prefix table (§5.1) ----
    def lookup(self, ns, a, v, tokens, d_prefix=0.0, s_prefix=0.0, d_adapter=0.0,
               max_blocks=None):
        p = self.p
        tokens = list(tokens)
        nb = len(tokens) // BS
        max_blocks = nb if max_blocks is None else max_blocks
        self.now += 1
        self._node(ns, (), True)  # the namespace's root exists from its first use
        out, matching = [], True
        for i in range(nb):
            node = self._node(ns, tokens[:BS * (i + 1)], False)
            if node is None:
                break
            self._bump(self.hp, node, p["lambda_p"],
                       1.0 + p["beta"] * d_prefix + p["chi"] * s_prefix)
            key = (ns, tuple(tokens[:BS * (i + 1)]), a, v)
            if matching and key in self.records and len(out) < max_blocks:
                out.append(self.records[key])
            else:
                matching = False
        staged = self.staged.get(a)
        self._bump(self.ha, (a, v), p["lambda_a"],
                   1.0 + p["eta"] * d_adapter + (p["zeta"] if staged == v else 0.0))
        if staged is not None and staged != v:
            self._bump(self.ha, (a, staged), p["lambda_a"], p["zeta"])
        return out

    def insert(self, ns, a, v, tokens, blocks, first=0):
        tokens = list(tokens)
        assert first + len(blocks) <= len(tokens) // BS
        for j in range(first):  # the path is recorded up to `first`
            assert (ns, tuple(tokens[:BS * (j + 1)]), a, v) in self.records
        self._node(ns, (), True)
        rec = []
        for i, b in enumerate(blocks):
            assert self.state[b] == "allocated" and self.tags[b] == v
            path = tuple(tokens[:BS * (first + i + 1)])
            self._node(ns, path, True)
            key = (ns, path, a, v)
            if key in self.records:
                rec.append(0)
            else:
                self.records[key] = b
                self.state[b] = "recorded"
                rec.append(1)
        return rec

    def _has_child_record(self, ns, path, a, v):
        return any(k[0] == ns and k[2] == a and k[3] == v and len(k[1]) == len(path) + BS
                   and k[1][:len(path)] == path for k in self.records)

    # ---- stale-coverage prefill (§5.3) ----
    def plan_stale_prefill(self, a, max_prefixes=8):
        c, s = self.committed[a], self.staged[a]
        cands = []
        for (ns, path, aa, vv), _ in self.records.items():
            if aa != a or vv != c or self._has_child_record(ns, path, a, c):
                continue
            depth = len(path) // BS
            cov = 0
            while cov < depth and (ns, path[:BS * (cov + 1)], a, s) in self.records:
                cov += 1
            if cov == depth:
                continue
            node = self.node_ids[(ns, path)]
            cands.append((-self.h_kv(node, a, s), node, cov, depth))
        cands.sort()
        return [(node, cov, depth) for _, node, cov, depth in cands[:max_prefixes]]

    def path(self, node):
        ns, path = self.node_of[node]
        return ns, list(path)

    # ---- retention and offload (§5.2, §5.4) ----
    def evict(self, n_free):
        """Release records until n_free blocks are free: among the eligible
        ones (not pinned, nothing of the same adapter state below), the first
        in the order (Pi_keep ascending, larger footprint B first, smaller
        block id), one at a time."""
        freed = []
        B = self.p["block_bytes"]  # every record owns one block
        while sum(st == "free" for st in self.state) < n_free:
            cands = []
            for (ns, path, a, v), b in self.records.items():
                if self.pins.get(b, 0) or self._has_child_record(ns, path, a, v):
                    continue
                node = self.node_ids[(ns, path)]
                cands.append(((self.keep(node, a, v), -B, b), b, (ns, path, a, v)))
            if not cands:
                break
            cands.sort(key=lambda c: c[0])
            _, b, key = cands[0]
            del self.records[key]
            self._free(b)
            freed.append(b)
        return freed

    def stats(self):
        return (sum(st == "free" for st in self.state), len(self.records), len(self.node_of))
