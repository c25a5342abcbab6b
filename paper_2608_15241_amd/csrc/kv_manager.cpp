// Host-side KV cache manager (declared in local_kv.h): the radix-indexed
// prefix table of validity keys (§5.1), hot-prefix statistics and the
// retention priority (§5.2), staged adapter versions with stale-coverage
// prefill planning and publication (§5.3), and priority-based offload that
// never touches the KV an active request holds (§5.4). Plain C++; nothing here touches
// the GPU. It produces the block tables and the `block_version` tags that
// the kernels consume.
#include <algorithm>
#include <cmath>
#include <cstdint>
#include <cstring>
#include <queue>
#include <set>
#include <unordered_map>
#include <vector>

#include "../../include/local_kv.h"

local_status_t local_fail(local_status_t code, const char* fmt, ...);  // capi.hip

namespace {

constexpr int kBS = 16;  // tokens per KV block

// (adapter, version) as one key
uint64_t akey(int32_t adapter, int32_t version) {
  return (static_cast<uint64_t>(static_cast<uint32_t>(adapter)) << 32) |
         static_cast<uint32_t>(version);
}

// FNV-1a over the 16 tokens of a block: the hash of a child edge (children
// with equal hashes are told apart by their tokens)
uint64_t block_hash(const int32_t* t) {
  uint64_t h = 1469598103934665603ull;
  for (int i = 0; i < kBS; ++i) {
    uint32_t v = static_cast<uint32_t>(t[i]);
    for (int b = 0; b < 4; ++b) {
      h ^= (v >> (8 * b)) & 0xffu;
      h *= 1099511628211ull;
    }
  }
  return h;
}

// A value with lazy exponential decay: worth h * lambda^(now - tick).
struct Heat {
  double h = 0.0;
  int64_t tick = 0;
  double at(double lambda, int64_t now) const {
    return now == tick ? h : h * std::pow(lambda, static_cast<double>(now - tick));
  }
  // H <- lambda H + (1 - lambda) * signal, at clock `now`
  void update(double lambda, int64_t now, double signal) {
    h = at(lambda, now) + (1.0 - lambda) * signal;
    tick = now;
  }
};

struct Node {
  int32_t parent = -1;
  int32_t depth = 0;  // blocks from the namespace root
  int32_t ns = 0;
  int32_t tok[kBS] = {};
  Heat hp;
  std::unordered_map<uint64_t, std::vector<int32_t>> children;  // block hash -> nodes
  std::unordered_map<uint64_t, int32_t> rec;                    // akey -> physical block
};

struct AdapterState {
  int32_t committed = 0;
  int32_t staged = 0;
  std::set<int32_t> seen;  // every version the adapter has had
};

enum : uint8_t { kFree = 0, kAllocated = 1, kRecorded = 2 };

}  // namespace

struct local_kvm {
  local_kvm_params_t prm{};
  int32_t num_blocks = 0;
  std::vector<int32_t> tags;
  std::vector<uint8_t> state;
  std::set<int32_t> free_ids;
  std::vector<int32_t> owner;  // node of a recorded block
  std::vector<int32_t> pins;   // active requests holding a recorded block
  std::unordered_map<int32_t, int32_t> version_owner;  // version -> its adapter
  std::vector<Node> nodes;
  std::unordered_map<int32_t, int32_t> roots;  // namespace -> root node
  std::unordered_map<int32_t, AdapterState> adapters;
  std::unordered_map<uint64_t, Heat> ha;  // adapter heat per (adapter, version)
  int64_t now = 0;
  int32_t n_recorded = 0;

  double hp_of(int32_t node) const { return nodes[node].hp.at(prm.lambda_p, now); }
  double ha_of(uint64_t k) const {
    auto it = ha.find(k);
    return it == ha.end() ? 0.0 : it->second.at(prm.lambda_a, now);
  }
  // H_KV of the record (node, k) (§5.2): both heats floored by eps and the
  // covered length L = 16 * depth, capped at l_max
  double hkv(int32_t node, uint64_t k) const {
    const double L = static_cast<double>(kBS) * nodes[node].depth;
    return (prm.eps + hp_of(node)) * (prm.eps + ha_of(k)) *
           (1.0 + prm.alpha_l * std::min(L, prm.l_max) / prm.l_max);
  }
  // Pi_keep = H_KV * C_recompute / max(1, B); rebuilding one block of the
  // span costs 16 * (c_tok + c_ctx * L)
  double keep(int32_t node, uint64_t k) const {
    const double L = static_cast<double>(kBS) * nodes[node].depth;
    const double c = kBS * (prm.c_tok + prm.c_ctx * L);
    return hkv(node, k) * c / std::max(1.0, prm.block_bytes);
  }
  int32_t child(int32_t node, const int32_t* t) const {
    const auto& ch = nodes[node].children;
    auto it = ch.find(block_hash(t));
    if (it == ch.end()) return -1;
    for (int32_t c : it->second)
      if (std::memcmp(nodes[c].tok, t, sizeof(int32_t) * kBS) == 0) return c;
    return -1;
  }
  int32_t root(int32_t ns) {
    auto it = roots.find(ns);
    if (it != roots.end()) return it->second;
    Node r;
    r.ns = ns;
    nodes.push_back(r);
    const int32_t id = static_cast<int32_t>(nodes.size()) - 1;
    roots[ns] = id;
    return id;
  }
  int32_t add_child(int32_t node, const int32_t* t) {
    Node c;
    c.parent = node;
    c.depth = nodes[node].depth + 1;
    c.ns = nodes[node].ns;
    std::memcpy(c.tok, t, sizeof(int32_t) * kBS);
    nodes.push_back(c);
    const int32_t id = static_cast<int32_t>(nodes.size()) - 1;
    nodes[node].children[block_hash(t)].push_back(id);
    return id;
  }
  bool has_child_record(int32_t node, uint64_t k) const {
    for (const auto& kv : nodes[node].children)
      for (int32_t c : kv.second)
        if (nodes[c].rec.count(k)) return true;
    return false;
  }
  void free_block(int32_t b) {
    state[b] = kFree;
    tags[b] = 0;
    owner[b] = -1;
    free_ids.insert(b);
  }
};

namespace {

bool params_ok(const local_kvm_params_t& p) {
  const double v[] = {p.lambda_p, p.lambda_a, p.beta, p.chi,   p.eta,   p.zeta,
                      p.eps,      p.alpha_l,  p.l_max, p.c_tok, p.c_ctx, p.block_bytes};
  for (double x : v)
    if (!std::isfinite(x)) return false;
  return p.lambda_p > 0.0 && p.lambda_p < 1.0 && p.lambda_a > 0.0 && p.lambda_a < 1.0 &&
         p.eps > 0.0 && p.l_max > 0.0 && p.beta >= 0.0 && p.chi >= 0.0 && p.eta >= 0.0 &&
         p.zeta >= 0.0 && p.alpha_l >= 0.0 && p.c_tok >= 0.0 && p.c_ctx >= 0.0 &&
         p.block_bytes >= 0.0;
}

AdapterState* find_adapter(local_kvm_t* m, int32_t a) {
  auto it = m->adapters.find(a);
  return it == m->adapters.end() ? nullptr : &it->second;
}

}  // namespace

extern "C" {

void local_kvm_default_params(local_kvm_params_t* p) {
  if (!p) return;
  p->lambda_p = 0.9;
  p->lambda_a = 0.9;
  p->beta = 0.5;
  p->chi = 0.5;
  p->eta = 0.5;
  p->zeta = 1.0;
  p->eps = 0.01;
  p->alpha_l = 1.0;
  p->l_max = 4096.0;
  p->c_tok = 1.0;
  p->c_ctx = 1.0 / 4096.0;
  p->block_bytes = 1.0;
}

local_kvm_t* local_kvm_create(int32_t num_blocks, const local_kvm_params_t* params) {
  local_kvm_params_t p;
  if (params)
    p = *params;
  else
    local_kvm_default_params(&p);
  if (num_blocks < 1) {
    local_fail(LOCAL_ERR_SHAPE, "kvm_create: num_blocks=%d", num_blocks);
    return nullptr;
  }
  if (!params_ok(p)) {
    local_fail(LOCAL_ERR_SHAPE, "kvm_create: coefficients out of range");
    return nullptr;
  }
  local_kvm_t* m = new local_kvm_t;
  m->prm = p;
  m->num_blocks = num_blocks;
  m->tags.assign(num_blocks, 0);
  m->state.assign(num_blocks, kFree);
  m->owner.assign(num_blocks, -1);
  m->pins.assign(num_blocks, 0);
  for (int32_t b = 0; b < num_blocks; ++b) m->free_ids.insert(m->free_ids.end(), b);
  return m;
}

void local_kvm_destroy(local_kvm_t* m) { delete m; }

const int32_t* local_kvm_tags(const local_kvm_t* m) { return m ? m->tags.data() : nullptr; }

local_status_t local_kvm_set_committed(local_kvm_t* m, int32_t adapter, int32_t version) {
  if (!m) return local_fail(LOCAL_ERR_NULL, "kvm_set_committed: NULL manager");
  if (adapter < 0 || version < 1)
    return local_fail(LOCAL_ERR_SHAPE, "kvm_set_committed: adapter=%d version=%d", adapter,
                      version);
  AdapterState* s = find_adapter(m, adapter);
  if (s && s->staged)
    return local_fail(LOCAL_ERR_SHAPE, "kvm_set_committed: adapter %d has a staged version",
                      adapter);
  auto vo = m->version_owner.find(version);
  if (vo != m->version_owner.end() && vo->second != adapter)
    return local_fail(LOCAL_ERR_SHAPE, "kvm_set_committed: version %d belongs to adapter %d",
                      version, vo->second);
  AdapterState& st = m->adapters[adapter];
  st.committed = version;
  st.seen.insert(version);
  m->version_owner[version] = adapter;
  return LOCAL_OK;
}

local_status_t local_kvm_stage(local_kvm_t* m, int32_t adapter, int32_t version) {
  if (!m) return local_fail(LOCAL_ERR_NULL, "kvm_stage: NULL manager");
  AdapterState* s = find_adapter(m, adapter);
  if (!s) return local_fail(LOCAL_ERR_SHAPE, "kvm_stage: adapter %d not registered", adapter);
  if (s->staged)
    return local_fail(LOCAL_ERR_SHAPE, "kvm_stage: adapter %d already has staged version %d",
                      adapter, s->staged);
  if (version < 1 || s->seen.count(version))
    return local_fail(LOCAL_ERR_SHAPE, "kvm_stage: version %d not new for adapter %d", version,
                      adapter);
  auto vo = m->version_owner.find(version);
  if (vo != m->version_owner.end() && vo->second != adapter)
    return local_fail(LOCAL_ERR_SHAPE, "kvm_stage: version %d belongs to adapter %d", version,
                      vo->second);
  s->staged = version;
  s->seen.insert(version);
  m->version_owner[version] = adapter;
  m->ha[akey(adapter, version)].update(m->prm.lambda_a, m->now, m->prm.zeta);
  return LOCAL_OK;
}

local_status_t local_kvm_publish(local_kvm_t* m, int32_t adapter, int32_t* old_version) {
  if (!m) return local_fail(LOCAL_ERR_NULL, "kvm_publish: NULL manager");
  AdapterState* s = find_adapter(m, adapter);
  if (!s || !s->staged)
    return local_fail(LOCAL_ERR_SHAPE, "kvm_publish: adapter %d has no staged version", adapter);
  if (old_version) *old_version = s->committed;
  s->committed = s->staged;
  s->staged = 0;
  return LOCAL_OK;
}

local_status_t local_kvm_discard_staged(local_kvm_t* m, int32_t adapter, int32_t* n_freed) {
  if (!m) return local_fail(LOCAL_ERR_NULL, "kvm_discard_staged: NULL manager");
  AdapterState* s = find_adapter(m, adapter);
  if (!s || !s->staged)
    return local_fail(LOCAL_ERR_SHAPE, "kvm_discard_staged: adapter %d has no staged version",
                      adapter);
  const uint64_t k = akey(adapter, s->staged);
  for (const auto& node : m->nodes) {
    auto it = node.rec.find(k);
    if (it != node.rec.end() && m->pins[it->second] > 0)
      return local_fail(LOCAL_ERR_SHAPE, "kvm_discard_staged: block %d of adapter %d's staged "
                        "version is pinned by an active request", it->second, adapter);
  }
  int32_t n = 0;
  for (auto& node : m->nodes) {
    auto it = node.rec.find(k);
    if (it == node.rec.end()) continue;
    m->free_block(it->second);
    node.rec.erase(it);
    --m->n_recorded;
    ++n;
  }
  s->staged = 0;
  if (n_freed) *n_freed = n;
  return LOCAL_OK;
}

local_status_t local_kvm_versions(const local_kvm_t* m, int32_t adapter, int32_t* committed,
                                  int32_t* staged) {
  if (!m) return local_fail(LOCAL_ERR_NULL, "kvm_versions: NULL manager");
  auto it = m->adapters.find(adapter);
  if (it == m->adapters.end())
    return local_fail(LOCAL_ERR_SHAPE, "kvm_versions: adapter %d not registered", adapter);
  if (committed) *committed = it->second.committed;
  if (staged) *staged = it->second.staged;
  return LOCAL_OK;
}

local_status_t local_kvm_alloc(local_kvm_t* m, int32_t n, int32_t version, int32_t* blocks) {
  if (!m) return local_fail(LOCAL_ERR_NULL, "kvm_alloc: NULL manager");
  if (n < 0 || version < 1)
    return local_fail(LOCAL_ERR_SHAPE, "kvm_alloc: n=%d version=%d", n, version);
  if (n > 0 && !blocks) return local_fail(LOCAL_ERR_NULL, "kvm_alloc: NULL blocks");
  if (static_cast<size_t>(n) > m->free_ids.size())
    return local_fail(LOCAL_ERR_SHAPE, "kvm_alloc: %d blocks asked, %zu free", n,
                      m->free_ids.size());
  for (int32_t i = 0; i < n; ++i) {
    const int32_t b = *m->free_ids.begin();
    m->free_ids.erase(m->free_ids.begin());
    m->state[b] = kAllocated;
    m->tags[b] = version;
    blocks[i] = b;
  }
  return LOCAL_OK;
}

local_status_t local_kvm_release(local_kvm_t* m, const int32_t* blocks, int32_t n) {
  if (!m) return local_fail(LOCAL_ERR_NULL, "kvm_release: NULL manager");
  if (n < 0) return local_fail(LOCAL_ERR_SHAPE, "kvm_release: n=%d", n);
  if (n > 0 && !blocks) return local_fail(LOCAL_ERR_NULL, "kvm_release: NULL blocks");
  std::set<int32_t> seen;
  for (int32_t i = 0; i < n; ++i) {
    const int32_t b = blocks[i];
    if (b < 0 || b >= m->num_blocks || m->state[b] != kAllocated || !seen.insert(b).second)
      return local_fail(LOCAL_ERR_SHAPE, "kvm_release: block %d is not an allocated block",
                        b);
  }
  for (int32_t i = 0; i < n; ++i) m->free_block(blocks[i]);
  return LOCAL_OK;
}

local_status_t local_kvm_pin(local_kvm_t* m, const int32_t* blocks, int32_t n) {
  if (!m) return local_fail(LOCAL_ERR_NULL, "kvm_pin: NULL manager");
  if (n < 0) return local_fail(LOCAL_ERR_SHAPE, "kvm_pin: n=%d", n);
  if (n > 0 && !blocks) return local_fail(LOCAL_ERR_NULL, "kvm_pin: NULL blocks");
  for (int32_t i = 0; i < n; ++i) {
    const int32_t b = blocks[i];
    if (b < 0 || b >= m->num_blocks || m->state[b] != kRecorded)
      return local_fail(LOCAL_ERR_SHAPE, "kvm_pin: block %d is not a recorded block", b);
  }
  for (int32_t i = 0; i < n; ++i) ++m->pins[blocks[i]];
  return LOCAL_OK;
}

local_status_t local_kvm_unpin(local_kvm_t* m, const int32_t* blocks, int32_t n) {
  if (!m) return local_fail(LOCAL_ERR_NULL, "kvm_unpin: NULL manager");
  if (n < 0) return local_fail(LOCAL_ERR_SHAPE, "kvm_unpin: n=%d", n);
  if (n > 0 && !blocks) return local_fail(LOCAL_ERR_NULL, "kvm_unpin: NULL blocks");
  std::unordered_map<int32_t, int32_t> need;
  for (int32_t i = 0; i < n; ++i) {
    const int32_t b = blocks[i];
    if (b < 0 || b >= m->num_blocks || ++need[b] > m->pins[b])
      return local_fail(LOCAL_ERR_SHAPE, "kvm_unpin: block %d is not pinned that often", b);
  }
  for (int32_t i = 0; i < n; ++i) --m->pins[blocks[i]];
  return LOCAL_OK;
}

local_status_t local_kvm_lookup(local_kvm_t* m, int32_t ns, int32_t adapter, int32_t version,
                                const int32_t* tokens, int64_t n_tokens, double d_prefix,
                                double s_prefix, double d_adapter, int32_t* blocks,
                                int32_t max_blocks, int32_t* n_matched) {
  if (!m || !n_matched) return local_fail(LOCAL_ERR_NULL, "kvm_lookup: NULL argument");
  if (n_tokens < 0 || max_blocks < 0 || adapter < 0 || version < 1)
    return local_fail(LOCAL_ERR_SHAPE, "kvm_lookup: n_tokens=%lld max_blocks=%d adapter=%d "
                      "version=%d", (long long)n_tokens, max_blocks, adapter, version);
  if ((n_tokens > 0 && !tokens) || (max_blocks > 0 && !blocks))
    return local_fail(LOCAL_ERR_NULL, "kvm_lookup: NULL array");
  if (!(std::isfinite(d_prefix) && std::isfinite(s_prefix) && std::isfinite(d_adapter)) ||
      d_prefix < 0.0 || s_prefix < 0.0 || d_adapter < 0.0)
    return local_fail(LOCAL_ERR_SHAPE, "kvm_lookup: demand and sharing signals must be >= 0");
  AdapterState* st = find_adapter(m, adapter);
  if (!st) return local_fail(LOCAL_ERR_SHAPE, "kvm_lookup: adapter %d not registered", adapter);

  ++m->now;
  const local_kvm_params_t& p = m->prm;
  const uint64_t k = akey(adapter, version);
  const double sig_p = 1.0 + p.beta * d_prefix + p.chi * s_prefix;
  int32_t node = m->root(ns);
  int32_t matched = 0;
  bool matching = true;
  const int64_t nb = n_tokens / kBS;
  for (int64_t i = 0; i < nb; ++i) {
    node = m->child(node, tokens + kBS * i);
    if (node < 0) break;
    m->nodes[node].hp.update(p.lambda_p, m->now, sig_p);
    if (matching) {
      auto it = m->nodes[node].rec.find(k);
      if (it != m->nodes[node].rec.end() && matched < max_blocks) {
        blocks[matched++] = it->second;
      } else {
        matching = false;
      }
    }
  }
  const bool is_staged = st->staged == version;
  m->ha[k].update(p.lambda_a, m->now, 1.0 + p.eta * d_adapter + (is_staged ? p.zeta : 0.0));
  if (st->staged && !is_staged)
    m->ha[akey(adapter, st->staged)].update(p.lambda_a, m->now, p.zeta);
  *n_matched = matched;
  return LOCAL_OK;
}

local_status_t local_kvm_insert(local_kvm_t* m, int32_t ns, int32_t adapter, int32_t version,
                                const int32_t* tokens, int64_t n_tokens, int32_t first,
                                const int32_t* blocks, int32_t n_blocks, int32_t* recorded) {
  if (!m) return local_fail(LOCAL_ERR_NULL, "kvm_insert: NULL manager");
  if (n_tokens < 0 || n_blocks < 0 || first < 0 ||
      static_cast<int64_t>(first) + n_blocks > n_tokens / kBS || adapter < 0 || version < 1)
    return local_fail(LOCAL_ERR_SHAPE, "kvm_insert: n_tokens=%lld first=%d n_blocks=%d "
                      "adapter=%d version=%d", (long long)n_tokens, first, n_blocks, adapter,
                      version);
  if ((first + n_blocks > 0 && !tokens) || (n_blocks > 0 && !blocks))
    return local_fail(LOCAL_ERR_NULL, "kvm_insert: NULL array");
  if (!find_adapter(m, adapter))
    return local_fail(LOCAL_ERR_SHAPE, "kvm_insert: adapter %d not registered", adapter);
  std::set<int32_t> seen;
  for (int32_t i = 0; i < n_blocks; ++i) {
    const int32_t b = blocks[i];
    if (b < 0 || b >= m->num_blocks || m->state[b] != kAllocated || m->tags[b] != version ||
        !seen.insert(b).second)
      return local_fail(LOCAL_ERR_SHAPE,
                        "kvm_insert: block %d is not an allocated block tagged %d", b, version);
  }
  const uint64_t k = akey(adapter, version);
  {  // the first `first` blocks must be recorded under this adapter state
    auto rit = m->roots.find(ns);
    int32_t q = rit == m->roots.end() ? -1 : rit->second;
    for (int32_t j = 0; j < first && q >= 0; ++j) {
      q = m->child(q, tokens + kBS * static_cast<int64_t>(j));
      if (q >= 0 && !m->nodes[q].rec.count(k)) q = -1;
    }
    if (first > 0 && q < 0)
      return local_fail(LOCAL_ERR_SHAPE, "kvm_insert: the first %d blocks of the path are not "
                        "recorded under adapter %d version %d", first, adapter, version);
  }
  int32_t node = m->root(ns);
  for (int32_t j = 0; j < first; ++j) node = m->child(node, tokens + kBS * static_cast<int64_t>(j));
  for (int32_t i = 0; i < n_blocks; ++i) {
    const int32_t* t = tokens + kBS * (static_cast<int64_t>(first) + i);
    int32_t c = m->child(node, t);
    if (c < 0) c = m->add_child(node, t);
    node = c;
    const bool fresh = m->nodes[node].rec.count(k) == 0;
    if (fresh) {
      m->nodes[node].rec[k] = blocks[i];
      m->state[blocks[i]] = kRecorded;
      m->owner[blocks[i]] = node;
      ++m->n_recorded;
    }
    if (recorded) recorded[i] = fresh ? 1 : 0;
  }
  return LOCAL_OK;
}

local_status_t local_kvm_plan_stale_prefill(local_kvm_t* m, int32_t adapter,
                                            int32_t max_prefixes, int32_t* nodes,
                                            int32_t* covered, int32_t* total, int32_t* n_out) {
  if (!m || !n_out) return local_fail(LOCAL_ERR_NULL, "kvm_plan_stale_prefill: NULL argument");
  if (max_prefixes < 0)
    return local_fail(LOCAL_ERR_SHAPE, "kvm_plan_stale_prefill: max_prefixes=%d", max_prefixes);
  if (max_prefixes > 0 && (!nodes || !covered || !total))
    return local_fail(LOCAL_ERR_NULL, "kvm_plan_stale_prefill: NULL array");
  AdapterState* st = find_adapter(m, adapter);
  if (!st || !st->staged)
    return local_fail(LOCAL_ERR_SHAPE, "kvm_plan_stale_prefill: adapter %d has no staged "
                      "version", adapter);
  const uint64_t kc = akey(adapter, st->committed), ks = akey(adapter, st->staged);
  struct Cand {
    double score;
    int32_t node, cov;
  };
  std::vector<Cand> cands;
  for (int32_t id = 0; id < static_cast<int32_t>(m->nodes.size()); ++id) {
    const Node& n = m->nodes[id];
    if (!n.rec.count(kc) || m->has_child_record(id, kc)) continue;
    // leading blocks of the path already recorded under the staged version
    std::vector<int32_t> path;
    for (int32_t q = id; m->nodes[q].parent >= 0; q = m->nodes[q].parent) path.push_back(q);
    int32_t cov = 0;
    for (auto it = path.rbegin(); it != path.rend() && m->nodes[*it].rec.count(ks); ++it) ++cov;
    if (cov == n.depth) continue;
    cands.push_back({m->hkv(id, ks), id, cov});
  }
  std::sort(cands.begin(), cands.end(), [](const Cand& x, const Cand& y) {
    return x.score != y.score ? x.score > y.score : x.node < y.node;
  });
  const int32_t n = std::min<int32_t>(max_prefixes, static_cast<int32_t>(cands.size()));
  for (int32_t i = 0; i < n; ++i) {
    nodes[i] = cands[i].node;
    covered[i] = cands[i].cov;
    total[i] = m->nodes[cands[i].node].depth;
  }
  *n_out = n;
  return LOCAL_OK;
}

local_status_t local_kvm_path(const local_kvm_t* m, int32_t node, int32_t* ns, int32_t* tokens,
                              int64_t max_tokens, int64_t* n_tokens) {
  if (!m || !n_tokens) return local_fail(LOCAL_ERR_NULL, "kvm_path: NULL argument");
  if (node < 0 || node >= static_cast<int32_t>(m->nodes.size()))
    return local_fail(LOCAL_ERR_SHAPE, "kvm_path: node %d", node);
  const int64_t n = static_cast<int64_t>(kBS) * m->nodes[node].depth;
  if (ns) *ns = m->nodes[node].ns;
  *n_tokens = n;
  if (max_tokens >= n && n > 0) {
    if (!tokens) return local_fail(LOCAL_ERR_NULL, "kvm_path: NULL tokens");
    for (int32_t q = node; m->nodes[q].parent >= 0; q = m->nodes[q].parent)
      std::memcpy(tokens + kBS * static_cast<int64_t>(m->nodes[q].depth - 1), m->nodes[q].tok,
                  sizeof(int32_t) * kBS);
  }
  return LOCAL_OK;
}

local_status_t local_kvm_evict(local_kvm_t* m, int32_t n_free, int32_t* freed, int32_t max_freed,
                               int32_t* n_freed) {
  if (!m || !n_freed) return local_fail(LOCAL_ERR_NULL, "kvm_evict: NULL argument");
  if (n_free < 0 || max_freed < 0)
    return local_fail(LOCAL_ERR_SHAPE, "kvm_evict: n_free=%d max_freed=%d", n_free, max_freed);
  if (max_freed > 0 && !freed) return local_fail(LOCAL_ERR_NULL, "kvm_evict: NULL freed");
  // §5.4: eligible records (not held by an active request, nothing of the
  // same adapter state below) in the order (Pi_keep ascending, larger
  // footprint first, smaller block id), released one at a time until the
  // target is reached: the shortest prefix of the order that reaches it. A
  // parent becomes eligible when its last such child goes. Every record owns
  // one block, so the footprints are equal and the second key never decides.
  struct Cand {
    double keep, bytes;
    int32_t block, node;
    uint64_t k;
  };
  auto later = [](const Cand& x, const Cand& y) {  // min-heap on (keep, -bytes, block)
    if (x.keep != y.keep) return x.keep > y.keep;
    if (x.bytes != y.bytes) return x.bytes < y.bytes;
    return x.block > y.block;
  };
  const double bytes = m->prm.block_bytes;
  auto eligible = [&](int32_t node, uint64_t k, int32_t block) {
    return m->pins[block] == 0 && !m->has_child_record(node, k);
  };
  std::priority_queue<Cand, std::vector<Cand>, decltype(later)> heap(later);
  for (int32_t id = 0; id < static_cast<int32_t>(m->nodes.size()); ++id)
    for (const auto& r : m->nodes[id].rec)
      if (eligible(id, r.first, r.second))
        heap.push({m->keep(id, r.first), bytes, r.second, id, r.first});
  int32_t n = 0;
  while (static_cast<int64_t>(m->free_ids.size()) < n_free && !heap.empty()) {
    const Cand c = heap.top();
    heap.pop();
    m->nodes[c.node].rec.erase(c.k);
    m->free_block(c.block);
    --m->n_recorded;
    if (n < max_freed) freed[n] = c.block;
    ++n;
    const int32_t par = m->nodes[c.node].parent;
    if (par >= 0) {
      auto it = m->nodes[par].rec.find(c.k);
      if (it != m->nodes[par].rec.end() && eligible(par, c.k, it->second))
        heap.push({m->keep(par, c.k), bytes, it->second, par, c.k});
    }
  }
  *n_freed = n;
  return LOCAL_OK;
}

local_status_t local_kvm_scores(const local_kvm_t* m, int32_t node, int32_t adapter,
                                int32_t version, double* h_p, double* h_a, double* h_kv,
                                double* keep) {
  if (!m) return local_fail(LOCAL_ERR_NULL, "kvm_scores: NULL manager");
  if (node < 0 || node >= static_cast<int32_t>(m->nodes.size()))
    return local_fail(LOCAL_ERR_SHAPE, "kvm_scores: node %d", node);
  const uint64_t k = akey(adapter, version);
  if (h_p) *h_p = m->hp_of(node);
  if (h_a) *h_a = m->ha_of(k);
  if (h_kv) *h_kv = m->hkv(node, k);
  if (keep) *keep = m->keep(node, k);
  return LOCAL_OK;
}

local_status_t local_kvm_stats(const local_kvm_t* m, int32_t* n_free, int32_t* n_recorded,
                               int32_t* n_nodes) {
  if (!m) return local_fail(LOCAL_ERR_NULL, "kvm_stats: NULL manager");
  if (n_free) *n_free = static_cast<int32_t>(m->free_ids.size());
  if (n_recorded) *n_recorded = m->n_recorded;
  if (n_nodes) *n_nodes = static_cast<int32_t>(m->nodes.size());
  return LOCAL_OK;
}

}  // extern "C"
