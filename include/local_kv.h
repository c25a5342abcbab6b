/*
 * local_kv.h — C ABI of the host-side KV cache manager that produces the
 * block tables and version tags the kernels of local.h consume.
 *
 * It implements the version-aware KV management of §5:
 *   - §5.1 validity keys: a KV record is reusable only when its key
 *     kappa = (token span, context namespace, adapter, adapter version)
 *     matches the request. Records live in a radix-indexed prefix table: one
 *     token trie per context namespace whose nodes are 16-token blocks, each
 *     node holding one physical KV block per (adapter, version) that covers
 *     it, so a token path shared by several adapter states is stored once.
 *   - §5.2 hot-prefix statistics: a decayed prefix heat H_P per trie node
 *     and a decayed adapter heat H_A per (adapter, version), their product
 *     H_KV with a capped length term, and the retention priority
 *     Pi_keep = H_KV * C_recompute / max(1, B) that orders eviction.
 *   - §5.3 stale-coverage prefill: a newly trained adapter version is staged
 *     (private: foreground requests keep binding the committed version), the
 *     manager plans which hot prefixes to re-prefill under it, the caller
 *     runs those chunks with the kernels under the staged version, and
 *     publication makes the staged version the committed one.
 *   - §5.4 priority-based retention and offload: records held by an active
 *     request (pinned, below) are never offload candidates; the others are
 *     released coldest first (Pi_keep ascending, larger footprint first),
 *     the shortest prefix of that order that reaches the target.
 *   - §4.3 failed work creates no reusable coverage: discarding a staged
 *     version drops every record made under it.
 *
 * Conventions
 * -----------
 *  Memory      Every pointer is HOST memory owned by the caller, except the
 *              manager itself (created and destroyed by the calls below) and
 *              the tag array returned by local_kvm_tags, which the manager
 *              owns. Nothing here touches the GPU.
 *  Blocks      Physical block ids 0 .. num_blocks-1 of the KV pools passed to
 *              the kernels. A block is free, allocated (handed to the caller,
 *              not yet recorded) or recorded (owned by one record). A
 *              recorded block may also be pinned by the requests that hold
 *              it (local_kvm_pin): pinned blocks are never evicted.
 *  Versions    A version number belongs to the first adapter that uses it
 *              (committed or staged); every other adapter is refused it, so
 *              that a block's tag alone identifies both the adapter and the
 *              version of the validity key.
 *  Tags        local_kvm_tags returns the version tag of every block, the
 *              `block_version` array the kernels read (the caller copies it
 *              to the device). An allocated or recorded block carries the
 *              version its KV is written under; a free block carries 0, which
 *              no request binds (versions are >= 1). Because a staged version
 *              is bound only by the re-prefill chunks that write it, KV under
 *              it is private until publication with no tag change, and after
 *              publication the blocks of the superseded version fail the
 *              kernels' tag test for every request that binds the new one.
 *  Heat clock  Every local_kvm_lookup is one request and advances the clock
 *              by one; heat decays by lambda per tick, applied lazily when a
 *              value is read or updated.
 *  Errors      Arguments are validated before anything changes; on error the
 *              manager is unchanged and local_last_error() (local.h) says why.
 *              The manager is not thread-safe: one thread at a time.
 *  Determinism Every result is a function of the call sequence alone (ties in
 *              any ranking are broken by the smaller node or block id).
 */
#ifndef LOCAL_KV_H
#define LOCAL_KV_H

#include <stdint.h>

#include "local.h"

#ifdef __cplusplus
extern "C" {
#endif

typedef struct local_kvm local_kvm_t;

/* Coefficients of §5.2. All must be finite; lambda_p and lambda_a in (0, 1),
 * eps > 0, l_max > 0, the others >= 0. */
typedef struct {
  double lambda_p;    /* decay of prefix heat per request                     */
  double lambda_a;    /* decay of adapter heat per request                    */
  double beta;        /* weight of predicted downstream demand in H_P         */
  double chi;         /* weight of cross-agent sharing in H_P                 */
  double eta;         /* weight of predicted demand in H_A                    */
  double zeta;        /* weight of staged-version urgency in H_A              */
  double eps;         /* floor of each factor of H_KV                         */
  double alpha_l;     /* weight of the length term of H_KV                    */
  double l_max;       /* length cap of the length term, tokens                */
  double c_tok;       /* recompute cost per token of a block ...              */
  double c_ctx;       /* ... plus this much per token per token of context    */
  double block_bytes; /* resident footprint B of one recorded block           */
} local_kvm_params_t;

/* Fills *p with the defaults: lambda 0.9 (both), beta = chi = eta = 0.5,
 * zeta = 1, eps = 0.01, alpha_l = 1, l_max = 4096, c_tok = 1,
 * c_ctx = 1/4096, block_bytes = 1. */
void local_kvm_default_params(local_kvm_params_t* p);

/* A manager of `num_blocks` (>= 1) free blocks; params NULL = defaults.
 * Returns NULL on invalid arguments (message in local_last_error()). */
local_kvm_t* local_kvm_create(int32_t num_blocks, const local_kvm_params_t* params);
void local_kvm_destroy(local_kvm_t* m);

/* Tags of all blocks, [num_blocks]; valid until the next call that changes
 * the manager. */
const int32_t* local_kvm_tags(const local_kvm_t* m);

/* ---- adapters (§4.2: foreground requests bind the last committed version;
 * §5.3: a trained version is staged, then published) ---- */

/* Registers adapter `adapter` (>= 0) with committed version `version`
 * (>= 1), or sets the committed version of a registered adapter that has no
 * staged version. LOCAL_ERR_SHAPE when another adapter has used `version`. */
local_status_t local_kvm_set_committed(local_kvm_t* m, int32_t adapter, int32_t version);

/* Stages `version` (>= 1, different from the committed one and from every
 * version the adapter has had, and never used by another adapter) for a
 * registered adapter with no staged version. Its adapter heat gets the
 * staged-urgency signal (g_A = 1). */
local_status_t local_kvm_stage(local_kvm_t* m, int32_t adapter, int32_t version);

/* Publication: the staged version becomes the committed one. *old_version
 * (may be NULL) receives the superseded version, whose records stay resident
 * as stale coverage until evicted. */
local_status_t local_kvm_publish(local_kvm_t* m, int32_t adapter, int32_t* old_version);

/* A staged version that will not be published (failed training, §4.3): every
 * record under it is dropped and its blocks freed; *n_freed (may be NULL)
 * receives their number. Blocks allocated under it and not yet recorded
 * stay with the caller, who releases them. LOCAL_ERR_SHAPE (nothing dropped)
 * while a record under it is pinned: the chunk holding it must end first. */
local_status_t local_kvm_discard_staged(local_kvm_t* m, int32_t adapter, int32_t* n_freed);

/* *committed and *staged (either may be NULL) of a registered adapter;
 * *staged = 0 when none. */
local_status_t local_kvm_versions(const local_kvm_t* m, int32_t adapter, int32_t* committed,
                                  int32_t* staged);

/* ---- blocks ---- */

/* Allocates the n (>= 0) free blocks of smallest id into blocks[0..n) and
 * tags them `version` (>= 1): the version their KV will be written under.
 * LOCAL_ERR_SHAPE when fewer than n are free (then evict first). */
local_status_t local_kvm_alloc(local_kvm_t* m, int32_t n, int32_t version, int32_t* blocks);

/* Returns allocated, unrecorded blocks to the pool (tag 0): blocks of a
 * failed chunk, or blocks local_kvm_insert did not record. */
local_status_t local_kvm_release(local_kvm_t* m, const int32_t* blocks, int32_t n);

/* Pins the recorded blocks blocks[0..n) for an active request (§5.4: the
 * active request's KV state is not an offload candidate), typically the
 * blocks its local_kvm_lookup matched, for as long as it runs. Pins count:
 * requests sharing a block pin it once each. LOCAL_ERR_SHAPE (nothing
 * pinned) if any block is not recorded. */
local_status_t local_kvm_pin(local_kvm_t* m, const int32_t* blocks, int32_t n);

/* Drops one pin of each of blocks[0..n) (a block listed k times drops k).
 * LOCAL_ERR_SHAPE (nothing changed) if a block has fewer pins than that. */
local_status_t local_kvm_unpin(local_kvm_t* m, const int32_t* blocks, int32_t n);

/* ---- the prefix table (§5.1) ---- */

/* One request of context namespace `ns`, adapter `adapter` bound to
 * `version`, whose prompt is tokens[0..n_tokens). Matching is by whole
 * 16-token blocks: blocks[0..*n_matched) receive the physical blocks of the
 * longest prefix whose every block has a record under (adapter, version)
 * (*n_matched <= max_blocks; the rest of the prompt must be prefilled). Heat
 * (§5.2), refreshed only along the request's path: the clock advances, every
 * trie node on the request's token path gets the use signal
 * H_P <- l H_P + (1 - l)(1 + beta d_prefix + chi s_prefix), whether or not it
 * holds a record for this adapter state; H_A(adapter, version) gets
 * (1 + eta d_adapter + zeta g) with g = 1 for a staged version; and a staged
 * version of the adapter other than `version` gets (zeta). `blocks` may be
 * NULL when max_blocks is 0. */
local_status_t local_kvm_lookup(local_kvm_t* m, int32_t ns, int32_t adapter, int32_t version,
                                const int32_t* tokens, int64_t n_tokens, double d_prefix,
                                double s_prefix, double d_adapter, int32_t* blocks,
                                int32_t max_blocks, int32_t* n_matched);

/* Records that blocks[i] (allocated and tagged `version`) now holds the KV of
 * block first + i, tokens [16 (first + i), 16 (first + i) + 16), of the path
 * tokens[0..n_tokens) under (ns, adapter, version), for i < n_blocks, with
 * first + n_blocks <= n_tokens / 16. The first `first` blocks of the path
 * must already be recorded under that adapter state (as after a lookup that
 * matched them), so that an adapter state's records always form a prefix of
 * each path. recorded[i] = 1 when the block was recorded, 0 when the node
 * already had a record for this adapter state (that record stays; the caller
 * releases blocks[i]). recorded may be NULL. */
local_status_t local_kvm_insert(local_kvm_t* m, int32_t ns, int32_t adapter, int32_t version,
                                const int32_t* tokens, int64_t n_tokens, int32_t first,
                                const int32_t* blocks, int32_t n_blocks, int32_t* recorded);

/* ---- stale-coverage prefill (§5.3) ---- */

/* For an adapter with a staged version s and committed version c: the hot
 * prefixes to warm under s. Candidates are the trie nodes p that end a path
 * of records under (adapter, c) (no child has one) and whose path is not
 * fully recorded under s. They are ranked by the KV hotness the coverage
 * would have under s, H_KV((p, s)), largest first (ties: smaller node id),
 * and the first max_prefixes are returned: nodes[i], covered[i] = leading
 * blocks of the path already recorded under s, total[i] = blocks of the
 * path. The caller prefills blocks covered[i] .. total[i] of each (in chunks
 * of its choice) under s and inserts them. *n_out <= max_prefixes. */
local_status_t local_kvm_plan_stale_prefill(local_kvm_t* m, int32_t adapter,
                                            int32_t max_prefixes, int32_t* nodes,
                                            int32_t* covered, int32_t* total, int32_t* n_out);

/* The token path of trie node `node`: *ns, *n_tokens = 16 * depth, and, when
 * max_tokens >= *n_tokens, the tokens into tokens[0..*n_tokens). */
local_status_t local_kvm_path(const local_kvm_t* m, int32_t node, int32_t* ns, int32_t* tokens,
                              int64_t max_tokens, int64_t* n_tokens);

/* ---- retention and offload (§5.2, §5.4) ---- */

/* Releases records until at least `n_free` blocks are free or no eligible
 * record is left (the target release R is n_free minus the free blocks). A
 * record is eligible when it is not pinned and no record of the same adapter
 * state lies below it in the trie (a record past a missing one could never
 * be matched; a parent becomes eligible once its last such child goes).
 * Eligible records go in the offload order of §5.4, Pi_keep ascending, then
 * the larger footprint B first (every record owns one block, so B is equal),
 * then the smaller block id: the shortest prefix of that order reaching R.
 * Released blocks are freed (tag 0) and written to freed[0..*n_freed) up to
 * max_freed entries (freed may be NULL when max_freed is 0); *n_freed counts
 * them all. The KV of a released record is the caller's to move to host
 * memory first, if it wants it back later. */
local_status_t local_kvm_evict(local_kvm_t* m, int32_t n_free, int32_t* freed, int32_t max_freed,
                               int32_t* n_freed);

/* ---- inspection ---- */

/* H_P of `node`, H_A of (adapter, version), H_KV and Pi_keep of the record
 * (node, adapter, version) as they stand at the current clock (any output
 * may be NULL; the record need not exist). Reading does not change them. */
local_status_t local_kvm_scores(const local_kvm_t* m, int32_t node, int32_t adapter,
                                int32_t version, double* h_p, double* h_a, double* h_kv,
                                double* keep);

/* Counts: free blocks, recorded blocks, trie nodes (roots included). */
local_status_t local_kvm_stats(const local_kvm_t* m, int32_t* n_free, int32_t* n_recorded,
                               int32_t* n_nodes);

#ifdef __cplusplus
}
#endif

#endif /* LOCAL_KV_H */
