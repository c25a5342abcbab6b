/*
 * local.h — C ABI of the mixed-adapter LoRA step and version-tagged paged
 * attention ("LOCAL: Enabling Learning On-device Contiguously for Agent LLMs").
 *
 * The library implements the data-parallel step that every foreground request
 * of the runtime shares:
 *   - a projection made of a frozen base weight plus a low-rank adapter delta,
 *     with every token routed to its own adapter (§2.2, "LoRA adapters": many
 *     adapters share one frozen base model and each request is routed to its
 *     adapter);
 *   - attention over a paged KV cache whose blocks carry the adapter version
 *     that produced them, so that KV written under another version is rejected
 *     (§1 challenge (2) and §5.1: the adapter and its version are part of the
 *     validity key kappa; §3: a publish stales only KV owned by that adapter);
 *  and the backward of the projection for the training chunks that produce
 *  new adapter versions (adapter gradients and the input gradient).
 *  The host-side KV manager and cooperative scheduler have C ABIs of their
 *  own (local_kv.h, local_sched.h) in the same library.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 *  Memory      Every pointer is DEVICE memory owned by the caller. The library
 *              allocates nothing and keeps no pointer after the call returns.
 *              All tensors are dense, row-major and contiguous in the layout
 *              stated per argument.
 *  bf16        `uint16_t` storage of IEEE bfloat16. Conversions to bf16 inside
 *              the library round to nearest even.
 *  Streams     `stream` is a hipStream_t passed as `void*` (NULL = the null
 *              stream). All work is enqueued asynchronously on it; outputs are
 *              valid once the stream has reached that point.
 *  Workspace   Scratch device memory is supplied by the caller. Call once with
 *              `ws == NULL`: the required size is written to `*ws_bytes`, the
 *              call returns LOCAL_OK and launches nothing. Then call with
 *              `ws != NULL` and `*ws_bytes` >= that size. The size depends only
 *              on the host-side scalar arguments. The workspace needs no
 *              initial contents and its contents after the call are undefined.
 *              Calls that share one workspace must be ordered on one stream.
 *  Errors      Arguments are validated on the host before anything is
 *              launched; on error nothing is launched and nothing is written.
 *              `local_last_error()` returns a message for the calling thread's
 *              most recent failure. Values held in device memory (block ids,
 *              lengths, adapter indices) cannot be checked on the host: they
 *              are the caller's contract, stated per argument.
 *  Version tags are read-only. The library never writes `block_version`: tags
 *              belong to the KV manager, which changes them only when an
 *              adapter version is published (§4.2, §5.3: in-progress adapter
 *              state and the KV it produces stay private until publication;
 *              §4.3: failed work creates no reusable coverage).
 *
 * KV block pool layout (one attention layer)
 * ------------------------------------------
 *  The pool holds `num_blocks` physical blocks of BS = 16 token slots for Hkv
 *  KV heads of head dimension D (D = 64 or 128). K and V use different
 *  in-block orders so that the matrix-core operands load as contiguous rows:
 *    k_cache  [num_blocks][Hkv][D/8][BS][8]   K(p,g,slot,d) at
 *             (((p*Hkv + g)*(D/8) + d/8)*BS + slot)*8 + d%8
 *    v_cache  [num_blocks][Hkv][D][BS]        V(p,g,slot,d) at
 *             ((p*Hkv + g)*D + d)*BS + slot
 *  A (block, head) pair therefore owns one contiguous 16*D*2-byte tile in each
 *  of k_cache and v_cache. A multi-layer pool is the caller's business: it
 *  passes the base pointers of one layer's K and V pools.
 *
 *  Logical position pi of request b lives in physical block
 *  block_table[b*max_blocks + pi/16], slot pi%16. Request b owns
 *  nb_b = min(ceil(ctx_lens[b]/16), max_blocks) logical blocks; table entries
 *  beyond them are never read. Block ids should lie in [0, num_blocks); an
 *  id outside that range is never dereferenced and its block is treated as
 *  stale (so a corrupt table degrades to excluded context, never to a wild
 *  memory access).
 *
 * Staleness (one rule for every entry point)
 * ------------------------------------------
 *  Logical block j < nb_b of request b is STALE iff its id p =
 *  block_table[b][j] lies outside [0, num_blocks) or
 *      block_version[p] != req_version[b].
 *  Any inequality is stale: an older tag was produced by a superseded version,
 *  a newer one by a staged version that is not yet published (§5.3). Tags are
 *  meant to be unique across adapters (for instance a runtime-wide publish
 *  counter), so that one equality test checks both the adapter and its
 *  version of the validity key (§5.1). A stale block is excluded as a whole.
 */
#ifndef LOCAL_H_
#define LOCAL_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  LOCAL_OK = 0,
  LOCAL_ERR_NULL = 1,        /* a required pointer is NULL                    */
  LOCAL_ERR_SHAPE = 2,       /* inconsistent or non-positive sizes            */
  LOCAL_ERR_UNSUPPORTED = 3, /* a size outside what the kernels implement     */
  LOCAL_ERR_WORKSPACE = 4,   /* ws_bytes NULL, or *ws_bytes below the need    */
  LOCAL_ERR_HIP = 5          /* the HIP runtime reported an error on launch   */
} local_status_t;

/* Message for the calling thread's most recent failed call ("" if none). */
const char* local_last_error(void);

/* Library version as MAJOR*10000 + MINOR*100 + PATCH. */
int32_t local_version(void);

/*
 * local_lora_linear — mixed-adapter LoRA projection (§2.2 "LoRA adapters";
 * the adapter delta is the low-rank update of the LoRA method the paper
 * builds on).
 *
 *   y[t,n] = res[t,n] + sum_k x[t,k] W[n,k]
 *            + scale[t] * sum_{j < rank(a)} (sum_k x[t,k] A[a,j,k]) B[a,n,j]
 *   with a = adapter_idx[t]; the adapter term is absent when a < 0 and the
 *   residual term when `residual` is NULL (it carries the layer's residual
 *   stream into the output projection without a separate pass).
 *
 *   x            [T][K]               bf16, activations
 *   W            [N][K]               bf16, frozen base weight (out x in)
 *   A            [n_adapters][r_max][K]  bf16, adapter down-projections
 *   B            [n_adapters][N][r_max]  bf16, adapter up-projections
 *   ranks        [n_adapters] int32 in [1, r_max], or NULL (every rank = r_max).
 *                Rows j >= rank of A and columns j >= rank of B are never used;
 *                a rank outside [0, r_max] is clamped to that range.
 *   adapter_idx  [T] int32 in [-1, n_adapters); -1 = base projection only
 *                (any value outside [0, n_adapters) is read as -1)
 *   scale        [T] float32, the per-token adapter scale s
 *   residual     [T][N]               bf16, or NULL
 *   y            [T][N]               bf16 output; must not alias the inputs
 *
 *  Sizes: T >= 0 (T = 0 launches nothing), K and N positive multiples of 64,
 *  0 <= n_adapters <= 256, r_max a multiple of 8 in [8, 128] (ignored when
 *  n_adapters = 0, in which case A, B, ranks, adapter_idx and scale may be
 *  NULL and every adapter_idx is taken as -1).
 *  Accumulation is float32 (residual included); y is rounded once to bf16.
 *  The low-rank intermediate s*(x A^T) is rounded to bf16 before the
 *  up-projection.
 */
local_status_t local_lora_linear(
    const uint16_t* x, int64_t T, int64_t K,
    const uint16_t* W, int64_t N,
    const uint16_t* A, const uint16_t* B,
    int32_t n_adapters, int32_t r_max,
    const int32_t* ranks,
    const int32_t* adapter_idx, const float* scale,
    const uint16_t* residual,
    uint16_t* y,
    void* ws, size_t* ws_bytes, void* stream);

/*
 * local_lora_linear_grouped — G (1..4) mixed-adapter LoRA projections of the
 * same activations, e.g. the q, k and v projections of a layer (§2.2 "LoRA
 * adapters"): for every g, y[g] equals what local_lora_linear computes from
 * (x, W[g], N[g], A[g], B[g], n_adapters, r_max, ranks[g], adapter_idx,
 * scale) with no residual, up to float32 summation order.
 *
 *   W, N, A, B, ranks, y   HOST arrays of G entries: device pointers (or, for
 *                          N, the sizes) of each projection, with the layouts
 *                          of local_lora_linear. A, B and ranks may be NULL
 *                          when n_adapters = 0; ranks or an entry of it may be
 *                          NULL (every rank = r_max). The arrays are read
 *                          during the call only.
 *
 *  All projections share x, T, K, adapter_idx, scale, n_adapters and r_max;
 *  sizes as for local_lora_linear, for every N[g]. At decode sizes (T <= 256)
 *  the projections run as one virtual weight of sum N[g] rows, so one pass
 *  of launches serves all of them. Above, one shrink pass reads x once for
 *  every projection and one product covers the tiles of all of them when
 *  every N[g] is a multiple of 256; otherwise they run one after another.
 *  Errors as for local_lora_linear; LOCAL_ERR_UNSUPPORTED for G outside 1..4,
 *  LOCAL_ERR_NULL for a NULL array.
 */
local_status_t local_lora_linear_grouped(
    const uint16_t* x, int64_t T, int64_t K, int32_t G,
    const uint16_t* const* W, const int64_t* N,
    const uint16_t* const* A, const uint16_t* const* B,
    int32_t n_adapters, int32_t r_max,
    const int32_t* const* ranks,
    const int32_t* adapter_idx, const float* scale,
    uint16_t* const* y,
    void* ws, size_t* ws_bytes, void* stream);

/*
 * local_lora_grad — adapter gradients of the mixed-adapter projection, for
 * the training chunks that update adapters while the frozen base serves
 * (§2.2: adapters trained on a frozen base model; §4: background training
 * in bounded chunks). With the forward of local_lora_linear, upstream
 * gradient dy, a = adapter_idx[t], r = rank(a), j < r:
 *
 *   u[t,j] = sum_k x[t,k] A[a,j,k]          g[t,j] = scale[t] sum_n dy[t,n] B[a,n,j]
 *   dB[a,n,j] = sum_{t : adapter t = a} scale[t] dy[t,n] u[t,j]
 *   dA[a,j,k] = sum_{t : adapter t = a} g[t,j] x[t,k]
 *
 *  and dB[a,n,j] = dA[a,j,k] = 0 for j >= r and for adapters without tokens.
 *  The base weight is frozen: it has no gradient and is not an argument.
 *
 *   x            [T][K]               bf16, the forward's activations
 *   dy           [T][N]               bf16, upstream gradient of y
 *   A, B, ranks, adapter_idx, scale   as for local_lora_linear (n_adapters >= 1;
 *                                     tokens with an index outside
 *                                     [0, n_adapters) contribute nothing)
 *   dA           [n_adapters][r_max][K]  float32 output
 *   dB           [n_adapters][N][r_max]  float32 output
 *
 *  Sizes: T >= 0 (T = 0 writes zero gradients), K and N positive multiples
 *  of 64, 1 <= n_adapters <= 256, r_max a multiple of 8 in [8, 128].
 *  u and g are float32 (not rounded); every sum is float32, over the tokens
 *  of one adapter in token order within chunks of 64, chunks added in
 *  order: the result does not depend on the launch. Outputs must not alias
 *  the inputs. Errors as for local_lora_linear.
 */
local_status_t local_lora_grad(
    const uint16_t* x, int64_t T, int64_t K,
    const uint16_t* dy, int64_t N,
    const uint16_t* A, const uint16_t* B,
    int32_t n_adapters, int32_t r_max,
    const int32_t* ranks,
    const int32_t* adapter_idx, const float* scale,
    float* dA, float* dB,
    void* ws, size_t* ws_bytes, void* stream);

/*
 * local_lora_grad_grouped — adapter gradients of G (1..4) projections of the
 * same activations, e.g. the q, k and v projections of a layer (the same
 * passage as local_lora_grad): for every g, dA[g] and dB[g] equal what
 * local_lora_grad computes from (x, dy[g], N[g], A[g], B[g], ranks[g]), up
 * to float32 summation order. One call sorts the tokens once, reads x once
 * for every u_g = x A_g^T, and runs every projection's outer products and
 * reductions in one launch each.
 *
 *   dy, N, A, B, ranks, dA, dB   HOST arrays of G entries: device pointers (or,
 *                          for N, the sizes) of each projection, with the
 *                          layouts of local_lora_grad; ranks or an entry of
 *                          it may be NULL (every rank = r_max). The arrays are
 *                          read during the call only.
 *  Sizes and errors as for local_lora_grad, for every N[g];
 *  LOCAL_ERR_UNSUPPORTED for G outside 1..4, LOCAL_ERR_NULL for a NULL array.
 */
local_status_t local_lora_grad_grouped(
    const uint16_t* x, int64_t T, int64_t K, int32_t G,
    const uint16_t* const* dy, const int64_t* N,
    const uint16_t* const* A, const uint16_t* const* B,
    int32_t n_adapters, int32_t r_max,
    const int32_t* const* ranks,
    const int32_t* adapter_idx, const float* scale,
    float* const* dA, float* const* dB,
    void* ws, size_t* ws_bytes, void* stream);

/*
 * local_lora_grad_input — input gradient of the mixed-adapter projection
 * (the same passage as local_lora_grad):
 *
 *   dx[t,k] = sum_n dy[t,n] W[n,k] + sum_{j < r} g[t,j] A[a,j,k]
 *
 *  with g as above; tokens without an adapter get the base term only.
 *   dy           [T][N]   bf16
 *   Wt           [K][N]   bf16, the frozen base weight TRANSPOSED (W^T; a
 *                         frozen weight is transposed once, at load)
 *   A, B, ranks, adapter_idx, scale   as for local_lora_grad
 *   dx           [T][K]   bf16 output; must not alias the inputs
 *
 *  This is local_lora_linear applied to dy with weight Wt and the adapters
 *  transposed (B^T as the down-projection, A^T as the up-projection, built
 *  in the workspace), so its numerics are those of local_lora_linear: float32
 *  accumulation, g rounded to bf16 before the product with A, dx rounded
 *  once. Sizes and errors as for local_lora_grad (T = 0 launches nothing).
 */
local_status_t local_lora_grad_input(
    const uint16_t* dy, int64_t T, int64_t N,
    const uint16_t* Wt, int64_t K,
    const uint16_t* A, const uint16_t* B,
    int32_t n_adapters, int32_t r_max,
    const int32_t* ranks,
    const int32_t* adapter_idx, const float* scale,
    uint16_t* dx,
    void* ws, size_t* ws_bytes, void* stream);

/*
 * local_paged_attn_decode — one new token per request attends over its paged
 * KV cache with the per-block version mask (§2.2 "KV cache and prefix
 * caching"; §5.1 validity key; stale coverage is rejected, never reused).
 *
 *  First, when k_new/v_new are given, the new token's key and value are
 *  written at logical position ctx_lens[b]-1 (the decoded token is part of its
 *  own context). Then for every request b and query head h, with
 *  g = h / (Hq/Hkv):
 *    S = { pi < ctx_lens[b], pi < 16*nb_b : logical block pi/16 of b is
 *          not stale }
 *    s_pi = sm_scale * sum_d q[b,h,d] K(bt[b][pi/16], g, pi%16, d)
 *    out[b,h,:] = sum_{pi in S} softmax(s)_pi V(bt[b][pi/16], g, pi%16, :)
 *    lse[b,h]   = log sum_{pi in S} exp(s_pi)            (natural log)
 *  If S is empty, out[b,h,:] = 0 and lse[b,h] = -inf.
 *
 *   q            [B][Hq][D]  bf16
 *   k_new,v_new  [B][Hkv][D] bf16, or both NULL (nothing appended)
 *   k_cache,v_cache  pool of num_blocks blocks, layout above; written only at
 *                the appended slots
 *   block_table  [B][max_blocks] int32
 *   ctx_lens     [B] int32 in [1, 16*max_blocks] (the append is skipped when
 *                position ctx_lens[b]-1 has no block or an out-of-range id)
 *   block_version [num_blocks] int32, req_version [B] int32
 *   out          [B][Hq][D] bf16;  lse [B][Hq] float32 or NULL
 *
 *  Sizes: B >= 0, Hq % Hkv == 0, Hq/Hkv <= 16, D in {64,128},
 *  block_size == 16. The appended slots of different requests must be
 *  distinct physical slots, and no other request of the same call may read
 *  them (a request's newest slot belongs to that request alone).
 */
local_status_t local_paged_attn_decode(
    const uint16_t* q, int32_t B, int32_t Hq, int32_t Hkv, int32_t D,
    const uint16_t* k_new, const uint16_t* v_new,
    uint16_t* k_cache, uint16_t* v_cache,
    int64_t num_blocks, int32_t block_size,
    const int32_t* block_table, int32_t max_blocks,
    const int32_t* ctx_lens,
    const int32_t* block_version, const int32_t* req_version,
    float sm_scale,
    uint16_t* out, float* lse,
    void* ws, size_t* ws_bytes, void* stream);

/*
 * local_paged_attn_decode_checked — local_paged_attn_decode and
 * local_block_version_check of the same requests in one call (§5.1: the
 * stale blocks the validity key rejects are reported while attention skips
 * them; §1: stale coverage is rejected, never reused). The attention reads
 * every owned block's id and tag anyway; it records which are stale, and
 * its merge launch writes the canonical list, so the check costs no launch
 * of its own.
 *
 *  Arguments q .. lse and the results in out/lse: as local_paged_attn_decode.
 *  stale_pairs, cap, n_stale, valid_tokens: as local_block_version_check over
 *  block_table, ctx_lens, block_version (num_blocks tags), req_version, with
 *  the same results bit for bit (the (b, j) list in canonical order, the
 *  full count in *n_stale even past cap, the live tokens of valid blocks).
 *
 *  Sizes and errors as local_paged_attn_decode, and LOCAL_ERR_SHAPE for
 *  cap < 0, LOCAL_ERR_NULL for a NULL n_stale (or valid_tokens with B > 0,
 *  or stale_pairs with cap > 0), LOCAL_ERR_UNSUPPORTED for a table wider
 *  than 32 * D blocks. B = 0 writes *n_stale = 0 and nothing else.
 */
local_status_t local_paged_attn_decode_checked(
    const uint16_t* q, int32_t B, int32_t Hq, int32_t Hkv, int32_t D,
    const uint16_t* k_new, const uint16_t* v_new,
    uint16_t* k_cache, uint16_t* v_cache,
    int64_t num_blocks, int32_t block_size,
    const int32_t* block_table, int32_t max_blocks,
    const int32_t* ctx_lens,
    const int32_t* block_version, const int32_t* req_version,
    float sm_scale,
    uint16_t* out, float* lse,
    int32_t* stale_pairs, int64_t cap, int32_t* n_stale, int32_t* valid_tokens,
    void* ws, size_t* ws_bytes, void* stream);

/*
 * local_paged_attn_decode_noalloc — local_paged_attn_decode for callers that
 * cannot allocate device memory or pass a workspace: code under HIP graph
 * capture that must not call hipMalloc, tight serving loops, harnesses that
 * forbid allocation. The caller still passes every input and output.
 *
 *  Same arguments, computation, results (bit for bit) and errors as
 *  local_paged_attn_decode, without ws / ws_bytes. The split-KV partials go
 *  to a scratch array of LOCAL_DECODE_NOALLOC_SCRATCH_BYTES that the library
 *  holds in device memory, one copy per GPU it runs on, from the first call
 *  on that GPU until the process ends. The call allocates nothing and calls
 *  no allocating routine.
 *
 *  Limit: the partials need B * Hq * ceil(max_blocks / P) * (D + 2) * 4
 *  bytes (the size local_paged_attn_decode asks for), P the partition length
 *  in blocks: 32 for tables up to 256 blocks wide, 48 up to 512, 64 beyond.
 *  A call needing more than LOCAL_DECODE_NOALLOC_SCRATCH_BYTES returns
 *  LOCAL_ERR_UNSUPPORTED and launches nothing. (131072 partials at D = 128:
 *  for instance 512 requests x 32 heads with a 256-block table, or 256
 *  requests x 32 heads with a 1024-block table.)
 *  Every call on one GPU shares that GPU's scratch: calls that overlap on one
 *  GPU (different streams, or different threads' streams) race and give
 *  undefined results. Calls ordered on one stream are safe. Nothing in the
 *  scratch needs to start at zero: each call writes every partial it reads.
 */
#define LOCAL_DECODE_NOALLOC_SCRATCH_BYTES ((size_t)68157440) /* 65 MiB */

local_status_t local_paged_attn_decode_noalloc(
    const uint16_t* q, int32_t B, int32_t Hq, int32_t Hkv, int32_t D,
    const uint16_t* k_new, const uint16_t* v_new,
    uint16_t* k_cache, uint16_t* v_cache,
    int64_t num_blocks, int32_t block_size,
    const int32_t* block_table, int32_t max_blocks,
    const int32_t* ctx_lens,
    const int32_t* block_version, const int32_t* req_version,
    float sm_scale,
    uint16_t* out, float* lse, void* stream);

/*
 * local_paged_attn_prefill — a chunk of new tokens per request is appended to
 * the paged cache and attends causally over the cached prefix plus the chunk,
 * with the per-block version mask (§4.1 chunked prefill; §5.3 stale-coverage
 * prefill runs this same computation under a staged version).
 *
 *  Request b owns query rows [q_indptr[b], q_indptr[b+1]) (n_b rows; a
 *  request whose range is reversed or not inside [0, T] is skipped whole:
 *  nothing of its chunk is appended and none of its rows is written) and has
 *  ctx_lens[b] = P_b + n_b tokens after the chunk, P_b its cached prefix.
 *  When k_new/v_new are given, row t of the chunk is first written at logical
 *  position P_b + (t - q_indptr[b]). Query row i of request b (position
 *  P_b + i) then attends over
 *    S_i = { pi <= P_b + i : logical block pi/16 of b is not stale }
 *  with the same score, softmax, output and empty-set rule as decode.
 *
 *   q            [T][Hq][D] bf16;  q_indptr [B+1] int32, q_indptr[0] = 0,
 *                non-decreasing, q_indptr[B] = T, n_b <= ctx_lens[b]
 *   k_new,v_new  [T][Hkv][D] bf16, or both NULL
 *   out          [T][Hq][D] bf16;  lse [T][Hq] float32 or NULL
 *   other arguments as in decode.
 */
local_status_t local_paged_attn_prefill(
    const uint16_t* q, const int32_t* q_indptr, int32_t B, int64_t T,
    int32_t Hq, int32_t Hkv, int32_t D,
    const uint16_t* k_new, const uint16_t* v_new,
    uint16_t* k_cache, uint16_t* v_cache,
    int64_t num_blocks, int32_t block_size,
    const int32_t* block_table, int32_t max_blocks,
    const int32_t* ctx_lens,
    const int32_t* block_version, const int32_t* req_version,
    float sm_scale,
    uint16_t* out, float* lse,
    void* ws, size_t* ws_bytes, void* stream);

/*
 * local_block_version_check — report the KV blocks that the validity key
 * rejects (§5.1; §1: stale coverage is rejected at lookup, and reusing it
 * would mix hidden states of different adapter versions).
 *
 *  For request b with nb_b = min(ceil(ctx_lens[b]/16), max_blocks) blocks
 *  and j < nb_b, tok(b,j) = min(16, ctx_lens[b] - 16*j) live tokens:
 *    valid_tokens[b] = sum of tok(b,j) over the blocks that are not stale
 *    stale list      = every stale (b, j), ordered by b, then by j
 *  stale_pairs receives the first min(n, cap) entries of the list as int32
 *  pairs (b, j) (j is the LOGICAL block index; its physical id is
 *  block_table[b][j]); *n_stale receives n, the full length, even when
 *  n > cap, so a caller can detect truncation.
 *
 *   block_table  [B][max_blocks] int32;  ctx_lens [B] int32 in
 *                [0, 16*max_blocks]
 *   block_version [num_blocks] int32
 *   req_version  [B] int32
 *   stale_pairs  [cap][2] int32 (may be NULL when cap == 0)
 *   n_stale      one int32 (device)
 *   valid_tokens [B] int32
 *
 *  Sizes: B >= 0, max_blocks >= 1, num_blocks >= 1, block_size == 16,
 *  cap >= 0.
 *  The result is exact and deterministic.
 */
local_status_t local_block_version_check(
    const int32_t* block_table, int32_t B, int32_t max_blocks,
    const int32_t* ctx_lens, int32_t block_size,
    const int32_t* block_version, int64_t num_blocks,
    const int32_t* req_version,
    int32_t* stale_pairs, int64_t cap,
    int32_t* n_stale,
    int32_t* valid_tokens,
    void* ws, size_t* ws_bytes, void* stream);

/*
 * local_kv_pool_import / local_kv_pool_export — convert one layer's paged KV
 * pool between the token-major layout and this library's pool layout (§2.2
 * "KV cache": fixed-size blocks of key/value states addressed through a block
 * table). Block ids, slots and values are unchanged: the block table and the
 * tags stay valid across the conversion; only the in-block order differs.
 *
 *   token-major  k_tok, v_tok [num_blocks][Hkv][16][D] bf16: K(p,g,slot,d)
 *                at ((p*Hkv + g)*16 + slot)*D + d (V alike)
 *   library      k_cache [num_blocks][Hkv][D/8][16][8], v_cache
 *                [num_blocks][Hkv][D][16] bf16 (the pool layout above)
 *
 *  import reads k_tok, v_tok and writes k_cache, v_cache; export reads
 *  k_cache, v_cache and writes k_tok, v_tok. Every element is copied exactly
 *  (a permutation of 2-byte values, bit for bit).
 *
 *  Sizes: num_blocks >= 0 (0: nothing is launched and the pointers may be
 *  NULL), Hkv >= 1, D in {64,128}, block_size == 16. Errors: LOCAL_ERR_NULL
 *  for a NULL pool,
 *  LOCAL_ERR_SHAPE for a negative num_blocks, Hkv < 1, or pools that
 *  overlap (the conversion is not in place), LOCAL_ERR_UNSUPPORTED for
 *  another D or block_size. No workspace.
 */
local_status_t local_kv_pool_import(
    const uint16_t* k_tok, const uint16_t* v_tok,
    int64_t num_blocks, int32_t Hkv, int32_t D, int32_t block_size,
    uint16_t* k_cache, uint16_t* v_cache, void* stream);

local_status_t local_kv_pool_export(
    const uint16_t* k_cache, const uint16_t* v_cache,
    int64_t num_blocks, int32_t Hkv, int32_t D, int32_t block_size,
    uint16_t* k_tok, uint16_t* v_tok, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* LOCAL_H_ */
