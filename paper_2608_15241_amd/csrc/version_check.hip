// local_block_version_check: the stale (request, block) list, its length and
// the valid-token count of every request (§5.1 validity key; §1: stale
// coverage is rejected at lookup, never reused).
//
// Two launches, both one workgroup per request:
//   count: per request, the number of stale blocks (into the workspace) and
//          the live tokens of its non-stale blocks (valid_tokens[b]);
//   emit:  per request, its output offset = sum of the counts of earlier
//          requests, then the stale pairs in ascending j, compacted with
//          wavefront ballots. The order is the canonical (b, j) order for
//          any number of workgroups, so the result is exact and
//          deterministic without atomics.
// (One launch for small tables, as a single workgroup scanning stale flags in
// table order or as per-request workgroups recounting the earlier requests,
// measured no faster: the check is bound by its chain of dependent loads.)
#include "common.hpp"

namespace localk {
namespace {

constexpr int kVcThreads = 256;
constexpr int kVcWaves = kVcThreads / kWave;

// Stale: the tag differs, or the id is outside the pool (never read then).
__device__ __forceinline__ bool is_stale(const int32_t* __restrict__ table_row,
                                         const int32_t* __restrict__ block_version,
                                         int64_t num_blocks, int32_t rv, int j) {
  const int32_t p = table_row[j];
  return p < 0 || p >= num_blocks || block_version[p] != rv;
}

__device__ __forceinline__ int owned_blocks(int L, int max_blocks) {
  return L <= 0 ? 0 : min((L + kBlockSize - 1) / kBlockSize, max_blocks);
}

// Sums two ints over the workgroup; every thread gets the totals.
template <int WAVES = kVcWaves>
__device__ __forceinline__ void block_sum2(int& a, int& b, int* lds) {
  for (int off = kWave / 2; off > 0; off >>= 1) {
    a += __shfl_xor(a, off);
    b += __shfl_xor(b, off);
  }
  const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
  if (lane == 0) {
    lds[2 * wave] = a;
    lds[2 * wave + 1] = b;
  }
  __syncthreads();
  a = 0;
  b = 0;
  for (int w = 0; w < WAVES; ++w) {
    a += lds[2 * w];
    b += lds[2 * w + 1];
  }
  __syncthreads();
}

// Stale pairs of request b in ascending j from `running` on (capped), with
// wavefront ballots; returns the new running count. All threads must call it.
template <int THREADS>
__device__ int64_t emit_request(const int32_t* row, int nb, const int32_t* block_version,
                                int64_t num_blocks, int rv, int b, int64_t running,
                                int32_t* stale_pairs, int64_t cap, int* wave_tot) {
  constexpr int WAVES = THREADS / kWave;
  const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
  for (int base = 0; base < nb; base += THREADS) {
    const int j = base + threadIdx.x;
    const bool st = j < nb && is_stale(row, block_version, num_blocks, rv, j);
    const uint64_t mask = __ballot(st);
    const int before = __popcll(mask & ((1ull << lane) - 1ull));
    if (lane == 0) wave_tot[wave] = __popcll(mask);
    __syncthreads();
    int wave_off = 0, total = 0;
    for (int w = 0; w < WAVES; ++w) {
      if (w < wave) wave_off += wave_tot[w];
      total += wave_tot[w];
    }
    if (st) {
      const int64_t idx = running + wave_off + before;
      if (idx < cap) {
        stale_pairs[2 * idx] = b;
        stale_pairs[2 * idx + 1] = j;
      }
    }
    running += total;
    __syncthreads();
  }
  return running;
}

__global__ __launch_bounds__(kVcThreads) void version_count_kernel(
    const int32_t* __restrict__ block_table, int max_blocks,
    const int32_t* __restrict__ ctx_lens,
    const int32_t* __restrict__ block_version, int64_t num_blocks,
    const int32_t* __restrict__ req_version, int32_t* __restrict__ counts,
    int32_t* __restrict__ valid_tokens) {
  __shared__ int lds[2 * kVcWaves];
  const int b = blockIdx.x;
  const int L = ctx_lens[b];
  const int nb = owned_blocks(L, max_blocks);
  const int rv = req_version[b];
  const int32_t* row = block_table + static_cast<int64_t>(b) * max_blocks;
  int n_stale = 0, valid = 0;
  for (int j = threadIdx.x; j < nb; j += kVcThreads) {
    if (is_stale(row, block_version, num_blocks, rv, j))
      ++n_stale;
    else
      valid += min(kBlockSize, L - j * kBlockSize);
  }
  block_sum2(n_stale, valid, lds);
  if (threadIdx.x == 0) {
    counts[b] = n_stale;
    valid_tokens[b] = valid;
  }
}

__global__ __launch_bounds__(kVcThreads) void version_emit_kernel(
    const int32_t* __restrict__ block_table, int B, int max_blocks,
    const int32_t* __restrict__ ctx_lens,
    const int32_t* __restrict__ block_version, int64_t num_blocks,
    const int32_t* __restrict__ req_version,
    const int32_t* __restrict__ counts, int32_t* __restrict__ stale_pairs,
    int64_t cap, int32_t* __restrict__ n_stale_out) {
  __shared__ int lds[2 * kVcWaves];
  __shared__ int wave_tot[kVcWaves];
  const int b = blockIdx.x;
  // offset of request b = counts[0] + ... + counts[b-1]
  int off = 0, dummy = 0;
  for (int i = threadIdx.x; i < b; i += kVcThreads) off += counts[i];
  block_sum2(off, dummy, lds);

  const int L = ctx_lens[b];
  const int nb = owned_blocks(L, max_blocks);
  const int rv = req_version[b];
  const int32_t* row = block_table + static_cast<int64_t>(b) * max_blocks;
  const int64_t running = emit_request<kVcThreads>(row, nb, block_version, num_blocks, rv, b,
                                                   off, stale_pairs, cap, wave_tot);
  if (b == B - 1 && threadIdx.x == 0) *n_stale_out = static_cast<int32_t>(running);
}

__global__ void write_zero_kernel(int32_t* p) { *p = 0; }

}  // namespace
}  // namespace localk

using namespace localk;

extern "C" local_status_t local_block_version_check(
    const int32_t* block_table, int32_t B, int32_t max_blocks,
    const int32_t* ctx_lens, int32_t block_size,
    const int32_t* block_version, int64_t num_blocks, const int32_t* req_version,
    int32_t* stale_pairs, int64_t cap, int32_t* n_stale,
    int32_t* valid_tokens, void* ws, size_t* ws_bytes, void* stream) {
  if (!ws_bytes) return local_fail(LOCAL_ERR_WORKSPACE, "version_check: ws_bytes is NULL");
  if (B < 0 || max_blocks < 1 || num_blocks < 1 || cap < 0)
    return local_fail(LOCAL_ERR_SHAPE,
                      "version_check: B=%d max_blocks=%d num_blocks=%lld cap=%lld", B,
                      max_blocks, (long long)num_blocks, (long long)cap);
  if (block_size != kBlockSize)
    return local_fail(LOCAL_ERR_UNSUPPORTED, "version_check: block_size %d (only 16)",
                      block_size);
  const size_t need = static_cast<size_t>(B > 0 ? B : 1) * sizeof(int32_t);
  if (!ws) {
    *ws_bytes = need;
    return LOCAL_OK;
  }
  if (*ws_bytes < need)
    return local_fail(LOCAL_ERR_WORKSPACE, "version_check: workspace %zu < %zu", *ws_bytes,
                      need);
  if (!n_stale || (B > 0 && (!block_table || !ctx_lens || !block_version ||
                             !req_version || !valid_tokens)) ||
      (cap > 0 && !stale_pairs))
    return local_fail(LOCAL_ERR_NULL, "version_check: NULL pointer argument");
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (B == 0) {
    write_zero_kernel<<<1, 1, 0, s>>>(n_stale);
    return local_check_launch("version_check");
  }
  int32_t* counts = static_cast<int32_t*>(ws);
  version_count_kernel<<<B, kVcThreads, 0, s>>>(block_table, max_blocks, ctx_lens,
                                                block_version, num_blocks, req_version,
                                                counts, valid_tokens);
  version_emit_kernel<<<B, kVcThreads, 0, s>>>(block_table, B, max_blocks, ctx_lens,
                                               block_version, num_blocks, req_version,
                                               counts, stale_pairs, cap, n_stale);
  return local_check_launch("version_check");
}
