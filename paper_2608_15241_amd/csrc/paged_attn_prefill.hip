// local_paged_attn_prefill: a chunk of new tokens per request is appended to
// the paged KV cache, then attends causally over cached prefix plus chunk
// with the per-block version mask (§4.1 chunked prefill; §5.3 stale-coverage
// prefill is the same computation under a staged version).
//
// Design (matrix-core bound):
//  * Append: a workgroup per (request, block of its chunk, KV head) writes
//    that block's new K slots as 16-byte pieces and its new V slots through
//    an LDS transpose (V is dim-major in the pool), as whole 32-byte dim rows
//    when the block is all new. Every attention workgroup runs after it.
//    Workgroup 0 of that launch (a launch of its own without an append)
//    writes the schedule of the attention grid: its units (a tile, or a key
//    range of a long tile) longest first, each entry with its request's
//    sizes, so an attention workgroup knows its work after one load.
//  * Attention workgroup = (tile of 128 query rows, query head h, request b):
//    4 waves of 32 rows (two 16-column MFMA tiles each). The request's
//    non-stale blocks up to the tile's causal limit are listed in ascending
//    order with ballots; then they stream, two blocks (32 keys) per step,
//    through a ring of 4 LDS stages filled by direct global-to-LDS loads:
//    each wave moves one 16*D*2-byte (block, head) tile of K or V per step,
//    in the pool's own layout, so every operand read is a contiguous LDS
//    slice, and the loads of step s + 3 go out as step s starts.
//  * S^T = K Q^T and O^T += V^T P^T on v_mfma_f32_16x16x32_bf16, the same
//    transposed formulation as decode: the score accumulator is already the
//    B operand of the value product, so no lane shuffle of P is needed.
//    Causal masking per key, dead slots past the context end zeroed in V,
//    online softmax in the log2 domain. Steps wholly past a wave's causal
//    limit skip its arithmetic (the wave still takes part in the loads).
#include <utility>

#include "common.hpp"

namespace localk {
namespace {

constexpr int kPaWaves = 4;
constexpr int kPaThreads = kPaWaves * kWave;
constexpr int kPaQT = 2;                        // 16-row query tiles per wave
constexpr int kPaRows = kPaWaves * 16 * kPaQT;  // query rows per workgroup (128)
constexpr int kPaStages = 4;                    // LDS ring depth
constexpr int kPaWindow = 256;                  // block-table entries listed per pass
constexpr float kNegBigPf = -1.0e30f;      // initial running maximum (finite)
constexpr float kMaskedScore = -3.0e38f;   // score of a key a row may not see
constexpr float kPaLazy = 8.0f;            // log2 of the largest weight before a rescale
constexpr float kPaLazyWeight = 256.0f;    // 2^kPaLazy

// max(a, b, c) in one instruction (fmaxf chains add NaN-quieting maxima)
__device__ __forceinline__ float max3f(float a, float b, float c) {
  float r;
  asm("v_max3_f32 %0, %1, %2, %3" : "=v"(r) : "v"(a), "v"(b), "v"(c));
  return r;
}
// Tiles whose causal range spans more than kPaSplitBlocks blocks are split
// into up to kPaMaxSplit key ranges of equal length, each its own workgroup;
// a merge launch combines their partial results. (With the units dispatched
// longest first, a high threshold pays: the partial results cost HBM
// traffic, and a long unit that starts first does not set the end.)
#ifndef LOCAL_PA_SPLIT_BLOCKS
#define LOCAL_PA_SPLIT_BLOCKS 96
#endif
#ifndef LOCAL_PA_MAX_SPLIT
#define LOCAL_PA_MAX_SPLIT 4
#endif
constexpr int kPaSplitBlocks = LOCAL_PA_SPLIT_BLOCKS;
constexpr int kPaMaxSplit = LOCAL_PA_MAX_SPLIT;

struct PrefillArgs {
  const uint16_t* q;
  const int32_t* q_indptr;
  const uint16_t* k_new;
  const uint16_t* v_new;
  uint16_t* k_cache;
  uint16_t* v_cache;
  const int32_t* block_table;
  const int32_t* ctx_lens;
  const int32_t* block_version;
  const int32_t* req_version;
  uint16_t* out;
  float* lse;
  float* part;  // workspace: partial results of split tiles
  int* plan_total;  // workspace: the number of units and of split tiles,
  int4* plan;       // the schedule (two int4 per unit, in dispatch order),
  int4* splits;     // the split tiles (one int4 each, in any order)
  int64_t T, num_blocks;
  int B, Hq, Hkv, group, max_blocks;
  float scale_log2;  // |sm_scale| * log2(e)
  uint32_t q_sign;   // 0x80008000 when sm_scale < 0 (q's sign bits flipped), else 0
};

__device__ __forceinline__ bool id_ok(int p, int64_t num_blocks) {
  return p >= 0 && p < num_blocks;
}

// Request b's query rows [r0, r1) form a row range of q: inside [0, T] and
// not reversed. A request whose range is not is skipped as a whole: it gets
// no unit of either grid, appends nothing and writes no output row.
__device__ __forceinline__ bool rows_ok(int r0, int r1, int64_t T) {
  return r0 >= 0 && r1 >= r0 && r1 <= T;
}

// The k-th unit of work (k >= 0), counting units from the last request
// backwards and, within a request, from its last unit, where request b has
// units(b) >= 0 of them. Returns the request (-1 when k is past the total)
// and, in *u, the unit's index within its request. The host sizes grids by
// an upper bound of the total, since the requests' sizes are device data; a
// grid mapped this way has no idle workgroups among the working ones (they
// all come at its end), and the dispatch order takes the last requests,
// commonly those with the longest prefixes, first. The wave scans 64
// requests at a time; every lane returns the same result.
template <typename Units>
__device__ int unit_from_end(int B, int k, Units units, int* u) {
  const int lane = threadIdx.x % kWave;
  for (int base = B - 1; base >= 0; base -= kWave) {
    const int bb = base - lane;
    const int n = bb >= 0 ? units(bb) : 0;
    int incl = n;  // inclusive prefix over lanes (requests base, base-1, ...)
#pragma unroll
    for (int off = 1; off < kWave; off <<= 1) {
      const int v = __shfl_up(incl, off);
      if (lane >= off) incl += v;
    }
    const int total = __shfl(incl, kWave - 1);
    if (k < total) {
      const uint64_t m = __ballot(incl > k);
      const int l0 = __ffsll(static_cast<long long>(m)) - 1;
      const int before = __shfl(incl - n, l0);
      const int nb = __shfl(n, l0);
      *u = nb - 1 - (k - before);
      return base - l0;
    }
    k -= total;
  }
  return -1;
}

// s_waitcnt encodings (gfx9 layout): wait until at most N vector memory
// operations are outstanding / until all LDS operations are done, then the
// workgroup barrier. The compiler does not track the LDS writes of direct
// loads, so these waits are explicit.
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}
__device__ __forceinline__ void wait_lgkm0_barrier() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_waitcnt(15 | (3 << 14) | (7 << 4));
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}
// one 16-byte direct load: lane l of the wave writes at lds + 16 l
__device__ __forceinline__ void lds_load16(const void* g, void* lds) {
  __builtin_amdgcn_global_load_lds(g, lds, 16, 0, 0);
}
// the same through a buffer descriptor: the lane reads at byte off of it
__device__ __forceinline__ void lds_load16(__amdgpu_buffer_rsrc_t r, uint32_t off, void* lds) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(r, lds, 16, off, 0, 0, 0);
}

// LDS reads issued exactly as written: the compiler neither pairs them into
// ds_read2 forms nor waits for them (the kernel waits on the LDS counter
// itself, then passes the registers through an empty asm so that nothing
// reads them earlier). addr is a byte address in LDS.
template <int OFF>
__device__ __forceinline__ u32x4 lds_read16(uint32_t addr) {
  u32x4 r;
  asm volatile("ds_read_b128 %0, %1 offset:%2" : "=v"(r) : "v"(addr), "i"(OFF));
  return r;
}
template <int OFF>
__device__ __forceinline__ u32x2 lds_read8(uint32_t addr) {
  u32x2 r;
  asm volatile("ds_read_b64 %0, %1 offset:%2" : "=v"(r) : "v"(addr), "i"(OFF));
  return r;
}
template <int N>
__device__ __forceinline__ void lds_wait() {  // at most N LDS operations outstanding
  static_assert(N >= 0 && N < 16, "lgkmcnt range");
  asm volatile("s_waitcnt lgkmcnt(%0)" ::"i"(N) : "memory");
}
__device__ __forceinline__ uint32_t lds_addr(const void* p) {
  return static_cast<uint32_t>(
      reinterpret_cast<uintptr_t>((const __attribute__((address_space(3))) uint8_t*)p));
}
// f(IC<0>{}), ..., f(IC<N-1>{}): loop indices usable as template arguments
template <int I>
struct IC {
  static constexpr int v = I;
};
template <typename F, int... I>
__device__ __forceinline__ void static_for_(F&& f, std::integer_sequence<int, I...>) {
  (f(IC<I>{}), ...);
}
template <int N, typename F>
__device__ __forceinline__ void static_for(F&& f) {
  static_for_(f, std::make_integer_sequence<int, N>{});
}

constexpr int kPlanThreads = 256;  // threads of the workgroup that plans the units
__device__ void plan_units(const PrefillArgs& a);

// Append. Workgroup = (one block that request b's chunk writes, KV head g),
// mapped from a 1D grid (heads fastest); the block's slots [lo, hi) are new
// (positions P_b .. L_b - 1). Thread t handles slot t / (D/8), dims
// 8 (t % (D/8)) .. +8.
template <int D>
__global__ __launch_bounds__(256) void prefill_append_kernel(PrefillArgs a) {
  constexpr int C8 = D / 8;
  __shared__ uint16_t vt[D][kBlockSize + 2];  // V of the block, dim-major (+2: banks)
  // workgroup 0 (dispatched first) plans the attention grid's units
  if (blockIdx.x == 0) {
    plan_units(a);
    return;
  }
  const unsigned bid = blockIdx.x - 1;
  const int g = bid % a.Hkv;
  int jb = 0;
  // blocks request b's chunk writes: from its first new position's block to
  // its last one's (none for an empty chunk or a chunk past the context)
  auto chunk_blocks = [&](int bb) {
    const int r0 = a.q_indptr[bb], r1 = a.q_indptr[bb + 1];
    const int n = r1 - r0;
    const int L = a.ctx_lens[bb];
    if (!rows_ok(r0, r1, a.T) || n <= 0 || L <= 0) return 0;
    const int P = max(L - n, 0);
    return (L - 1) / kBlockSize - P / kBlockSize + 1;
  };
  const int b = unit_from_end(a.B, static_cast<int>(bid / a.Hkv), chunk_blocks, &jb);
  if (b < 0) return;
  const int r0 = a.q_indptr[b], r1 = a.q_indptr[b + 1];
  if (!rows_ok(r0, r1, a.T)) return;  // never given a unit; checked before any row is read
  const int n_b = r1 - r0;
  const int L = a.ctx_lens[b], P = L - n_b;
  const int j = (P >= 0 ? P : 0) / kBlockSize + jb;  // the block
  const int lo = max(P, j * kBlockSize), hi = min(L, (j + 1) * kBlockSize);
  if (lo >= hi || j >= a.max_blocks) return;
  const int p = a.block_table[static_cast<int64_t>(b) * a.max_blocks + j];
  if (!id_ok(p, a.num_blocks)) return;  // blocks outside the pool are not written
  const int64_t tile = (static_cast<int64_t>(p) * a.Hkv + g) * (kBlockSize * D);
  for (int e = threadIdx.x; e < kBlockSize * C8; e += blockDim.x) {
    const int slot = e / C8, c = e % C8;
    const int pos = j * kBlockSize + slot;
    u32x4 vv = {0u, 0u, 0u, 0u};
    if (pos >= lo && pos < hi) {
      const int64_t row = r0 + (pos - P);
      const u32x4 kv = ld_global<u32x4>(a.k_new + (row * a.Hkv + g) * D + 8 * c);
      vv = ld_global<u32x4>(a.v_new + (row * a.Hkv + g) * D + 8 * c);
      *reinterpret_cast<u32x4*>(a.k_cache + tile + c * (kBlockSize * 8) + slot * 8) = kv;
    }
    const uint32_t w[4] = {vv.x, vv.y, vv.z, vv.w};
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      vt[8 * c + 2 * q][slot] = static_cast<uint16_t>(w[q] & 0xffffu);
      vt[8 * c + 2 * q + 1][slot] = static_cast<uint16_t>(w[q] >> 16);
    }
  }
  __syncthreads();
  const bool whole = lo == j * kBlockSize && hi == (j + 1) * kBlockSize;
  if (whole) {  // dim rows of 16 slots as two 16-byte pieces
    for (int e = threadIdx.x; e < 2 * D; e += blockDim.x) {
      const int d = e / 2, h = e % 2;
      uint32_t w[4];
#pragma unroll
      for (int q = 0; q < 4; ++q)
        w[q] = static_cast<uint32_t>(vt[d][8 * h + 2 * q]) |
               (static_cast<uint32_t>(vt[d][8 * h + 2 * q + 1]) << 16);
      *reinterpret_cast<u32x4*>(a.v_cache + tile + d * kBlockSize + 8 * h) =
          u32x4{w[0], w[1], w[2], w[3]};
    }
  } else {  // the chunk's first or last block: only its new slots
    for (int e = threadIdx.x; e < kBlockSize * D; e += blockDim.x) {
      const int d = e / kBlockSize, slot = e % kBlockSize;
      const int pos = j * kBlockSize + slot;
      if (pos >= lo && pos < hi) a.v_cache[tile + d * kBlockSize + slot] = vt[d][slot];
    }
  }
}

// Logical blocks that tile t of a request (prefix P, n_b rows) sees: up to
// its last row's position, at most the table's width.
__device__ __forceinline__ int tile_blocks(int P, int n_b, int t, int max_blocks) {
  const int lim = P + min((t + 1) * kPaRows, n_b) - 1;
  return lim < 0 ? 0 : min(lim / kBlockSize + 1, max_blocks);
}

// Key ranges a tile of nbl blocks is split into.
__device__ __forceinline__ int tile_splits(int nbl) {
  return nbl <= kPaSplitBlocks ? 1 : min(kPaMaxSplit, (nbl + kPaSplitBlocks - 1) / kPaSplitBlocks);
}

// Partial-result slot of (tile t of request b with rows from r0, head h,
// split): r0/128 + b + t is unique over the requests' tiles and below
// T/128 + B, the bound the host sizes the workspace by.
__device__ __forceinline__ int64_t part_slot(int r0, int b, int t, int h, int Hq, int split) {
  return (static_cast<int64_t>(r0 / kPaRows + b + t) * Hq + h) * kPaMaxSplit + split;
}

// Length class of the key ranges of a tile of nbl blocks split into ns:
// classes of 8 blocks of the mean range, the last one open-ended; the grid
// takes the classes longest first.
constexpr int kPaClasses = 8;
__device__ __forceinline__ int tile_class(int nbl, int ns) {
  return min((nbl / ns) >> 3, kPaClasses - 1);
}

// The unit schedule, written once per call by one workgroup of
// kPlanThreads threads before the attention grid runs. Entry k (two int4)
// names the k-th unit in dispatch order: {b, tile | split << 24 |
// nsplit << 28, r0, n} and {P, 0, 0, 0} (request b's first row, rows and
// cached prefix). Units go longest first, by length class; within a class
// from the last request backwards, a request's tiles from its last one, a
// tile's key ranges ascending. So the longest units start first, whatever
// request they belong to, and the grid ends on the short ones; an attention
// workgroup reads its unit with one load instead of deriving it.
__device__ void plan_units(const PrefillArgs& a) {
  __shared__ int scan[kPaClasses][kPlanThreads];
  __shared__ int totals[kPaClasses];
  __shared__ int n_split_tiles;
  const int tid = threadIdx.x;
  // request bb's first row, rows and prefix (false: no rows, or a bad range)
  auto rows = [&](int bb, int* r0, int* n, int* P) {
    const int q0 = a.q_indptr[bb], q1 = a.q_indptr[bb + 1];
    if (!rows_ok(q0, q1, a.T) || q1 == q0) return false;
    *r0 = q0;
    *n = q1 - q0;
    *P = a.ctx_lens[bb] - *n;
    return true;
  };
  auto count = [&](int P, int n, int (&cnt)[kPaClasses]) {
    for (int t = 0; t * kPaRows < n; ++t) {
      const int nbl = tile_blocks(P, n, t, a.max_blocks), ns = tile_splits(nbl);
      const int c = tile_class(nbl, ns);
#pragma unroll
      for (int cc = 0; cc < kPaClasses; ++cc) cnt[cc] += c == cc ? ns : 0;
    }
  };
  if (tid < kPaClasses) totals[tid] = 0;
  if (tid == 0) n_split_tiles = 0;
  __syncthreads();
  for (int bb = tid; bb < a.B; bb += kPlanThreads) {
    int r0, n, P, cnt[kPaClasses];
#pragma unroll
    for (int c = 0; c < kPaClasses; ++c) cnt[c] = 0;
    if (!rows(bb, &r0, &n, &P)) continue;
    count(P, n, cnt);
#pragma unroll
    for (int c = 0; c < kPaClasses; ++c)
      if (cnt[c]) atomicAdd(&totals[c], cnt[c]);
  }
  __syncthreads();
  int first[kPaClasses];  // next entry of each class
  {
    int acc = 0;
#pragma unroll
    for (int c = kPaClasses - 1; c >= 0; --c) {
      first[c] = acc;
      acc += totals[c];
    }
    if (tid == 0) *a.plan_total = acc;
  }
  // requests from the last backwards, kPlanThreads at a time: each thread's
  // request takes the next entries of its classes (a scan over the threads)
  for (int chunk = 0; chunk < a.B; chunk += kPlanThreads) {
    const int bb = a.B - 1 - chunk - tid;
    int r0 = 0, n = 0, P = 0, cnt[kPaClasses];
#pragma unroll
    for (int c = 0; c < kPaClasses; ++c) cnt[c] = 0;
    const bool ok = bb >= 0 && rows(bb, &r0, &n, &P);
    if (ok) count(P, n, cnt);
#pragma unroll
    for (int c = 0; c < kPaClasses; ++c) scan[c][tid] = cnt[c];
    __syncthreads();
    for (int off = 1; off < kPlanThreads; off <<= 1) {
      int v[kPaClasses];
#pragma unroll
      for (int c = 0; c < kPaClasses; ++c) v[c] = tid >= off ? scan[c][tid - off] : 0;
      __syncthreads();
#pragma unroll
      for (int c = 0; c < kPaClasses; ++c) scan[c][tid] += v[c];
      __syncthreads();
    }
    int pos[kPaClasses];
#pragma unroll
    for (int c = 0; c < kPaClasses; ++c) pos[c] = first[c] + scan[c][tid] - cnt[c];
    if (ok) {
      for (int t = (n - 1) / kPaRows; t >= 0; --t) {
        const int nbl = tile_blocks(P, n, t, a.max_blocks), ns = tile_splits(nbl);
        const int c = tile_class(nbl, ns);
        int e = 0;
#pragma unroll
        for (int cc = 0; cc < kPaClasses; ++cc) e = c == cc ? pos[cc] : e;
        for (int sp = 0; sp < ns; ++sp) {
          a.plan[2 * (e + sp)] = make_int4(bb, t | (sp << 24) | (ns << 28), r0, n);
          a.plan[2 * (e + sp) + 1] = make_int4(P, 0, 0, 0);
        }
        if (ns > 1) {  // a tile the merge launch combines
          const int i = atomicAdd(&n_split_tiles, 1);
          a.splits[i] = make_int4(bb, t | (ns << 28), r0, n);
        }
#pragma unroll
        for (int cc = 0; cc < kPaClasses; ++cc) pos[cc] += c == cc ? ns : 0;
      }
    }
#pragma unroll
    for (int c = 0; c < kPaClasses; ++c) first[c] += scan[c][kPlanThreads - 1];
    __syncthreads();  // before the next chunk rewrites the scan
  }
  if (tid == 0) a.plan_total[1] = n_split_tiles;
}

// The planner alone, for calls without an append.
__global__ __launch_bounds__(kPlanThreads) void prefill_plan_kernel(PrefillArgs a) {
  plan_units(a);
}

template <int D>
constexpr int64_t part_slot_floats() {
  return static_cast<int64_t>(kPaRows) * (D + 2);  // O [128][D], then (m, l) [128][2]
}

template <int D>
__global__ __launch_bounds__(kPaThreads, 2) void prefill_attn_kernel(PrefillArgs a) {
  constexpr int QT = kPaQT, KC = D / 32, VT = D / 16;
  constexpr int TILE = kBlockSize * D;     // elements of a (block, head) tile
  constexpr int TILE_B = 2 * TILE;         // its bytes
  constexpr int DMA = TILE_B / 1024;       // 1 KB direct loads per tile
  constexpr int STAGE_B = 4 * TILE_B;      // K and V tiles of two blocks
  extern __shared__ __attribute__((aligned(16))) uint8_t ring[];  // [kPaStages][STAGE_B]
  // the listed blocks, ascending: {logical block j, physical id}, the last
  // entry repeated once past the end (so a step's pair is one 16-byte read)
  __shared__ __attribute__((aligned(16))) int2 ent[kPaWindow + 2];
  __shared__ int wave_cnt[kPaWaves];

  // (query tile, key range, head h, request b) from a 1D grid, heads
  // fastest, the units in the planned order (longest first, so that no long
  // workgroup starts behind short ones). A tile with a long causal range is
  // split into key ranges (units of their own) so that no workgroup holds
  // far more work than the mean. Workgroups past the units leave.
  const int h = blockIdx.x % a.Hq;
  const int k = static_cast<int>(blockIdx.x / a.Hq);
  const int n_units = *a.plan_total;
  const int4 e0 = a.plan[2 * k], e1 = a.plan[2 * k + 1];
  if (k >= n_units) return;
  const int b = e0.x, qtile = e0.y & 0xffffff, split = (e0.y >> 24) & 15, n_split = e0.y >> 28;
  const int r0 = e0.z, n_b = e0.w, P = e1.x;
  const int L = P + n_b;
  const int row0 = qtile * kPaRows;
  if (row0 >= n_b) return;
  const int tid = threadIdx.x;
  const int wave = __builtin_amdgcn_readfirstlane(tid / kWave), lane = tid % kWave;
  const int col = lane % 16, kgrp = lane / 16;
  const int g = h / a.group;
  const int rv = a.req_version[b];
  const int32_t* table = a.block_table + static_cast<int64_t>(b) * a.max_blocks;

  // this unit's key range: logical blocks [j_lo, j_hi) of the tile's range
  const int nb_tile = tile_blocks(P, n_b, qtile, a.max_blocks);
  const int j_lo = split * nb_tile / n_split, j_hi = (split + 1) * nb_tile / n_split;
  // The first window's block-table entry goes out before the query, so that
  // the version loads it feeds need not wait for the query.
  int p_first = 0;
  if (j_lo + tid < j_hi) p_first = table[j_lo + tid];

  // Query columns of this wave: rows row0 + 32 wave + 16 ct + col. For a
  // negative softmax scale the query's sign bits are flipped (exact), so
  // the kernel only ever scales by |sm_scale|.
  bf16x8 qv[QT][KC];
  int qpos[QT];
  u32x4 qraw[QT][KC];
#pragma unroll
  for (int ct = 0; ct < QT; ++ct) {
    const int row = row0 + wave * 16 * QT + 16 * ct + col;
    qpos[ct] = P + row;
    const int rc = row < n_b ? row : 0;  // rows past the chunk load row 0, never stored
#pragma unroll
    for (int c = 0; c < KC; ++c)
      qraw[ct][c] =
          ld_global<u32x4>(a.q + (static_cast<int64_t>(r0 + rc) * a.Hq + h) * D + 32 * c + 8 * kgrp);
  }
  const float scl = a.scale_log2;
  const int wave_last_row = min(row0 + (wave + 1) * 16 * QT, n_b) - 1;
  const int wave_limit = P + wave_last_row;  // largest key position this wave sees
  const int wave_first = P + row0 + wave * 16 * QT;  // position of its first row

  f32x4 acc[QT][VT];
  float m_run[QT];             // running maximum in raw score units
  float l_run[QT];             // this lane's part of the running sum of p
#pragma unroll
  for (int ct = 0; ct < QT; ++ct) {
    m_run[ct] = kNegBigPf;
    l_run[ct] = 0.f;
#pragma unroll
    for (int t = 0; t < VT; ++t) acc[ct][t] = f32x4{0.f, 0.f, 0.f, 0.f};
  }

  // A ring stage holds one step (two blocks A, B): K_A [KC][1 KB], K_B
  // [KC][1 KB], then V of A as VT rows of 512 bytes (row t: dims 16t ..
  // 16t+15), then V of B alike. Within a 512-byte V row the 16-byte chunks
  // are swizzled: chunk (dim d, slots 8 half .. +8) sits at chunk index
  // 2 (d % 16) + (half ^ bit 3 of d), so that the 32 lanes of each half of a
  // value-fragment read cover 256 contiguous bytes of banks. The stage is
  // filled by NPIECE direct 1 KB loads, NPIECE / 4 per wave; lane l of a
  // piece fetches the 16 bytes that land at byte 16 l of it.
  constexpr int NPIECE = 2 * DMA + VT;
  constexpr int PPW = NPIECE / kPaWaves;
  static_assert(NPIECE % kPaWaves == 0 && STAGE_B == NPIECE * 1024, "stage layout");
  // Every wave loads from one block, so that the tile's address is
  // wave-uniform (scalar arithmetic): waves 0 and 2 read block A, waves 1
  // and 3 block B. Waves 0 and 1 load K (1 KB piece i of the tile at byte
  // 1024 i, lane l's 16 bytes at 16 l); waves 2 and 3 load V, piece i
  // holding rows 2i (lanes 0-31) and 2i + 1 (lanes 32-63), row t at byte
  // 512 t of the tile, lane l's 16 bytes at its swizzled chunk.
  static_assert(PPW == DMA && 2 * DMA == VT, "K and V pieces in separate waves");
  const bool k_wave = wave < 2;
  const bool wave_b = (wave & 1) != 0;  // the wave reads block B
  uint32_t lane_src;  // byte offset of piece 0's 16 bytes within the block's tile
  if (k_wave) {
    lane_src = static_cast<uint32_t>(16 * lane);
  } else {
    const int cidx = lane & 31;
    const int dl = cidx >> 1;  // dim within the row (d = 16 t + dl)
    const int half = (cidx & 1) ^ ((dl >> 3) & 1);
    lane_src = static_cast<uint32_t>(512 * (lane >> 5) + 32 * dl + 16 * half);
  }
  uint32_t piece_src[PPW];  // byte offsets of the lane's 16 bytes of each piece
#pragma unroll
  for (int i = 0; i < PPW; ++i) piece_src[i] = lane_src + 1024 * i;
  // this lane's value fragment in V row t of a stage (A's; B's is VT * 512
  // bytes on): dim 16 t + col, slots 4 kgrp .. +4
  const uint32_t v_off = 32 * col + 16 * ((kgrp >> 1) ^ ((col >> 3) & 1)) + 8 * (kgrp & 1);

  // ---- list the non-stale blocks of window w0 (ascending j); returns the
  // count. p_pre is the window's table entry when already loaded.
  auto build_list = [&](int w0, bool pre, int p_pre) {
    const int j = w0 + tid;
    bool ok = false;
    int p = 0;
    if (j < j_hi) {
      p = pre ? p_pre : table[j];
      ok = id_ok(p, a.num_blocks) && a.block_version[p] == rv;
    }
    const uint64_t mask = __ballot(ok);
    const int before = __popcll(mask & ((1ull << lane) - 1ull));
    if (lane == 0) wave_cnt[wave] = __popcll(mask);
    __syncthreads();
    int off = 0, n = 0;
    for (int w = 0; w < kPaWaves; ++w) {
      if (w < wave) off += wave_cnt[w];
      n += wave_cnt[w];
    }
    if (ok) {
      ent[off + before] = int2{j, p};
      if (off + before == n - 1) ent[n] = int2{j, p};
    }
    __syncthreads();
    return n;
  };
  int cnt = build_list(j_lo, true, p_first);
  // The query is waited for here (the version loads above have waited for
  // it already), before any direct load is issued: a wait for it after them
  // would wait for them too.
#pragma unroll
  for (int ct = 0; ct < QT; ++ct)
#pragma unroll
    for (int c = 0; c < KC; ++c) {
      asm volatile("" : "+v"(qraw[ct][c]));
      qv[ct][c] = as_bf16x8(qraw[ct][c] ^ a.q_sign);
    }
  for (int w0 = j_lo; w0 < j_hi; w0 += kPaWindow) {
    if (w0 != j_lo) cnt = build_list(w0, false, 0);
    if (cnt == 0) continue;
    const int steps = (cnt + 1) / 2;

    // loads of step s into ring stage `stage`: this wave's pieces. Physical
    // ids come from LDS (a load of the block table here would make the wave
    // wait for every load before it). A step's second block past the list
    // end repeats its first (never used), and steps past the last repeat the
    // last into the free stage, so every step issues the same loads and the
    // wait counts hold.
    // entries 2s and 2s + 1 of the list: {jA, pA, jB, pB}
    auto pair = [&](int s) { return *reinterpret_cast<const int4*>(&ent[2 * s]); };
    auto issue = [&](int stage, int4 e) {
      uint8_t* dst = ring + stage * STAGE_B + wave * PPW * 1024;
      const int pw = __builtin_amdgcn_readfirstlane(wave_b ? e.w : e.y);
      const int64_t tile = (static_cast<int64_t>(pw) * a.Hkv + g) * TILE;
      // a buffer descriptor of the tile (scalar registers) and the lane's
      // fixed offsets: the loads take no vector arithmetic (the immediate
      // offset of an LDS-destination buffer load would move the LDS address
      // too, so the piece offset rides in the lane's offset register)
      const __amdgpu_buffer_rsrc_t r = make_rsrc((k_wave ? a.k_cache : a.v_cache) + tile, TILE_B);
#pragma unroll
      for (int i = 0; i < PPW; ++i)
        lds_load16(r, piece_src[i], dst + 1024 * i);
    };
    // Two steps per barrier: after the barrier of steps s, s + 1 (their
    // loads were issued one pair earlier), the loads of steps s + 2, s + 3
    // go into the stages of the previous pair. The list entries a pair needs
    // (the ids its loads fetch, the blocks it computes on) are read one pair
    // ahead, so that no LDS round trip stands between the barrier and the
    // loads or the arithmetic.
    static_assert(kPaStages == 4, "two stages per pair of steps");
    issue(0, pair(0));
    issue(1, pair(min(1, steps - 1)));
    int4 e_l0 = pair(min(2, steps - 1)), e_l1 = pair(min(3, steps - 1));
    int4 e_c0 = pair(0), e_c1 = pair(min(1, steps - 1));

    auto compute = [&](int s, int4 e) {
      // the step's blocks (wave-uniform, so that their tests are scalar)
      const int jA = __builtin_amdgcn_readfirstlane(e.x);
      const bool hasB = 2 * s + 1 < cnt;
      const int jB = hasB ? __builtin_amdgcn_readfirstlane(e.z) : jA;
      if (jA * kBlockSize > wave_limit) return;  // wholly past this wave's rows
      // every key of the step precedes every row of the wave (so it is also
      // before the context end): no masking
      const bool unmasked = hasB && jB * kBlockSize + kBlockSize - 1 <= wave_first;
      // Operand reads of the stage: K of A and B (1 KB contiguous per
      // instruction), then V (slots 4 kgrp .. +4 of each block; zeroed past
      // the context end just before the value product) as single 8-byte
      // reads. Compiled, the V reads of A and B (512 bytes apart) would be
      // paired into ds_read2st64_b64, whose two addresses per lane share a
      // bank: measured on gfx950, 77 bytes per clock and compute unit
      // against 215 for single 8-byte reads and 256 for 16-byte ones.
      const uint32_t st_addr = lds_addr(ring) + static_cast<uint32_t>((s % kPaStages) * STAGE_B);
      const uint32_t k_addr = st_addr + 16 * lane;
      const uint32_t v_addr = st_addr + 2 * TILE_B + v_off;
      u32x4 kra[KC], krb[KC];
      u32x2 vra[VT], vrb[VT];
      static_for<KC>([&](auto c) {
        kra[c.v] = lds_read16<1024 * c.v>(k_addr);
        krb[c.v] = lds_read16<TILE_B + 1024 * c.v>(k_addr);
      });
      static_for<VT / 2>([&](auto t) {
        vra[t.v] = lds_read8<512 * t.v>(v_addr);
        vrb[t.v] = lds_read8<512 * (VT + t.v)>(v_addr);
      });
      lds_wait<VT>();  // the K reads have landed (the VT V reads may not)
      static_for<VT / 2>([&](auto t) {
        vra[VT / 2 + t.v] = lds_read8<512 * (VT / 2 + t.v)>(v_addr);
        vrb[VT / 2 + t.v] = lds_read8<512 * (VT + VT / 2 + t.v)>(v_addr);
      });
      bf16x8 kfa[KC], kfb[KC];
#pragma unroll
      for (int c = 0; c < KC; ++c) {
        asm volatile("" : "+v"(kra[c]), "+v"(krb[c]));
        kfa[c] = as_bf16x8(kra[c]);
        kfb[c] = as_bf16x8(krb[c]);
      }
      // S^T of both column tiles, one column tile after the other (its two
      // chains of KC MFMAs interleaved), so that the first tile's maxima can
      // start while the second's products run (raw scores: the scale is
      // applied in the exponent)
      f32x4 sA[QT], sB[QT];
#pragma unroll
      for (int ct = 0; ct < QT; ++ct) {
        sA[ct] = f32x4{0.f, 0.f, 0.f, 0.f};
        sB[ct] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int c = 0; c < KC; ++c) {
          sA[ct] = mfma16x16x32(kfa[c], qv[ct][c], sA[ct]);
          sB[ct] = mfma16x16x32(kfb[c], qv[ct][c], sB[ct]);
        }
      }
      // raw scores; near the diagonal or the context end a key a row may
      // not see gets kMaskedScore, whose weight 2^(scale (s - m)) is 0 (the
      // scale is never 0: a zero scale runs as a vanishing positive one)
      float sc[QT][8];
#pragma unroll
      for (int ct = 0; ct < QT; ++ct) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          sc[ct][i] = sA[ct][i];
          sc[ct][4 + i] = sB[ct][i];
        }
      }
      if (!unmasked) {
#pragma unroll
        for (int ct = 0; ct < QT; ++ct)
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const int posA = jA * kBlockSize + 4 * kgrp + i;
            const int posB = jB * kBlockSize + 4 * kgrp + i;
            sc[ct][i] = posA <= qpos[ct] ? sc[ct][i] : kMaskedScore;
            sc[ct][4 + i] = (hasB && posB <= qpos[ct]) ? sc[ct][4 + i] : kMaskedScore;
          }
      }
      // Slots at or past the context end may hold anything and are zeroed;
      // only a step that holds the context end (or has no second block)
      // needs it, and that is the same for the whole wave. (Here, after the
      // score products, so that those wait only for the K fragments, and
      // before the exponentials, which share one block with the value
      // products.)
      lds_wait<0>();  // the V reads have landed
      bf16x8 vf[VT];
#pragma unroll
      for (int t = 0; t < VT; ++t) {
        asm volatile("" : "+v"(vra[t]), "+v"(vrb[t]));
        vf[t] = as_bf16x8(u32x4{vra[t].x, vra[t].y, vrb[t].x, vrb[t].y});
      }
      const bool tail = !hasB || (jA + 1) * kBlockSize > L || (jB + 1) * kBlockSize > L;
      if (tail) {
        const int la = L - jA * kBlockSize - 4 * kgrp;
        const int lb = hasB ? L - jB * kBlockSize - 4 * kgrp : 0;
        const u32x4 mk = {la >= 2 ? ~0u : (la == 1 ? 0xffffu : 0u),
                          la >= 4 ? ~0u : (la == 3 ? 0xffffu : 0u),
                          lb >= 2 ? ~0u : (lb == 1 ? 0xffffu : 0u),
                          lb >= 4 ? ~0u : (lb == 3 ? 0xffffu : 0u)};
#pragma unroll
        for (int t = 0; t < VT; ++t)
          vf[t] = as_bf16x8(__builtin_bit_cast(u32x4, vf[t]) & mk);
      }
      // p = 2^(scale (s - m)) with the running maximum m, one fused
      // multiply-add and one exponent each. Lazy rescale: m moves only when
      // a column's maximum exceeds it by more than 2^kPaLazy in weight, i.e.
      // when some p exceeds 2^kPaLazy (weights up to that stay exact in
      // float32 and bf16 alike, so the result is the same softmax); then m,
      // the sums and the weights are redone, which is rare after the first
      // step. Testing the weights instead of the scores leaves the common
      // step without the cross-lane maxima.
      float pr[QT][8];
      auto weights = [&](int ct) {
        const float nms = -m_run[ct] * scl;
#pragma unroll
        for (int i = 0; i < 8; ++i) pr[ct][i] = fast_exp2(__builtin_fmaf(sc[ct][i], scl, nms));
      };
      auto rescale_if_needed = [&](int ct) {
        const float pm = max3f(max3f(pr[ct][0], pr[ct][1], pr[ct][2]),
                               max3f(pr[ct][3], pr[ct][4], pr[ct][5]), max2f(pr[ct][6], pr[ct][7]));
        if (__ballot(pm > kPaLazyWeight) != 0ull) {
          float mx = max3f(max3f(sc[ct][0], sc[ct][1], sc[ct][2]),
                           max3f(sc[ct][3], sc[ct][4], sc[ct][5]), max2f(sc[ct][6], sc[ct][7]));
          mx = max_xor32(max_xor16(mx));
          const float m_new = max2f(m_run[ct], mx);
          const float alpha = fast_exp2((m_run[ct] - m_new) * scl);
          l_run[ct] *= alpha;
#pragma unroll
          for (int t = 0; t < VT; ++t) acc[ct][t] *= alpha;
          m_run[ct] = m_new;
          weights(ct);
        }
      };
      // Each column tile's value product follows its weights; the
      // scheduling groups interleave one tile's value product with the next
      // tile's exponentials (the matrix cores and the vector unit work side
      // by side). The float32 row sums as pairwise trees.
      weights(0);
      rescale_if_needed(0);
#pragma unroll
      for (int ct = 0; ct < QT; ++ct) {
        bf16x8 pb;
#pragma unroll
        for (int i = 0; i < 8; ++i) pb[i] = static_cast<__bf16>(pr[ct][i]);
        l_run[ct] += ((pr[ct][0] + pr[ct][1]) + (pr[ct][2] + pr[ct][3])) +
                     ((pr[ct][4] + pr[ct][5]) + (pr[ct][6] + pr[ct][7]));
#pragma unroll
        for (int t = 0; t < VT; ++t) acc[ct][t] = mfma16x16x32(vf[t], pb, acc[ct][t]);
        if (ct + 1 < QT) {
          weights(ct + 1);
#pragma unroll
          for (int i = 0; i < VT; ++i) {
            __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // a value MFMA of tile ct
            __builtin_amdgcn_sched_group_barrier(0x402, 4, 0);  // exponentials of tile ct + 1
          }
          rescale_if_needed(ct + 1);
        }
      }
    };
    for (int s = 0; s < steps; s += 2) {
      // this wave's loads of steps s, s + 1 are done; after the barrier
      // everyone's are, and the stages of steps s - 2, s - 1 are free
      wait_vmcnt<0>();
      wait_lgkm0_barrier();
      issue((s + 2) % kPaStages, e_l0);
      issue((s + 3) % kPaStages, e_l1);
      const int4 c0 = e_c0, c1 = e_c1;
      e_l0 = pair(min(s + 4, steps - 1));
      e_l1 = pair(min(s + 5, steps - 1));
      e_c0 = pair(min(s + 2, steps - 1));
      e_c1 = pair(min(s + 3, steps - 1));
      compute(s, c0);
      if (s + 1 < steps) compute(s + 1, c1);
    }
    // every load has landed before the ring or the list is reused
    wait_vmcnt<0>();
    wait_lgkm0_barrier();
  }

  // ---- this wave's rows: normalised output, or the partial result of a split
#pragma unroll
  for (int ct = 0; ct < QT; ++ct) {
    float l = l_run[ct];
    l += __shfl_xor(l, 16);
    l += __shfl_xor(l, 32);
    const int rl = wave * 16 * QT + 16 * ct + col;  // row within the tile
    const int row = row0 + rl;
    if (row >= n_b) continue;
    if (n_split == 1) {
      const int64_t orow = (static_cast<int64_t>(r0 + row) * a.Hq + h);
      const float inv = l > 0.f ? 1.f / l : 0.f;
#pragma unroll
      for (int t = 0; t < VT; ++t) {
        const int d0 = 16 * t + 4 * kgrp;
        uint32_t lo = pack_bf16x2(acc[ct][t][0] * inv, acc[ct][t][1] * inv);
        uint32_t hi = pack_bf16x2(acc[ct][t][2] * inv, acc[ct][t][3] * inv);
        *reinterpret_cast<u32x2*>(a.out + orow * D + d0) = u32x2{lo, hi};
      }
      if (kgrp == 0 && a.lse)
        a.lse[orow] = l > 0.f ? (m_run[ct] * scl + __log2f(l)) * kLn2 : -INFINITY;
    } else {
      float* slot = a.part + part_slot(r0, b, qtile, h, a.Hq, split) * part_slot_floats<D>();
#pragma unroll
      for (int t = 0; t < VT; ++t)
        *reinterpret_cast<f32x4*>(slot + rl * D + 16 * t + 4 * kgrp) = acc[ct][t];
      if (kgrp == 0)
        *reinterpret_cast<float2*>(slot + kPaRows * D + 2 * rl) = float2{m_run[ct], l};
    }
  }
}

// Merge of the split tiles: workgroup = (split tile, head, group of rows),
// the split tiles from the planner's list (tiles that were not split were
// written in place). A thread owns 8 dims of one row and issues every load of
// every key range before any arithmetic.
template <int D>
__global__ __launch_bounds__(256) void prefill_merge_kernel(PrefillArgs a) {
  constexpr int TPR = D / 8;           // threads per row
  constexpr int RPW = 256 / TPR;       // rows per workgroup
  constexpr int RG = kPaRows / RPW;    // row groups per tile
  const int rg = blockIdx.x % RG;
  const int h = (blockIdx.x / RG) % a.Hq;
  // the k-th split tile of the planner's list (workgroups past it leave)
  const int k = static_cast<int>(blockIdx.x / (RG * a.Hq));
  const int n_split_tiles = a.plan_total[1];
  const int4 e0 = a.splits[k];
  if (k >= n_split_tiles) return;
  const int b = e0.x, qtile = e0.y & 0xffffff, ns = e0.y >> 28;
  const int r0 = e0.z, n_b = e0.w;
  const int rl = rg * RPW + threadIdx.x / TPR;  // row within the tile
  const int d0 = 8 * (threadIdx.x % TPR);
  if (qtile * kPaRows + rl >= n_b) return;
  const float* base = a.part + part_slot(r0, b, qtile, h, a.Hq, 0) * part_slot_floats<D>();
  float2 ml[kPaMaxSplit];
  f32x4 o0[kPaMaxSplit], o1[kPaMaxSplit];
#pragma unroll
  for (int i = 0; i < kPaMaxSplit; ++i) {
    if (i < ns) {
      const float* sl = base + i * part_slot_floats<D>();
      ml[i] = *reinterpret_cast<const float2*>(sl + kPaRows * D + 2 * rl);
      o0[i] = *reinterpret_cast<const f32x4*>(sl + rl * D + d0);
      o1[i] = *reinterpret_cast<const f32x4*>(sl + rl * D + d0 + 4);
    }
  }
  const float scl = a.scale_log2;
  float M = kNegBigPf;
#pragma unroll
  for (int i = 0; i < kPaMaxSplit; ++i)
    if (i < ns) M = fmaxf(M, ml[i].x);
  float den = 0.f;
  f32x4 n0 = {0.f, 0.f, 0.f, 0.f}, n1 = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int i = 0; i < kPaMaxSplit; ++i) {
    if (i < ns) {
      const float f = fast_exp2((ml[i].x - M) * scl);
      den += ml[i].y * f;
      n0 += o0[i] * f;
      n1 += o1[i] * f;
    }
  }
  const float inv = den > 0.f ? 1.f / den : 0.f;
  const int64_t orow = static_cast<int64_t>(r0 + qtile * kPaRows + rl) * a.Hq + h;
  *reinterpret_cast<u32x4*>(a.out + orow * D + d0) =
      u32x4{pack_bf16x2(n0[0] * inv, n0[1] * inv), pack_bf16x2(n0[2] * inv, n0[3] * inv),
            pack_bf16x2(n1[0] * inv, n1[1] * inv), pack_bf16x2(n1[2] * inv, n1[3] * inv)};
  if (d0 == 0 && a.lse) a.lse[orow] = den > 0.f ? (M * scl + __log2f(den)) * kLn2 : -INFINITY;
}

// Workspace: the split tiles' partial results (one slot per tile bound,
// head and split), then the plan: its counts in 256 bytes, the unit schedule
// (two int4 per unit: at most kPaMaxSplit per tile bound) and the list of
// split tiles (one int4 each: at most one per tile bound).
template <int D>
size_t prefill_part_bytes(int64_t T, int B, int Hq) {
  const int64_t tiles = T / kPaRows + B;
  const size_t v =
      static_cast<size_t>(tiles) * Hq * kPaMaxSplit * part_slot_floats<D>() * sizeof(float);
  return (v + 255) & ~static_cast<size_t>(255);
}
template <int D>
size_t prefill_ws_bytes(int64_t T, int B, int Hq) {
  const int64_t tiles = T / kPaRows + B;
  return prefill_part_bytes<D>(T, B, Hq) + 256 +
         static_cast<size_t>(tiles) * (2 * kPaMaxSplit + 1) * sizeof(int4);
}

template <int D>
local_status_t launch_prefill(const PrefillArgs& a, hipStream_t s) {
  if (a.k_new) {
    // a chunk of n rows spans at most n / 16 + 2 blocks: T / 16 + 2 B in all;
    // workgroup 0 plans the attention units
    const int64_t units = a.T / kBlockSize + 2LL * a.B;
    prefill_append_kernel<D><<<static_cast<unsigned>(units * a.Hkv + 1), 256, 0, s>>>(a);
    local_status_t st = local_check_launch("paged_attn_prefill (append)");
    if (st != LOCAL_OK) return st;
  } else {
    prefill_plan_kernel<<<1, kPlanThreads, 0, s>>>(a);
    local_status_t st = local_check_launch("paged_attn_prefill (plan)");
    if (st != LOCAL_OK) return st;
  }
  constexpr int kLds = kPaStages * 4 * 2 * kBlockSize * D;
  static bool done = false;
  if (!done) {  // benign race: every caller sets the same value
    (void)hipFuncSetAttribute(reinterpret_cast<const void*>(prefill_attn_kernel<D>),
                              hipFuncAttributeMaxDynamicSharedMemorySize, kLds);
    done = true;
  }
  // a chunk of n rows has at most n / 128 + 1 tiles (T / 128 + B in all),
  // each of at most kPaMaxSplit key ranges
  const int64_t tiles = a.T / kPaRows + a.B;
  prefill_attn_kernel<D>
      <<<static_cast<unsigned>(tiles * kPaMaxSplit * a.Hq), kPaThreads, kLds, s>>>(a);
  local_status_t st = local_check_launch("paged_attn_prefill");
  if (st != LOCAL_OK) return st;
  prefill_merge_kernel<D><<<static_cast<unsigned>(tiles * a.Hq * (D / 16)), 256, 0, s>>>(a);
  return local_check_launch("paged_attn_prefill (merge)");
}

}  // namespace
}  // namespace localk

using namespace localk;

extern "C" local_status_t local_paged_attn_prefill(
    const uint16_t* q, const int32_t* q_indptr, int32_t B, int64_t T, int32_t Hq,
    int32_t Hkv, int32_t D, const uint16_t* k_new, const uint16_t* v_new,
    uint16_t* k_cache, uint16_t* v_cache, int64_t num_blocks, int32_t block_size,
    const int32_t* block_table, int32_t max_blocks, const int32_t* ctx_lens,
    const int32_t* block_version, const int32_t* req_version, float sm_scale,
    uint16_t* out, float* lse, void* ws, size_t* ws_bytes, void* stream) {
  if (!ws_bytes) return local_fail(LOCAL_ERR_WORKSPACE, "paged_attn_prefill: ws_bytes is NULL");
  if (B < 0 || T < 0 || Hq <= 0 || Hkv <= 0 || max_blocks < 1 || num_blocks < 1 ||
      Hq % Hkv != 0)
    return local_fail(LOCAL_ERR_SHAPE,
                      "paged_attn_prefill: B=%d T=%lld Hq=%d Hkv=%d max_blocks=%d", B,
                      (long long)T, Hq, Hkv, max_blocks);
  if (block_size != kBlockSize || (D != 64 && D != 128))
    return local_fail(LOCAL_ERR_UNSUPPORTED, "paged_attn_prefill: block_size=%d D=%d",
                      block_size, D);
  if ((k_new == nullptr) != (v_new == nullptr))
    return local_fail(LOCAL_ERR_NULL, "paged_attn_prefill: k_new and v_new must both be set");
  if ((T / kPaRows + 2LL * B) * (kPaMaxSplit > 8 ? kPaMaxSplit : 8) * Hq >= (1LL << 31) ||
      (T / kBlockSize + 2LL * B) * Hq >= (1LL << 31))
    return local_fail(LOCAL_ERR_UNSUPPORTED, "paged_attn_prefill: T=%lld too large", (long long)T);
  const size_t need = D == 64 ? prefill_ws_bytes<64>(T, B, Hq) : prefill_ws_bytes<128>(T, B, Hq);
  if (!ws) {
    *ws_bytes = need;
    return LOCAL_OK;
  }
  if (*ws_bytes < need)
    return local_fail(LOCAL_ERR_WORKSPACE, "paged_attn_prefill: workspace %zu < %zu", *ws_bytes,
                      need);
  if (B == 0 || T == 0) return LOCAL_OK;
  if (!q || !q_indptr || !k_cache || !v_cache || !block_table || !ctx_lens ||
      !block_version || !req_version || !out)
    return local_fail(LOCAL_ERR_NULL, "paged_attn_prefill: NULL pointer argument");
  if (T > static_cast<int64_t>(16) * max_blocks * B)
    return local_fail(LOCAL_ERR_SHAPE, "paged_attn_prefill: T=%lld exceeds the block tables",
                      (long long)T);
  PrefillArgs a;
  a.q = q;
  a.q_indptr = q_indptr;
  a.k_new = k_new;
  a.v_new = v_new;
  a.k_cache = k_cache;
  a.v_cache = v_cache;
  a.block_table = block_table;
  a.ctx_lens = ctx_lens;
  a.block_version = block_version;
  a.req_version = req_version;
  a.out = out;
  a.lse = lse;
  a.T = T;
  a.num_blocks = num_blocks;
  a.B = B;
  a.Hq = Hq;
  a.Hkv = Hkv;
  a.group = Hq / Hkv;
  a.max_blocks = max_blocks;
  a.part = static_cast<float*>(ws);
  {
    const size_t pb = D == 64 ? prefill_part_bytes<64>(T, B, Hq) : prefill_part_bytes<128>(T, B, Hq);
    a.plan_total = reinterpret_cast<int*>(static_cast<char*>(ws) + pb);
    a.plan = reinterpret_cast<int4*>(static_cast<char*>(ws) + pb + 256);
    a.splits = a.plan + 2 * (T / kPaRows + B) * kPaMaxSplit;
  }
  // |sm_scale|; a zero scale (every visible key weighs the same) runs as a
  // vanishing positive one, under which masked keys still weigh exactly 0
  a.scale_log2 = fmaxf(fabsf(sm_scale) * kLog2e, 1.0e-30f);
  a.q_sign = sm_scale < 0.f ? 0x80008000u : 0u;
  hipStream_t s = static_cast<hipStream_t>(stream);
  return D == 64 ? launch_prefill<64>(a, s) : launch_prefill<128>(a, s);
}
