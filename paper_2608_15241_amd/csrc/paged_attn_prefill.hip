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
#include "common.hpp"

namespace localk {
namespace {

constexpr int kPaWaves = 4;
constexpr int kPaThreads = kPaWaves * kWave;
constexpr int kPaQT = 2;                        // 16-row query tiles per wave
constexpr int kPaRows = kPaWaves * 16 * kPaQT;  // query rows per workgroup (128)
constexpr int kPaStages = 4;                    // LDS ring depth
constexpr int kPaWindow = 256;                  // block-table entries listed per pass
constexpr float kNegBigPf = -1.0e30f;

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
  int64_t T, num_blocks;
  int B, Hq, Hkv, group, max_blocks;
  float scale_log2;
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

// Append. Workgroup = (one block that request b's chunk writes, KV head g),
// mapped from a 1D grid (heads fastest); the block's slots [lo, hi) are new
// (positions P_b .. L_b - 1). Thread t handles slot t / (D/8), dims
// 8 (t % (D/8)) .. +8.
template <int D>
__global__ __launch_bounds__(256) void prefill_append_kernel(PrefillArgs a) {
  constexpr int C8 = D / 8;
  __shared__ uint16_t vt[D][kBlockSize + 2];  // V of the block, dim-major (+2: banks)
  const int g = blockIdx.x % a.Hkv;
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
  const int b = unit_from_end(a.B, static_cast<int>(blockIdx.x / a.Hkv), chunk_blocks, &jb);
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

template <int D>
__global__ __launch_bounds__(kPaThreads, 2) void prefill_attn_kernel(PrefillArgs a) {
  constexpr int QT = kPaQT, KC = D / 32, VT = D / 16;
  constexpr int TILE = kBlockSize * D;     // elements of a (block, head) tile
  constexpr int TILE_B = 2 * TILE;         // its bytes
  constexpr int DMA = TILE_B / 1024;       // 1 KB direct loads per tile
  constexpr int STAGE_B = 4 * TILE_B;      // K and V tiles of two blocks
  extern __shared__ __attribute__((aligned(16))) uint8_t ring[];  // [kPaStages][STAGE_B]
  __shared__ int list[kPaWindow];    // logical blocks j, ascending
  __shared__ int list_p[kPaWindow];  // their physical ids
  __shared__ int wave_cnt[kPaWaves];

  // (query tile, head h, request b) from a 1D grid, heads fastest: the last
  // requests' last tiles (a chunk's later rows see more keys, and requests
  // are commonly listed by growing prefix) are dispatched first, so that the
  // longest workgroups do not start behind short ones
  const int h = blockIdx.x % a.Hq;
  int qtile = 0;
  auto row_tiles = [&](int bb) {
    const int r0 = a.q_indptr[bb], r1 = a.q_indptr[bb + 1];
    const int n = r1 - r0;
    return rows_ok(r0, r1, a.T) && n > 0 ? (n + kPaRows - 1) / kPaRows : 0;
  };
  const int b = unit_from_end(a.B, static_cast<int>(blockIdx.x / a.Hq), row_tiles, &qtile);
  if (b < 0) return;
  const int r0 = a.q_indptr[b], r1 = a.q_indptr[b + 1];
  if (!rows_ok(r0, r1, a.T)) return;  // never given a unit
  const int n_b = r1 - r0;
  const int row0 = qtile * kPaRows;
  if (row0 >= n_b) return;
  const int tid = threadIdx.x;
  const int wave = __builtin_amdgcn_readfirstlane(tid / kWave), lane = tid % kWave;
  const int col = lane % 16, kgrp = lane / 16;
  const int L = a.ctx_lens[b];
  const int P = L - n_b;  // cached prefix
  const int g = h / a.group;
  const int rv = a.req_version[b];
  const int32_t* table = a.block_table + static_cast<int64_t>(b) * a.max_blocks;

  // Query columns of this wave: rows row0 + 32 wave + 16 ct + col.
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
  // the query is waited for here, before any direct load is issued (a wait
  // for it after them would wait for them too)
#pragma unroll
  for (int ct = 0; ct < QT; ++ct)
#pragma unroll
    for (int c = 0; c < KC; ++c) {
      asm volatile("" : "+v"(qraw[ct][c]));
      qv[ct][c] = as_bf16x8(qraw[ct][c]);
    }
  const int wave_last_row = min(row0 + (wave + 1) * 16 * QT, n_b) - 1;
  const int wave_limit = P + wave_last_row;  // largest key position this wave sees
  const int wave_first = P + row0 + wave * 16 * QT;  // position of its first row
  const int wg_limit = P + min(row0 + kPaRows, n_b) - 1;
  const int nb_lim = wg_limit < 0 ? 0 : min(wg_limit / kBlockSize + 1, a.max_blocks);

  f32x4 acc[QT][VT];
  float m_run[QT], l_run[QT];
#pragma unroll
  for (int ct = 0; ct < QT; ++ct) {
    m_run[ct] = kNegBigPf;
    l_run[ct] = 0.f;
#pragma unroll
    for (int t = 0; t < VT; ++t) acc[ct][t] = f32x4{0.f, 0.f, 0.f, 0.f};
  }

  // wave w moves tile w of a step: block w / 2 of the step, K (w even) or V
  const int my_blk = wave / 2, my_kind = wave % 2;
  const uint16_t* pool = my_kind ? a.v_cache : a.k_cache;

  for (int w0 = 0; w0 < nb_lim; w0 += kPaWindow) {
    // ---- list the non-stale blocks of this window, in ascending j
    const int j = w0 + tid;
    bool ok = false;
    int p = 0;
    if (j < nb_lim) {
      p = table[j];
      ok = id_ok(p, a.num_blocks) && a.block_version[p] == rv;
    }
    const uint64_t mask = __ballot(ok);
    const int before = __popcll(mask & ((1ull << lane) - 1ull));
    if (lane == 0) wave_cnt[wave] = __popcll(mask);
    __syncthreads();
    int off = 0, cnt = 0;
    for (int w = 0; w < kPaWaves; ++w) {
      if (w < wave) off += wave_cnt[w];
      cnt += wave_cnt[w];
    }
    if (ok) {
      list[off + before] = j;
      list_p[off + before] = p;
    }
    __syncthreads();
    if (cnt == 0) continue;
    const int steps = (cnt + 1) / 2;

    // loads of step s into ring stage `stage`: this wave's tile. Physical
    // ids come from LDS (a load of the block table here would make the wave
    // wait for every load before it). A step's second block past the list
    // end repeats its first (never used), and steps past the last repeat the
    // last into the free stage, so every step issues the same loads and the
    // wait counts hold.
    auto issue = [&](int stage, int s) {
      const int p = list_p[min(2 * s + my_blk, cnt - 1)];
      const uint8_t* src = reinterpret_cast<const uint8_t*>(
          pool + (static_cast<int64_t>(p) * a.Hkv + g) * TILE);
      uint8_t* dst = ring + stage * STAGE_B + wave * TILE_B;
#pragma unroll
      for (int q = 0; q < DMA; ++q) lds_load16(src + 1024 * q + 16 * lane, dst + 1024 * q);
    };
#pragma unroll
    for (int s = 0; s < kPaStages - 1; ++s) issue(s, min(s, steps - 1));

    for (int s = 0; s < steps; ++s) {
      // this wave's loads of step s are done (those of the two later steps
      // may still fly); after the barrier everyone's are, and the stage of
      // step s - 1 is free for step s + 3
      wait_vmcnt<DMA * (kPaStages - 2)>();
      wait_lgkm0_barrier();
      issue((s + kPaStages - 1) % kPaStages, min(s + kPaStages - 1, steps - 1));
      const int jA = list[2 * s];
      const bool hasB = 2 * s + 1 < cnt;
      const int jB = hasB ? list[2 * s + 1] : jA;
      if (jA * kBlockSize > wave_limit) continue;  // wholly past this wave's rows
      // every key of the step precedes every row of the wave (so it is also
      // before the context end): no masking
      const bool unmasked = hasB && jB * kBlockSize + kBlockSize - 1 <= wave_first;
      const uint8_t* st = ring + (s % kPaStages) * STAGE_B;
      const uint16_t* kA = reinterpret_cast<const uint16_t*>(st);
      const uint16_t* vA = reinterpret_cast<const uint16_t*>(st + TILE_B);
      const uint16_t* kB = reinterpret_cast<const uint16_t*>(st + 2 * TILE_B);
      const uint16_t* vB = reinterpret_cast<const uint16_t*>(st + 3 * TILE_B);
      bf16x8 kfa[KC], kfb[KC];
#pragma unroll
      for (int c = 0; c < KC; ++c) {
        kfa[c] = as_bf16x8(*reinterpret_cast<const u32x4*>(kA + c * 512 + lane * 8));
        kfb[c] = as_bf16x8(*reinterpret_cast<const u32x4*>(kB + c * 512 + lane * 8));
      }
      // V fragments: slots 4 kgrp .. +4 of each block; slots at or past the
      // context end are zeroed (they may hold anything)
      const int liveA = L - jA * kBlockSize - 4 * kgrp;
      const int liveB = hasB ? L - jB * kBlockSize - 4 * kgrp : 0;
      bf16x8 vf[VT];
#pragma unroll
      for (int t = 0; t < VT; ++t) {
        u32x2 va = *reinterpret_cast<const u32x2*>(vA + (16 * t + col) * kBlockSize + 4 * kgrp);
        u32x2 vb = *reinterpret_cast<const u32x2*>(vB + (16 * t + col) * kBlockSize + 4 * kgrp);
        if (liveA < 4) {
          va.x = liveA <= 0 ? 0u : (liveA == 1 ? va.x & 0xffffu : va.x);
          va.y = liveA <= 2 ? 0u : va.y & 0xffffu;
        }
        if (liveB < 4) {
          vb.x = liveB <= 0 ? 0u : (liveB == 1 ? vb.x & 0xffffu : vb.x);
          vb.y = liveB <= 2 ? 0u : vb.y & 0xffffu;
        }
        vf[t] = as_bf16x8(u32x4{va.x, va.y, vb.x, vb.y});
      }
      // S^T of both column tiles: 2 * QT independent chains of KC MFMAs,
      // interleaved so that no MFMA waits on the one before it
      f32x4 sA[QT], sB[QT];
#pragma unroll
      for (int ct = 0; ct < QT; ++ct) {
        sA[ct] = f32x4{0.f, 0.f, 0.f, 0.f};
        sB[ct] = f32x4{0.f, 0.f, 0.f, 0.f};
      }
#pragma unroll
      for (int c = 0; c < KC; ++c)
#pragma unroll
        for (int ct = 0; ct < QT; ++ct) {
          sA[ct] = mfma16x16x32(kfa[c], qv[ct][c], sA[ct]);
          sB[ct] = mfma16x16x32(kfb[c], qv[ct][c], sB[ct]);
        }
      // scaled (and, near the diagonal or the context end, masked) scores
      float sc[QT][8], m_new[QT];
#pragma unroll
      for (int ct = 0; ct < QT; ++ct) {
        if (unmasked) {
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            sc[ct][i] = sA[ct][i] * a.scale_log2;
            sc[ct][4 + i] = sB[ct][i] * a.scale_log2;
          }
        } else {
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const int posA = jA * kBlockSize + 4 * kgrp + i;
            const int posB = jB * kBlockSize + 4 * kgrp + i;
            sc[ct][i] = posA <= qpos[ct] ? sA[ct][i] * a.scale_log2 : -INFINITY;
            sc[ct][4 + i] = (hasB && posB <= qpos[ct]) ? sB[ct][i] * a.scale_log2 : -INFINITY;
          }
        }
        float mx = sc[ct][0];
#pragma unroll
        for (int i = 1; i < 8; ++i) mx = fmaxf(mx, sc[ct][i]);
        mx = max_xor32(max_xor16(mx));
        m_new[ct] = fmaxf(m_run[ct], mx);
      }
      // the running sums are rescaled only when some column's maximum grew
      // (elsewhere the factor is exactly 1)
      bool grew = false;
#pragma unroll
      for (int ct = 0; ct < QT; ++ct) grew = grew || m_new[ct] > m_run[ct];
      if (__ballot(grew) != 0ull) {
#pragma unroll
        for (int ct = 0; ct < QT; ++ct) {
          const float alpha = fast_exp2(m_run[ct] - m_new[ct]);
          l_run[ct] *= alpha;
#pragma unroll
          for (int t = 0; t < VT; ++t) acc[ct][t] *= alpha;
          m_run[ct] = m_new[ct];
        }
      }
      bf16x8 pb[QT];
#pragma unroll
      for (int ct = 0; ct < QT; ++ct) {
        float psum = 0.f;
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          const float pr = fast_exp2(sc[ct][i] - m_run[ct]);
          psum += pr;
          pb[ct][i] = static_cast<__bf16>(pr);
        }
        l_run[ct] += psum;
      }
#pragma unroll
      for (int t = 0; t < VT; ++t)
#pragma unroll
        for (int ct = 0; ct < QT; ++ct) acc[ct][t] = mfma16x16x32(vf[t], pb[ct], acc[ct][t]);
    }
    // every load has landed before the ring or the list is reused
    wait_vmcnt<0>();
    wait_lgkm0_barrier();
  }

  // ---- normalise and write this wave's rows
#pragma unroll
  for (int ct = 0; ct < QT; ++ct) {
    float l = l_run[ct];
    l += __shfl_xor(l, 16);
    l += __shfl_xor(l, 32);
    const int row = row0 + wave * 16 * QT + 16 * ct + col;
    if (row < n_b) {
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
        a.lse[orow] = l > 0.f ? (m_run[ct] + __log2f(l)) * kLn2 : -INFINITY;
    }
  }
}

template <int D>
local_status_t launch_prefill(const PrefillArgs& a, hipStream_t s) {
  if (a.k_new) {
    // a chunk of n rows spans at most n / 16 + 2 blocks: T / 16 + 2 B in all
    const int64_t units = a.T / kBlockSize + 2LL * a.B;
    prefill_append_kernel<D><<<static_cast<unsigned>(units * a.Hkv), 256, 0, s>>>(a);
    local_status_t st = local_check_launch("paged_attn_prefill (append)");
    if (st != LOCAL_OK) return st;
  }
  constexpr int kLds = kPaStages * 4 * 2 * kBlockSize * D;
  static bool done = false;
  if (!done) {  // benign race: every caller sets the same value
    (void)hipFuncSetAttribute(reinterpret_cast<const void*>(prefill_attn_kernel<D>),
                              hipFuncAttributeMaxDynamicSharedMemorySize, kLds);
    done = true;
  }
  // a chunk of n rows has at most n / 128 + 1 tiles: T / 128 + B in all
  const int64_t tiles = a.T / kPaRows + a.B;
  prefill_attn_kernel<D><<<static_cast<unsigned>(tiles * a.Hq), kPaThreads, kLds, s>>>(a);
  return local_check_launch("paged_attn_prefill");
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
  (void)ws;
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
  if (!ws) {
    *ws_bytes = 0;
    return LOCAL_OK;
  }
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
  a.scale_log2 = sm_scale * kLog2e;
  if ((T / kBlockSize + 2LL * B) * Hq >= (1LL << 31))
    return local_fail(LOCAL_ERR_UNSUPPORTED, "paged_attn_prefill: T=%lld too large", (long long)T);
  hipStream_t s = static_cast<hipStream_t>(stream);
  return D == 64 ? launch_prefill<64>(a, s) : launch_prefill<128>(a, s);
}
