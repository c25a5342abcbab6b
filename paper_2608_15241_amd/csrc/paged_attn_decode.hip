// local_paged_attn_decode: one new token per request attends over its paged
// KV cache; blocks whose adapter-version tag differs from the request's
// version are excluded (§5.1 validity key; §1 challenge (2)).
//
// Design (HBM-bound: every valid KV byte is read once, stale blocks are never
// read):
//  * Split-KV. A workgroup is one wave and owns a partition of 32 logical
//    blocks (512 tokens) of one request and one KV head. Partitions are
//    counted from the end of the context and their index is the slowest grid
//    dimension, so full partitions are dispatched first and each request's
//    partial one (its oldest blocks) last, which shortens the tail when
//    context lengths vary. A wave reads its 32 table entries and tags first,
//    keeps the non-stale blocks and walks them
//    in order through a ring of DEPTH register sets, so that DEPTH-1 blocks'
//    K/V loads are in flight while one block is computed. Block loads are
//    buffer loads issued unconditionally (a block past the end gets a
//    zero-size descriptor: zeros, no traffic) and the new token is merged in
//    with selects, so the loop has no data-dependent branch and each block
//    waits only for its own loads.
//  * Matrix cores, transposed. Per block, S^T[16 keys x 16 cols] =
//    K[16 x D] * Q^T[D x 16] on v_mfma_f32_16x16x32_bf16, where the columns
//    are the Hq/Hkv query heads that share KV head g (zero-padded to 16).
//    The K layout [D/8][16][8] makes each lane's 16-byte A-operand slice
//    contiguous and each MFMA's 64 loads one contiguous kilobyte. The score
//    tile's accumulator layout (lane: 4 keys of one column) is exactly the
//    B-operand layout of the next product O^T[D x 16] += V^T[D x 16] P^T on
//    v_mfma_f32_16x16x16_bf16, whose A operand comes straight from the V
//    layout [D][16] (each lane: 4 keys of one dim, 8 bytes).
//  * Online softmax in the log2 domain per column. A request that fits one
//    partition is finished in place; otherwise each partition leaves its
//    (max, sum, unnormalised O) and a second kernel merges them.
//  * The new token's K/V are written at position L-1 by the wave that owns
//    that block, which also substitutes them for the cache slot it reads, so
//    no other workgroup and no second launch is involved.
#include <mutex>

#include "common.hpp"

namespace localk {
namespace {

// Blocks per partition (one wave each), by the width of the block table:
// 32 up to 256 blocks, 48 up to 512, 64 beyond (at most 64: one bit per lane
// in the stale masks). Measured: the 32-layer decode with contexts up to 16K
// tokens (1024-block tables) is 3.2% faster a step with 64 than with 32, the
// GQA decode with 512-block tables 2% faster with 48, and the MHA decode with
// 256-block tables fastest with 32 (fewer, longer partitions: less merge
// traffic and fewer waves; shorter ones: more parallelism per request).
int part_blocks(int max_blocks) { return max_blocks <= 256 ? 32 : max_blocks <= 512 ? 48 : 64; }
constexpr float kNegBig = -1.0e30f;

struct DecodeArgs {
  const uint16_t* q;
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
  float* part_o;   // [B][Hq][n_parts][D]
  float* part_ml;  // [B][Hq][n_parts][2]  (max in log2 units, sum)
  // The version check of the same call (null when not asked for): per
  // (request, partition), the stale blocks as a bit mask (bit i = block
  // j0 + i) and the live tokens of the valid ones, written by KV head 0's
  // waves; the merge launch turns them into the canonical outputs.
  uint64_t* vc_mask;    // [B][n_parts]
  int32_t* vc_valid;    // [B][n_parts]
  int32_t* vc_pairs;    // [cap][2] (b, j), or null when cap == 0
  int64_t vc_cap;
  int32_t* vc_n_stale;  // one int32
  int32_t* vc_valid_tokens;  // [B]
  int64_t num_blocks;
  int Hq, Hkv, group, max_blocks, n_parts;
  int pb;            // blocks per partition (part_blocks of max_blocks)
  float scale_log2;  // sm_scale * log2(e)
};

// Logical blocks request b owns: ceil(L/16), at most the table's width.
__device__ __forceinline__ int owned_blocks(int L, int max_blocks) {
  return L <= 0 ? 0 : min((L + kBlockSize - 1) / kBlockSize, max_blocks);
}

// Position of the k-th (0-based) set bit of m (k < popcount(m)).
__device__ __forceinline__ int nth_set_bit(uint64_t m, int k) {
  for (int i = 0; i < k; ++i) m &= m - 1ull;
  return __ffsll(static_cast<long long>(m)) - 1;
}

// Requests a wavefront ranks at once: 64 per register, up to this many
// registers (larger batches use the grid order below without ranking).
constexpr int kRankChunks = 8;

// The unit of work of dispatch slot k, longest first: every full partition,
// row by row (partition z of each request that has it, ascending b), then
// each request's partial partition, longest first (ties: smaller b); an
// empty context is a partial partition of no block. Returns the request (-1
// past the last unit) and, in *part, its partition index (a partial one is
// numbered n_full, as in the merge). Every lane returns the same.
__device__ int decode_unit(const DecodeArgs& a, int B, int k, int* part) {
  const int lane = threadIdx.x % kWave;
  const int nc = (B + kWave - 1) / kWave;
  int nf[kRankChunks], rem[kRankChunks];
  bool has_partial[kRankChunks];
#pragma unroll
  for (int c = 0; c < kRankChunks; ++c) {
    const int b = c * kWave + lane;
    const int nb = b < B ? owned_blocks(a.ctx_lens[b], a.max_blocks) : -1;
    nf[c] = nb > 0 ? nb / a.pb : 0;
    rem[c] = nb > 0 ? nb % a.pb : 0;
    has_partial[c] = nb == 0 || rem[c] > 0;  // nb = -1: no request
  }
  // slots past the last unit leave before any ranking
  int units = 0;
#pragma unroll
  for (int c = 0; c < kRankChunks; ++c) units += nf[c] + (has_partial[c] ? 1 : 0);
#pragma unroll
  for (int off = kWave / 2; off > 0; off >>= 1) units += __shfl_xor(units, off);
  if (k >= units) return -1;
  for (int z = 0; z < a.n_parts; ++z) {
    int cnt = 0;
#pragma unroll
    for (int c = 0; c < kRankChunks; ++c) {
      if (c >= nc) break;
      cnt += __popcll(__ballot(nf[c] > z));
    }
    if (cnt == 0) break;
    if (k < cnt) {
#pragma unroll
      for (int c = 0; c < kRankChunks; ++c) {
        if (c >= nc) break;
        const uint64_t m = __ballot(nf[c] > z);
        const int n = __popcll(m);
        if (k < n) {
          *part = z;
          return c * kWave + nth_set_bit(m, k);
        }
        k -= n;
      }
    }
    k -= cnt;
  }
  for (int v = a.pb - 1; v >= 0; --v) {
#pragma unroll
    for (int c = 0; c < kRankChunks; ++c) {
      if (c >= nc) break;
      const uint64_t m = __ballot(has_partial[c] && rem[c] == v);
      const int n = __popcll(m);
      if (k < n) {
        const int l = nth_set_bit(m, k);
        *part = __shfl(nf[c], l);
        return c * kWave + l;
      }
      k -= n;
    }
  }
  return -1;
}

// The 4 V values a lane holds for one block (slots slot0..slot0+3), with
// slots past s_live set to 0 (their cache contents are undefined and must not
// reach the product) and slot s_new replaced by vnew. For a block that is
// neither the last nor the appended one, s_live = 15 and s_new = -1 leave it
// unchanged; everything is a select.
__device__ __forceinline__ u32x2 fix_v(u32x2 v, int slot0, int s_live, int s_new,
                                       uint32_t vnew) {
  uint32_t h[4] = {v.x & 0xffffu, v.x >> 16, v.y & 0xffffu, v.y >> 16};
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const int slot = slot0 + e;
    h[e] = slot > s_live ? 0u : (slot == s_new ? vnew : h[e]);
  }
  u32x2 r;
  r.x = h[0] | (h[1] << 16);
  r.y = h[2] | (h[3] << 16);
  return r;
}

#ifndef LOCAL_DECODE_APPEND_NT
#define LOCAL_DECODE_APPEND_NT 1  // non-temporal stores: measured 9 us faster on the 7B batch
#endif
// Store of a piece of the appended token.
template <typename T>
__device__ __forceinline__ void st_append(uint16_t* p, T v) {
#if LOCAL_DECODE_APPEND_NT
  __builtin_nontemporal_store(v, reinterpret_cast<T*>(p));
#else
  *reinterpret_cast<T*>(p) = v;
#endif
}

// K/V registers of one block.
template <int D>
struct BlockRegs {
  u32x4 k[D / 32];
  u32x2 v[D / 16];
};

template <int D, int DEPTH, bool RANKED>
__global__ __launch_bounds__(kWave) void decode_attn_kernel(DecodeArgs a, int B) {
  constexpr int KC = D / 32;  // 32-dim chunks of the QK product
  constexpr int VT = D / 16;  // 16-dim tiles of the PV product

  const int lane = threadIdx.x;
  const int col = lane % 16, kgrp = lane / 16;
  // Partition p covers blocks [nb - P(p+1), nb - Pp) of b (P = a.pb): the full ones
  // counted from the end of the context, then at most one partial one at the
  // start. An empty context runs partition 0 with no block (zero output,
  // lse = -inf). The grid is 1D, KV heads fastest, sized for n_parts + 1
  // partitions of every request; the slots map to units longest first (full
  // partitions, then the partial ones by decreasing length), so the last
  // waves to start are the shortest and the idle slots come last. Batches
  // wider than the ranking takes dispatch each partition row in request
  // order instead, the partial partitions last.
  const int g = blockIdx.x % a.Hkv;
  const int slot = blockIdx.x / a.Hkv;
  int b, part;
  if (RANKED) {
    b = decode_unit(a, B, slot, &part);
    if (b < 0) return;
  } else {
    b = slot % B;
    part = slot / B;
  }
  const int L = a.ctx_lens[b];
  const int nb = owned_blocks(L, a.max_blocks);
  const int n_full = nb / a.pb, rem = nb % a.pb;
  if (!RANKED) {
    if (part < a.n_parts) {
      if (part >= n_full && !(nb == 0 && part == 0)) return;
    } else {
      if (rem == 0) return;
      part = n_full;
    }
  }
  const int j_end_part = nb - part * a.pb;
  const int j0 = max(0, j_end_part - a.pb);
  const int n_parts_b = max(1, (nb + a.pb - 1) / a.pb);
  const int rv = a.req_version[b];
  const int32_t* table = a.block_table + static_cast<int64_t>(b) * a.max_blocks;
  const int G = a.group;

  // This partition's blocks: table entries and tags, keep the non-stale ones.
  const int jend = j_end_part;
  int my_phys = 0;
  bool ok = false;
  if (lane < a.pb && j0 + lane < jend) {
    my_phys = table[j0 + lane];
    ok = my_phys >= 0 && my_phys < a.num_blocks && a.block_version[my_phys] == rv;
    if (!ok) my_phys = 0;  // an id outside the pool is never dereferenced
  }
  uint64_t valid_mask = __ballot(ok);
  if (a.vc_mask && g == 0) {  // the version check of this partition's blocks
    const bool owned = lane < a.pb && j0 + lane < jend;
    const uint64_t stale = __ballot(owned && !ok);
    int live = ok ? min(kBlockSize, L - kBlockSize * (j0 + lane)) : 0;
#pragma unroll
    for (int off = kWave / 2; off > 0; off >>= 1) live += __shfl_xor(live, off);
    if (lane == 0) {
      const int64_t slot = static_cast<int64_t>(b) * a.n_parts + part;
      a.vc_mask[slot] = stale;
      a.vc_valid[slot] = live;
    }
  }

  // Query heads of this KV head, as the B operand (column = head).
  bf16x8 qv[KC];
  {
    const int h = g * G + col;
#pragma unroll
    for (int c = 0; c < KC; ++c) {
      u32x4 v = {0u, 0u, 0u, 0u};
      if (col < G)
        v = ld_global<u32x4>(a.q + (static_cast<int64_t>(b) * a.Hq + h) * D + 32 * c +
                             8 * kgrp);
      qv[c] = as_bf16x8(v);
    }
  }

  // The new token (position L-1), if its block is in this partition: its K/V
  // rows are substituted for the slot while the block is read, and written to
  // the pool after the last block (an id outside the pool is not written).
  const int j_new = (L - 1) / kBlockSize, s_last = (L - 1) % kBlockSize;
  const bool has_new = a.k_new != nullptr;
  const int64_t kvrow = (static_cast<int64_t>(b) * a.Hkv + g) * D;
  const bool append = has_new && j_new >= j0 && j_new < jend;
  const int p_new = append ? table[j_new] : -1;

  f32x4 acc[VT];
#pragma unroll
  for (int t = 0; t < VT; ++t) acc[t] = f32x4{0.f, 0.f, 0.f, 0.f};
  float m_run = kNegBig, l_run = 0.f;

  // the new token's K/V fragments, for the lanes that hold its slot
  u32x4 kn[KC];
  uint32_t vn[VT];
#pragma unroll
  for (int c = 0; c < KC; ++c) kn[c] = u32x4{0u, 0u, 0u, 0u};
#pragma unroll
  for (int t = 0; t < VT; ++t) vn[t] = 0u;
  if (has_new && j_new >= j0 && j_new < jend) {
#pragma unroll
    for (int c = 0; c < KC; ++c) kn[c] = ld_global<u32x4>(a.k_new + kvrow + 32 * c + 8 * kgrp);
#pragma unroll
    for (int t = 0; t < VT; ++t) vn[t] = a.v_new[kvrow + 16 * t + col];
  }

  // next valid block (partition-relative index), -1 when none is left
  auto next_block = [&]() -> int {
    if (!valid_mask) return -1;
    const int i = __builtin_ctzll(valid_mask);
    valid_mask &= valid_mask - 1;
    return i;
  };
  constexpr uint32_t kTileBytes = kBlockSize * D * 2;
  auto load_block = [&](BlockRegs<D>& R, int i) {
    const bool live = i >= 0;
    // the block id is the same in every lane: keep it (and the descriptors)
    // in scalar registers
    const int p = live ? __builtin_amdgcn_readlane(my_phys, i) : 0;
    const int64_t tile = (static_cast<int64_t>(p) * a.Hkv + g) * (kBlockSize * D);
    const __amdgpu_buffer_rsrc_t rk = make_rsrc(a.k_cache + tile, live ? kTileBytes : 0u);
    const __amdgpu_buffer_rsrc_t rv2 = make_rsrc(a.v_cache + tile, live ? kTileBytes : 0u);
#pragma unroll
    for (int c = 0; c < KC; ++c) R.k[c] = buf_load16_stream(rk, (c * 512 + lane * 8) * 2);
#pragma unroll
    for (int t = 0; t < VT; ++t)
      R.v[t] = buf_load8_stream(rv2, ((16 * t + col) * kBlockSize + 4 * kgrp) * 2);
  };
  auto compute_block = [&](BlockRegs<D>& R, int i) {
    const int j = j0 + i;
    const bool last = j == j_new;
    const int s_live = last ? s_last : kBlockSize - 1;
    const int s_new = (last && has_new) ? s_last : -1;
#pragma unroll
    for (int c = 0; c < KC; ++c) R.k[c] = col == s_new ? kn[c] : R.k[c];
#pragma unroll
    for (int t = 0; t < VT; ++t) R.v[t] = fix_v(R.v[t], 4 * kgrp, s_live, s_new, vn[t]);
    f32x4 sc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int c = 0; c < KC; ++c) sc = mfma16x16x32(as_bf16x8(R.k[c]), qv[c], sc);
    float s[4];
#pragma unroll
    for (int e = 0; e < 4; ++e)
      s[e] = j * kBlockSize + 4 * kgrp + e < L ? sc[e] * a.scale_log2 : -INFINITY;
    float mx = fmaxf(fmaxf(s[0], s[1]), fmaxf(s[2], s[3]));
    mx = max_xor32(max_xor16(mx));
    const float m_new = fmaxf(m_run, mx);
    const float alpha = fast_exp2(m_run - m_new);
    bf16x4 pb;
    float psum = 0.f;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const float p = fast_exp2(s[e] - m_new);
      psum += p;
      pb[e] = static_cast<__bf16>(p);
    }
    l_run = l_run * alpha + psum;
    m_run = m_new;
#pragma unroll
    for (int t = 0; t < VT; ++t) {
      acc[t] *= alpha;
      acc[t] = mfma16x16x16(as_bf16x4(R.v[t]), pb, acc[t]);
    }
  };

  // ring of DEPTH register sets: DEPTH-1 blocks load while one computes
  BlockRegs<D> R[DEPTH];
  int idx[DEPTH];
#pragma unroll
  for (int d = 0; d < DEPTH - 1; ++d) {
    idx[d] = next_block();
    load_block(R[d], idx[d]);
  }

  bool done = false;
  while (!done) {
#pragma unroll
    for (int d = 0; d < DEPTH; ++d) {
      const int fill = (d + DEPTH - 1) % DEPTH;
      idx[fill] = next_block();
      load_block(R[fill], idx[fill]);
      if (idx[d] < 0) {
        done = true;
        break;
      }
      compute_block(R[d], idx[d]);
    }
  }

  // ---- append: the new token's K/V rows from the registers that hold them
  // (K: k-group c8 = 4c + kgrp of the row in the 4 lanes of column 0; V: dim
  // 16t + col in the lanes of k-group 0), after every read of the block.
  // Written here rather than before the loop, a store ahead of the block
  // loads would hold them back (measured: 5 us per launch on the 7B batch).
  if (append && p_new >= 0 && p_new < a.num_blocks) {
    const int64_t tile = (static_cast<int64_t>(p_new) * a.Hkv + g) * (kBlockSize * D);
    if (col == 0) {
#pragma unroll
      for (int c = 0; c < KC; ++c)
        st_append<u32x4>(a.k_cache + tile + (4 * c + kgrp) * (kBlockSize * 8) + s_last * 8,
                         kn[c]);
    }
    if (kgrp == 0) {
#pragma unroll
      for (int t = 0; t < VT; ++t)
        st_append<uint16_t>(a.v_cache + tile + (16 * t + col) * kBlockSize + s_last,
                            static_cast<uint16_t>(vn[t]));
    }
  }

  // ---- finish: the column's sum over the 4 lane groups, then write
  l_run += __shfl_xor(l_run, 16);
  l_run += __shfl_xor(l_run, 32);
  if (col < G) {
    const int h = g * G + col;
    const int64_t bh = static_cast<int64_t>(b) * a.Hq + h;
    if (n_parts_b == 1) {
      const float inv = l_run > 0.f ? 1.f / l_run : 0.f;
#pragma unroll
      for (int t = 0; t < VT; ++t)
        *reinterpret_cast<u32x2*>(a.out + bh * D + 16 * t + 4 * kgrp) =
            u32x2{pack_bf16x2(acc[t][0] * inv, acc[t][1] * inv),
                  pack_bf16x2(acc[t][2] * inv, acc[t][3] * inv)};
      if (kgrp == 0 && a.lse)
        a.lse[bh] = l_run > 0.f ? (m_run + __log2f(l_run)) * kLn2 : -INFINITY;
    } else {
      const int64_t pi = bh * a.n_parts + part;
#pragma unroll
      for (int t = 0; t < VT; ++t)
        *reinterpret_cast<f32x4*>(a.part_o + pi * D + 16 * t + 4 * kgrp) = acc[t];
      if (kgrp == 0) {
        a.part_ml[pi * 2] = m_run;
        a.part_ml[pi * 2 + 1] = l_run;
      }
    }
  }
}

// Merge the partitions of every (request, head) that has more than one.
// The version check from the partitions' stale masks (one workgroup per
// request, D threads): the request's offset in the canonical list is the
// number of stale blocks of the requests before it; its own stale blocks
// follow in ascending j (partitions in descending index). Deterministic, no
// atomics.
__device__ void decode_version_check(const DecodeArgs& a, int b, int B, int* sh) {
  const int tid = threadIdx.x, nt = blockDim.x;
  auto parts_of = [&](int bb) {
    const int nbb = owned_blocks(a.ctx_lens[bb], a.max_blocks);
    return max(1, (nbb + a.pb - 1) / a.pb);
  };
  int before = 0;
  for (int e = tid; e < b * a.n_parts; e += nt) {
    const int bb = e / a.n_parts, pp = e % a.n_parts;
    if (pp < parts_of(bb)) before += __popcll(a.vc_mask[e]);
  }
  const int np = parts_of(b);
  // this request's partitions in ascending j: t-th is partition np - 1 - t
  int cnt = 0, valid = 0;
  uint64_t mask = 0ull;
  if (tid < np) {
    const int64_t slot = static_cast<int64_t>(b) * a.n_parts + (np - 1 - tid);
    mask = a.vc_mask[slot];
    cnt = __popcll(mask);
    valid = a.vc_valid[slot];
  }
  // block-wide sums of `before` and `valid`, exclusive prefix of `cnt` over t
  sh[tid] = cnt;
  __syncthreads();
  int pre = 0;
  for (int t = 0; t < tid && t < np; ++t) pre += sh[t];
  __syncthreads();
  sh[tid] = before;
  __syncthreads();
  for (int w = nt / 2; w > 0; w >>= 1) {
    if (tid < w) sh[tid] += sh[tid + w];
    __syncthreads();
  }
  const int offset = sh[0];
  __syncthreads();
  sh[tid] = valid;
  __syncthreads();
  for (int w = nt / 2; w > 0; w >>= 1) {
    if (tid < w) sh[tid] += sh[tid + w];
    __syncthreads();
  }
  if (tid == 0) a.vc_valid_tokens[b] = sh[0];
  if (tid < np) {  // (np <= n_parts <= nt: the host checks)
    const int nbb = owned_blocks(a.ctx_lens[b], a.max_blocks);
    const int p = np - 1 - tid;
    const int j0 = max(0, nbb - a.pb * (p + 1));
    int64_t pos = static_cast<int64_t>(offset) + pre;
    for (uint64_t m = mask; m; m &= m - 1ull, ++pos) {
      if (pos < a.vc_cap) {
        a.vc_pairs[2 * pos] = b;
        a.vc_pairs[2 * pos + 1] = j0 + __ffsll(static_cast<long long>(m)) - 1;
      }
    }
    if (b == B - 1 && tid == np - 1) *a.vc_n_stale = offset + pre + cnt;
  }
}

template <int D>
__global__ __launch_bounds__(D) void decode_merge_kernel(DecodeArgs a, int B) {
  const int bh = blockIdx.x;
  const int b = bh / a.Hq;
  const int d = threadIdx.x;
  if (a.vc_mask && bh % a.Hq == 0) {
    __shared__ int sh[D];
    decode_version_check(a, b, B, sh);
  }
  const int L = a.ctx_lens[b];
  const int nb = owned_blocks(L, a.max_blocks);
  const int np = max(1, (nb + a.pb - 1) / a.pb);
  if (np == 1) return;  // written by the main kernel
  // one pass over the partitions, 8 at a time with all their loads in flight;
  // the running sums are rescaled when a batch raises the maximum
  constexpr int kMergeBatch = 8;
  const float* ml = a.part_ml + static_cast<int64_t>(bh) * a.n_parts * 2;
  const float* po = a.part_o + static_cast<int64_t>(bh) * a.n_parts * D;
  float M = kNegBig, den = 0.f, num = 0.f;
  for (int p0 = 0; p0 < np; p0 += kMergeBatch) {
    float2 mlv[kMergeBatch];
    float ov[kMergeBatch];
#pragma unroll
    for (int q = 0; q < kMergeBatch; ++q) {
      const bool in = p0 + q < np;
      mlv[q] = in ? *reinterpret_cast<const float2*>(ml + 2 * (p0 + q)) : float2{kNegBig, 0.f};
      ov[q] = in ? po[static_cast<int64_t>(p0 + q) * D + d] : 0.f;
    }
    float Mb = M;
#pragma unroll
    for (int q = 0; q < kMergeBatch; ++q) Mb = fmaxf(Mb, mlv[q].x);
    const float c = fast_exp2(M - Mb);
    den *= c;
    num *= c;
#pragma unroll
    for (int q = 0; q < kMergeBatch; ++q) {
      const float f = fast_exp2(mlv[q].x - Mb);
      den += mlv[q].y * f;
      num += ov[q] * f;
    }
    M = Mb;
  }
  a.out[static_cast<int64_t>(bh) * D + d] = f32_to_bf16(den > 0.f ? num / den : 0.f);
  if (d == 0 && a.lse) a.lse[bh] = den > 0.f ? (M + __log2f(den)) * kLn2 : -INFINITY;
}

// Blocks in flight per wave: 4 with one query head per KV head, 3 with
// grouped heads (measured: 4 is 1.7% faster on the MHA decode step and 1.2%
// slower on the GQA one, whose waves do four heads' softmax per block).
#ifndef LOCAL_DECODE_DEPTH_MHA
#define LOCAL_DECODE_DEPTH_MHA 4
#endif
#ifndef LOCAL_DECODE_DEPTH
#define LOCAL_DECODE_DEPTH 3
#endif

template <int D>
local_status_t launch_decode(const DecodeArgs& a, int B, hipStream_t s) {
  const int64_t wgs = static_cast<int64_t>(a.Hkv) * B * (a.n_parts + 1);
  if (wgs >= (1LL << 31))
    return local_fail(LOCAL_ERR_UNSUPPORTED, "paged_attn_decode: grid of %lld workgroups",
                      (long long)wgs);
  const unsigned grid = static_cast<unsigned>(wgs);
  const bool ranked = B <= kRankChunks * kWave;
  if (a.group == 1) {
    if (ranked)
      decode_attn_kernel<D, LOCAL_DECODE_DEPTH_MHA, true><<<grid, kWave, 0, s>>>(a, B);
    else
      decode_attn_kernel<D, LOCAL_DECODE_DEPTH_MHA, false><<<grid, kWave, 0, s>>>(a, B);
  } else {
    if (ranked)
      decode_attn_kernel<D, LOCAL_DECODE_DEPTH, true><<<grid, kWave, 0, s>>>(a, B);
    else
      decode_attn_kernel<D, LOCAL_DECODE_DEPTH, false><<<grid, kWave, 0, s>>>(a, B);
  }
  if (a.n_parts > 1 || a.vc_mask) decode_merge_kernel<D><<<B * a.Hq, D, 0, s>>>(a, B);
  return local_check_launch("paged_attn_decode");
}

}  // namespace
}  // namespace localk

using namespace localk;

// Host-side validation shared by both entry points: fills *a (without the
// partials' pointers) and *need, the bytes of split-KV partials of the call.
static local_status_t decode_setup(const uint16_t* q, int32_t B, int32_t Hq, int32_t Hkv,
                                   int32_t D, const uint16_t* k_new, const uint16_t* v_new,
                                   uint16_t* k_cache, uint16_t* v_cache, int64_t num_blocks,
                                   int32_t block_size, const int32_t* block_table,
                                   int32_t max_blocks, const int32_t* ctx_lens,
                                   const int32_t* block_version, const int32_t* req_version,
                                   float sm_scale, uint16_t* out, float* lse, const char* who,
                                   DecodeArgs* a, size_t* part_elems, size_t* need) {
  if (B < 0 || Hq <= 0 || Hkv <= 0 || max_blocks < 1 || num_blocks < 1 || Hq % Hkv != 0)
    return local_fail(LOCAL_ERR_SHAPE, "%s: B=%d Hq=%d Hkv=%d max_blocks=%d num_blocks=%lld",
                      who, B, Hq, Hkv, max_blocks, (long long)num_blocks);
  if (block_size != kBlockSize || (D != 64 && D != 128) || Hq / Hkv > 16)
    return local_fail(LOCAL_ERR_UNSUPPORTED,
                      "%s: block_size=%d D=%d group=%d (need 16, 64|128, <=16)", who,
                      block_size, D, Hq / Hkv);
  if ((k_new == nullptr) != (v_new == nullptr))
    return local_fail(LOCAL_ERR_NULL, "%s: k_new and v_new must both be set", who);
  const int pb = part_blocks(max_blocks);
  const int n_parts = (max_blocks + pb - 1) / pb;
  *part_elems = static_cast<size_t>(B > 0 ? B : 1) * Hq * n_parts;
  *need = *part_elems * (D + 2) * sizeof(float);
  a->q = q;
  a->k_new = k_new;
  a->v_new = v_new;
  a->k_cache = k_cache;
  a->v_cache = v_cache;
  a->block_table = block_table;
  a->ctx_lens = ctx_lens;
  a->block_version = block_version;
  a->req_version = req_version;
  a->out = out;
  a->lse = lse;
  a->part_o = nullptr;
  a->part_ml = nullptr;
  a->vc_mask = nullptr;
  a->vc_valid = nullptr;
  a->vc_pairs = nullptr;
  a->vc_cap = 0;
  a->vc_n_stale = nullptr;
  a->vc_valid_tokens = nullptr;
  a->Hq = Hq;
  a->Hkv = Hkv;
  a->group = Hq / Hkv;
  a->num_blocks = num_blocks;
  a->max_blocks = max_blocks;
  a->n_parts = n_parts;
  a->pb = pb;
  a->scale_log2 = sm_scale * kLog2e;
  return LOCAL_OK;
}

static local_status_t decode_pointers_ok(const DecodeArgs& a, const char* who) {
  if (!a.q || !a.k_cache || !a.v_cache || !a.block_table || !a.ctx_lens ||
      !a.block_version || !a.req_version || !a.out)
    return local_fail(LOCAL_ERR_NULL, "%s: NULL pointer argument", who);
  return LOCAL_OK;
}

static local_status_t decode_launch(DecodeArgs& a, int B, int D, void* partials,
                                    size_t part_elems, void* stream) {
  a.part_o = static_cast<float*>(partials);
  a.part_ml = a.part_o + part_elems * D;
  hipStream_t s = static_cast<hipStream_t>(stream);
  return D == 64 ? launch_decode<64>(a, B, s) : launch_decode<128>(a, B, s);
}

extern "C" local_status_t local_paged_attn_decode(
    const uint16_t* q, int32_t B, int32_t Hq, int32_t Hkv, int32_t D,
    const uint16_t* k_new, const uint16_t* v_new, uint16_t* k_cache, uint16_t* v_cache,
    int64_t num_blocks, int32_t block_size, const int32_t* block_table,
    int32_t max_blocks, const int32_t* ctx_lens, const int32_t* block_version,
    const int32_t* req_version, float sm_scale, uint16_t* out, float* lse, void* ws,
    size_t* ws_bytes, void* stream) {
  const char* who = "paged_attn_decode";
  if (!ws_bytes) return local_fail(LOCAL_ERR_WORKSPACE, "%s: ws_bytes is NULL", who);
  DecodeArgs a;
  size_t part_elems = 0, need = 0;
  local_status_t st = decode_setup(q, B, Hq, Hkv, D, k_new, v_new, k_cache, v_cache,
                                   num_blocks, block_size, block_table, max_blocks, ctx_lens,
                                   block_version, req_version, sm_scale, out, lse, who, &a,
                                   &part_elems, &need);
  if (st != LOCAL_OK) return st;
  if (!ws) {
    *ws_bytes = need;
    return LOCAL_OK;
  }
  if (*ws_bytes < need)
    return local_fail(LOCAL_ERR_WORKSPACE, "%s: workspace %zu < %zu", who, *ws_bytes, need);
  if (B == 0) return LOCAL_OK;
  if ((st = decode_pointers_ok(a, who)) != LOCAL_OK) return st;
  return decode_launch(a, B, D, ws, part_elems, stream);
}

// ---------------------------------------------------------------- checked
namespace {
__global__ void decode_vc_empty_kernel(int32_t* n_stale) { *n_stale = 0; }
size_t align256(size_t v) { return (v + 255) & ~static_cast<size_t>(255); }
}  // namespace

extern "C" local_status_t local_paged_attn_decode_checked(
    const uint16_t* q, int32_t B, int32_t Hq, int32_t Hkv, int32_t D,
    const uint16_t* k_new, const uint16_t* v_new, uint16_t* k_cache, uint16_t* v_cache,
    int64_t num_blocks, int32_t block_size, const int32_t* block_table,
    int32_t max_blocks, const int32_t* ctx_lens, const int32_t* block_version,
    const int32_t* req_version, float sm_scale, uint16_t* out, float* lse,
    int32_t* stale_pairs, int64_t cap, int32_t* n_stale, int32_t* valid_tokens, void* ws,
    size_t* ws_bytes, void* stream) {
  const char* who = "paged_attn_decode_checked";
  if (!ws_bytes) return local_fail(LOCAL_ERR_WORKSPACE, "%s: ws_bytes is NULL", who);
  DecodeArgs a;
  size_t part_elems = 0, need = 0;
  local_status_t st = decode_setup(q, B, Hq, Hkv, D, k_new, v_new, k_cache, v_cache,
                                   num_blocks, block_size, block_table, max_blocks, ctx_lens,
                                   block_version, req_version, sm_scale, out, lse, who, &a,
                                   &part_elems, &need);
  if (st != LOCAL_OK) return st;
  if (cap < 0) return local_fail(LOCAL_ERR_SHAPE, "%s: cap=%lld", who, (long long)cap);
  if (a.n_parts > D)
    return local_fail(LOCAL_ERR_UNSUPPORTED, "%s: max_blocks=%d over %d blocks", who,
                      max_blocks, D * a.pb);
  const size_t masks = static_cast<size_t>(B > 0 ? B : 1) * a.n_parts;
  const size_t total =
      align256(need) + align256(masks * sizeof(uint64_t)) + align256(masks * sizeof(int32_t));
  if (!ws) {
    *ws_bytes = total;
    return LOCAL_OK;
  }
  if (*ws_bytes < total)
    return local_fail(LOCAL_ERR_WORKSPACE, "%s: workspace %zu < %zu", who, *ws_bytes, total);
  if (!n_stale || (B > 0 && !valid_tokens) || (cap > 0 && !stale_pairs))
    return local_fail(LOCAL_ERR_NULL, "%s: NULL version-check output", who);
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (B == 0) {
    decode_vc_empty_kernel<<<1, 1, 0, s>>>(n_stale);
    return local_check_launch(who);
  }
  if ((st = decode_pointers_ok(a, who)) != LOCAL_OK) return st;
  char* base = static_cast<char*>(ws);
  a.vc_mask = reinterpret_cast<uint64_t*>(base + align256(need));
  a.vc_valid = reinterpret_cast<int32_t*>(base + align256(need) + align256(masks * 8));
  a.vc_pairs = stale_pairs;
  a.vc_cap = cap;
  a.vc_n_stale = n_stale;
  a.vc_valid_tokens = valid_tokens;
  return decode_launch(a, B, D, ws, part_elems, stream);
}

// ---------------------------------------------------------------- no-alloc
// Scratch of local_paged_attn_decode_noalloc: the split-KV partials of up to
// 131072 (request, query head, partition) triples at D = 128, held
// by the library in device memory (one copy per GPU, for the life of the
// process). In host code `scratch` names a host-side stand-in, not the device
// copy: its device address is taken once per device with
// hipGetSymbolAddress and only that address is ever passed to a kernel.
constexpr size_t kNoAllocBytes = LOCAL_DECODE_NOALLOC_SCRATCH_BYTES;
static_assert(kNoAllocBytes == 131072 * (128 + 2) * sizeof(float), "partials at D = 128");
__device__ __align__(256) float scratch[kNoAllocBytes / sizeof(float)];

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

// The device address of `scratch` on the current device (taken on its first
// use there, with that device current). NULL with *st set on failure.
void* scratch_of_current_device(local_status_t* st) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess || dev < 0 || dev >= kMaxDevices) {
    *st = local_fail(LOCAL_ERR_HIP, "paged_attn_decode_noalloc: hipGetDevice: %s (device %d)",
                     hipGetErrorString(e), dev);
    return nullptr;
  }
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p) {
      *st = local_fail(LOCAL_ERR_HIP, "paged_attn_decode_noalloc: hipGetSymbolAddress: %s",
                       hipGetErrorString(e));
      return nullptr;
    }
    g_scratch_ptr[dev] = p;
  }
  return g_scratch_ptr[dev];
}
}  // namespace

extern "C" local_status_t local_paged_attn_decode_noalloc(
    const uint16_t* q, int32_t B, int32_t Hq, int32_t Hkv, int32_t D,
    const uint16_t* k_new, const uint16_t* v_new, uint16_t* k_cache, uint16_t* v_cache,
    int64_t num_blocks, int32_t block_size, const int32_t* block_table,
    int32_t max_blocks, const int32_t* ctx_lens, const int32_t* block_version,
    const int32_t* req_version, float sm_scale, uint16_t* out, float* lse, void* stream) {
  const char* who = "paged_attn_decode_noalloc";
  DecodeArgs a;
  size_t part_elems = 0, need = 0;
  local_status_t st = decode_setup(q, B, Hq, Hkv, D, k_new, v_new, k_cache, v_cache,
                                   num_blocks, block_size, block_table, max_blocks, ctx_lens,
                                   block_version, req_version, sm_scale, out, lse, who, &a,
                                   &part_elems, &need);
  if (st != LOCAL_OK) return st;
  if (need > kNoAllocBytes)
    return local_fail(LOCAL_ERR_UNSUPPORTED,
                      "%s: B*Hq*ceil(max_blocks/%d)*(D+2)*4 = %zu bytes of partials exceed the "
                      "library's fixed scratch of %zu bytes (use local_paged_attn_decode with a "
                      "workspace)", who, a.pb, need, kNoAllocBytes);
  if (B == 0) return LOCAL_OK;
  if ((st = decode_pointers_ok(a, who)) != LOCAL_OK) return st;
  void* partials = scratch_of_current_device(&st);
  if (!partials) return st;
  return decode_launch(a, B, D, partials, part_elems, stream);
}
