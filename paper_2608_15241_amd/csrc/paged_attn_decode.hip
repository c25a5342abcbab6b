// local_paged_attn_decode: one new token per request attends over its paged
// KV cache; blocks whose adapter-version tag differs from the request's
// version are excluded (§5.1 validity key; §1 challenge (2)).
//
// Design (HBM-bound: every valid KV byte is read once, stale blocks are never
// read):
//  * Split-KV. Workgroup (partition, kv head g, request b) owns 32 logical
//    blocks (512 tokens); each of its 4 waves owns 8 of them. A wave reads the
//    8 table entries and tags first, keeps the non-stale blocks and walks
//    them two at a time.
//  * Matrix cores, transposed. Per block, S^T[16 keys x 16 cols] =
//    K[16 x D] * Q^T[D x 16] on v_mfma_f32_16x16x32_bf16, where the columns
//    are the Hq/Hkv query heads that share KV head g (zero-padded to 16).
//    The K layout [D/8][16][8] makes each lane's 16-byte A-operand slice
//    contiguous and each MFMA's 64 loads one contiguous kilobyte. The score
//    tile's accumulator layout (lane: 4 keys of one column) is exactly the
//    B-operand layout of the next product O^T[D x 16] += V^T[D x 32] P^T
//    over a pair of blocks, whose A operand comes straight from the V layout
//    [D][16] (each lane: 4 keys of one dim per block, 8 bytes).
//  * Online softmax in the log2 domain per column; the wave's three
//    quantities (max, sum, O) are merged across the 4 waves in LDS, and a
//    second kernel merges partitions when a request has more than one.
//  * The new token's K/V are written at position L-1 by the wave that owns
//    that block; the same wave substitutes them for the cache slot it reads,
//    so no other workgroup and no second launch is involved.
#include "common.hpp"

namespace localk {
namespace {

constexpr int kDecWaves = 4;
constexpr int kDecThreads = kDecWaves * kWave;
constexpr int kBlocksPerWave = 8;
constexpr int kBlocksPerPart = kDecWaves * kBlocksPerWave;  // 32 blocks = 512 tokens
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
  int Hq, Hkv, group, max_blocks, n_parts;
  float scale_log2;  // sm_scale * log2(e)
};

// Replace the 4 V values a lane holds for one block (slots slot0..slot0+3)
// where needed: slots past the last live one become 0 (their cache contents
// are undefined and must not reach the product), the slot being appended
// takes the new value.
__device__ __forceinline__ u32x2 fix_v_last(u32x2 v, int slot0, int s_last, bool has_new,
                                            uint32_t vnew) {
  uint32_t h[4] = {v.x & 0xffffu, v.x >> 16, v.y & 0xffffu, v.y >> 16};
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const int slot = slot0 + e;
    if (slot > s_last) h[e] = 0;
    else if (has_new && slot == s_last) h[e] = vnew;
  }
  u32x2 r;
  r.x = h[0] | (h[1] << 16);
  r.y = h[2] | (h[3] << 16);
  return r;
}

template <int D>
__global__ __launch_bounds__(kDecThreads) void decode_attn_kernel(DecodeArgs a) {
  constexpr int KC = D / 32;  // 32-dim chunks of the QK product
  constexpr int VT = D / 16;  // 16-dim tiles of the PV product
  extern __shared__ float lds[];

  const int part = blockIdx.x, g = blockIdx.y, b = blockIdx.z;
  const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
  const int col = lane % 16, kgrp = lane / 16;
  const int L = a.ctx_lens[b];
  const int nb = (L + kBlockSize - 1) / kBlockSize;
  const int first_block = part * kBlocksPerPart;
  if (first_block >= nb) return;  // whole workgroup: nothing of b here
  const int n_parts_b = (nb + kBlocksPerPart - 1) / kBlocksPerPart;
  const int rv = a.req_version[b];
  const int32_t* table = a.block_table + static_cast<int64_t>(b) * a.max_blocks;
  const int G = a.group;

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

  // This wave's blocks: read table entries and tags, keep the non-stale ones.
  const int j0 = first_block + wave * kBlocksPerWave;
  const int jend = min(j0 + kBlocksPerWave, nb);
  int my_phys = 0;
  bool ok = false;
  if (lane < kBlocksPerWave && j0 + lane < jend) {
    my_phys = table[j0 + lane];
    ok = a.block_version[my_phys] == rv;
  }
  uint64_t valid_mask = __ballot(ok);

  // Append of the new token (position L-1) by the wave that owns its block.
  const int j_new = nb - 1, s_last = (L - 1) % kBlockSize;
  const bool has_new = a.k_new != nullptr;
  const int64_t kvrow = (static_cast<int64_t>(b) * a.Hkv + g) * D;
  if (has_new && j_new >= j0 && j_new < jend) {
    const int p = __shfl(my_phys, j_new - j0);
    const int64_t tile = (static_cast<int64_t>(p) * a.Hkv + g) * (kBlockSize * D);
    if (lane < D / 8) {
      const u32x4 kv = ld_global<u32x4>(a.k_new + kvrow + 8 * lane);
      *reinterpret_cast<u32x4*>(a.k_cache + tile + lane * (kBlockSize * 8) + s_last * 8) = kv;
    }
    for (int d = lane; d < D; d += kWave)
      a.v_cache[tile + d * kBlockSize + s_last] = a.v_new[kvrow + d];
  }

  f32x4 acc[VT];
#pragma unroll
  for (int t = 0; t < VT; ++t) acc[t] = f32x4{0.f, 0.f, 0.f, 0.f};
  float m_run = kNegBig, l_run = 0.f;

  while (valid_mask) {
    const int iA = __builtin_ctzll(valid_mask);
    valid_mask &= valid_mask - 1;
    const int iB = valid_mask ? __builtin_ctzll(valid_mask) : -1;
    if (valid_mask) valid_mask &= valid_mask - 1;
    const int jA = j0 + iA, jB = j0 + iB;
    const int pA = __shfl(my_phys, iA);
    const int pB = __shfl(my_phys, iB < 0 ? iA : iB);
    const int64_t tA = (static_cast<int64_t>(pA) * a.Hkv + g) * (kBlockSize * D);
    const int64_t tB = (static_cast<int64_t>(pB) * a.Hkv + g) * (kBlockSize * D);

    // ---- loads: K as the A operand, V^T as the A operand of the PV product
    u32x4 kA[KC], kB[KC];
    u32x2 vA[VT], vB[VT];
#pragma unroll
    for (int c = 0; c < KC; ++c) {
      const uint16_t* src = a.k_cache + tA + c * 512 + lane * 8;
      if (has_new && jA == j_new && col == s_last) src = a.k_new + kvrow + 32 * c + 8 * kgrp;
      kA[c] = ld_global<u32x4>(src);
    }
#pragma unroll
    for (int t = 0; t < VT; ++t)
      vA[t] = ld_global<u32x2>(a.v_cache + tA + (16 * t + col) * kBlockSize + 4 * kgrp);
    if (iB >= 0) {
#pragma unroll
      for (int c = 0; c < KC; ++c) {
        const uint16_t* src = a.k_cache + tB + c * 512 + lane * 8;
        if (has_new && jB == j_new && col == s_last) src = a.k_new + kvrow + 32 * c + 8 * kgrp;
        kB[c] = ld_global<u32x4>(src);
      }
#pragma unroll
      for (int t = 0; t < VT; ++t)
        vB[t] = ld_global<u32x2>(a.v_cache + tB + (16 * t + col) * kBlockSize + 4 * kgrp);
    } else {
#pragma unroll
      for (int c = 0; c < KC; ++c) kB[c] = u32x4{0u, 0u, 0u, 0u};
#pragma unroll
      for (int t = 0; t < VT; ++t) vB[t] = u32x2{0u, 0u};
    }
    // last block: clear dead slots of V and put the new value in
    if (jA == j_new) {
#pragma unroll
      for (int t = 0; t < VT; ++t)
        vA[t] = fix_v_last(vA[t], 4 * kgrp, s_last, has_new,
                           has_new ? a.v_new[kvrow + 16 * t + col] : 0u);
    }
    if (jB == j_new) {
#pragma unroll
      for (int t = 0; t < VT; ++t)
        vB[t] = fix_v_last(vB[t], 4 * kgrp, s_last, has_new,
                           has_new ? a.v_new[kvrow + 16 * t + col] : 0u);
    }

    // ---- scores S^T (rows = key slots 4*kgrp+i, column = head col)
    f32x4 sA = {0.f, 0.f, 0.f, 0.f}, sB = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int c = 0; c < KC; ++c) {
      sA = mfma16x16x32(as_bf16x8(kA[c]), qv[c], sA);
      sB = mfma16x16x32(as_bf16x8(kB[c]), qv[c], sB);
    }
    float s[8];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int posA = jA * kBlockSize + 4 * kgrp + i;
      const int posB = jB * kBlockSize + 4 * kgrp + i;
      s[i] = posA < L ? sA[i] * a.scale_log2 : -INFINITY;
      s[4 + i] = (iB >= 0 && posB < L) ? sB[i] * a.scale_log2 : -INFINITY;
    }
    float mx = s[0];
#pragma unroll
    for (int i = 1; i < 8; ++i) mx = fmaxf(mx, s[i]);
    mx = fmaxf(mx, __shfl_xor(mx, 16));
    mx = fmaxf(mx, __shfl_xor(mx, 32));
    const float m_new = fmaxf(m_run, mx);
    const float alpha = fast_exp2(m_run - m_new);
    float psum = 0.f;
    bf16x8 pb;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const float p = fast_exp2(s[i] - m_new);
      psum += p;
      pb[i] = static_cast<__bf16>(p);
    }
    l_run = l_run * alpha + psum;
    m_run = m_new;
#pragma unroll
    for (int t = 0; t < VT; ++t) {
      acc[t] *= alpha;
      u32x4 v4 = {vA[t].x, vA[t].y, vB[t].x, vB[t].y};
      acc[t] = mfma16x16x32(as_bf16x8(v4), pb, acc[t]);
    }
  }

  // ---- merge the 4 waves (per column: max, sum, O^T) in LDS
  l_run += __shfl_xor(l_run, 16);
  l_run += __shfl_xor(l_run, 32);
  float* o_lds = lds;                              // [waves][G][D]
  float* ml_lds = lds + kDecWaves * G * D;         // [waves][G][2]
  if (col < G) {
#pragma unroll
    for (int t = 0; t < VT; ++t)
      *reinterpret_cast<f32x4*>(o_lds + (wave * G + col) * D + 16 * t + 4 * kgrp) = acc[t];
    if (kgrp == 0) {
      ml_lds[(wave * G + col) * 2] = m_run;
      ml_lds[(wave * G + col) * 2 + 1] = l_run;
    }
  }
  __syncthreads();
  const bool single = n_parts_b == 1;
  for (int e = threadIdx.x; e < G * D; e += kDecThreads) {
    const int n = e / D, d = e % D;
    float M = kNegBig;
#pragma unroll
    for (int w = 0; w < kDecWaves; ++w) M = fmaxf(M, ml_lds[(w * G + n) * 2]);
    float den = 0.f, num = 0.f;
#pragma unroll
    for (int w = 0; w < kDecWaves; ++w) {
      const float f = fast_exp2(ml_lds[(w * G + n) * 2] - M);
      den += ml_lds[(w * G + n) * 2 + 1] * f;
      num += o_lds[(w * G + n) * D + d] * f;
    }
    const int h = g * G + n;
    const int64_t bh = static_cast<int64_t>(b) * a.Hq + h;
    if (single) {
      a.out[bh * D + d] = f32_to_bf16(den > 0.f ? num / den : 0.f);
      if (d == 0 && a.lse)
        a.lse[bh] = den > 0.f ? (M + __log2f(den)) * kLn2 : -INFINITY;
    } else {
      const int64_t pi = bh * a.n_parts + part;
      a.part_o[pi * D + d] = num;
      if (d == 0) {
        a.part_ml[pi * 2] = M;
        a.part_ml[pi * 2 + 1] = den;
      }
    }
  }
}

// Merge the partitions of every (request, head) that has more than one.
template <int D>
__global__ __launch_bounds__(D) void decode_merge_kernel(DecodeArgs a) {
  const int bh = blockIdx.x;
  const int b = bh / a.Hq;
  const int d = threadIdx.x;
  const int L = a.ctx_lens[b];
  const int nb = (L + kBlockSize - 1) / kBlockSize;
  const int np = (nb + kBlocksPerPart - 1) / kBlocksPerPart;
  if (np == 1) return;  // written by the main kernel
  float M = kNegBig;
  const float* ml = a.part_ml + static_cast<int64_t>(bh) * a.n_parts * 2;
  for (int p = 0; p < np; ++p) M = fmaxf(M, ml[2 * p]);
  float den = 0.f, num = 0.f;
  const float* po = a.part_o + static_cast<int64_t>(bh) * a.n_parts * D;
  for (int p = 0; p < np; ++p) {
    const float f = fast_exp2(ml[2 * p] - M);
    den += ml[2 * p + 1] * f;
    num += po[static_cast<int64_t>(p) * D + d] * f;
  }
  a.out[static_cast<int64_t>(bh) * D + d] = f32_to_bf16(den > 0.f ? num / den : 0.f);
  if (d == 0 && a.lse) a.lse[bh] = den > 0.f ? (M + __log2f(den)) * kLn2 : -INFINITY;
}

template <int D>
local_status_t launch_decode(const DecodeArgs& a, int B, hipStream_t s) {
  const size_t lds = (kDecWaves * a.group * D + kDecWaves * a.group * 2) * sizeof(float);
  dim3 grid(a.n_parts, a.Hkv, B);
  decode_attn_kernel<D><<<grid, kDecThreads, lds, s>>>(a);
  if (a.n_parts > 1) decode_merge_kernel<D><<<B * a.Hq, D, 0, s>>>(a);
  return local_check_launch("paged_attn_decode");
}

}  // namespace
}  // namespace localk

using namespace localk;

extern "C" local_status_t local_paged_attn_decode(
    const uint16_t* q, int32_t B, int32_t Hq, int32_t Hkv, int32_t D,
    const uint16_t* k_new, const uint16_t* v_new, uint16_t* k_cache, uint16_t* v_cache,
    int64_t num_blocks, int32_t block_size, const int32_t* block_table,
    int32_t max_blocks, const int32_t* ctx_lens, const int32_t* block_version,
    const int32_t* req_version, float sm_scale, uint16_t* out, float* lse, void* ws,
    size_t* ws_bytes, void* stream) {
  if (!ws_bytes) return local_fail(LOCAL_ERR_WORKSPACE, "paged_attn_decode: ws_bytes is NULL");
  if (B < 0 || Hq <= 0 || Hkv <= 0 || max_blocks < 1 || num_blocks < 1 || Hq % Hkv != 0)
    return local_fail(LOCAL_ERR_SHAPE,
                      "paged_attn_decode: B=%d Hq=%d Hkv=%d max_blocks=%d num_blocks=%lld", B,
                      Hq, Hkv, max_blocks, (long long)num_blocks);
  if (block_size != kBlockSize || (D != 64 && D != 128) || Hq / Hkv > 16)
    return local_fail(LOCAL_ERR_UNSUPPORTED,
                      "paged_attn_decode: block_size=%d D=%d group=%d (need 16, 64|128, <=16)",
                      block_size, D, Hq / Hkv);
  if ((k_new == nullptr) != (v_new == nullptr))
    return local_fail(LOCAL_ERR_NULL, "paged_attn_decode: k_new and v_new must both be set");
  const int n_parts = (max_blocks + kBlocksPerPart - 1) / kBlocksPerPart;
  const size_t part_elems = static_cast<size_t>(B > 0 ? B : 1) * Hq * n_parts;
  const size_t need = part_elems * (D + 2) * sizeof(float);
  if (!ws) {
    *ws_bytes = need;
    return LOCAL_OK;
  }
  if (*ws_bytes < need)
    return local_fail(LOCAL_ERR_WORKSPACE, "paged_attn_decode: workspace %zu < %zu",
                      *ws_bytes, need);
  if (B == 0) return LOCAL_OK;
  if (!q || !k_cache || !v_cache || !block_table || !ctx_lens || !block_version ||
      !req_version || !out)
    return local_fail(LOCAL_ERR_NULL, "paged_attn_decode: NULL pointer argument");
  DecodeArgs a;
  a.q = q;
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
  a.part_o = static_cast<float*>(ws);
  a.part_ml = a.part_o + part_elems * D;
  a.Hq = Hq;
  a.Hkv = Hkv;
  a.group = Hq / Hkv;
  a.max_blocks = max_blocks;
  a.n_parts = n_parts;
  a.scale_log2 = sm_scale * kLog2e;
  hipStream_t s = static_cast<hipStream_t>(stream);
  return D == 64 ? launch_decode<64>(a, B, s) : launch_decode<128>(a, B, s);
}
