// local_paged_attn_prefill: a chunk of new tokens per request is appended to
// the paged KV cache, then attends causally over cached prefix plus chunk
// with the per-block version mask (§4.1 chunked prefill; §5.3 stale-coverage
// prefill is the same computation under a staged version).
//
// Design (matrix-core bound):
//  * An append kernel first writes the chunk's K/V into its slots; every
//    attention workgroup that reads the chunk runs after it on the stream.
//  * Attention workgroup = (query tile of 64*QT rows, query head h, request b):
//    4 waves, each owning 16*QT query rows as matrix columns. The request's
//    non-stale blocks up to the tile's causal limit are compacted with
//    ballots, then staged KB blocks at a time into LDS in the pool's own
//    layout (so every operand read is a contiguous 16- or 8-byte LDS slice).
//  * S^T = K Q^T and O^T += V^T P^T on v_mfma_f32_16x16x32_bf16, the same
//    transposed formulation as decode: the score accumulator is already the
//    B operand of the value product, so no lane shuffle of P is needed.
//    Causal and dead-slot masking, online softmax in the log2 domain.
#include "common.hpp"

namespace localk {
namespace {

constexpr int kPfWaves = 4;
constexpr int kPfThreads = kPfWaves * kWave;
constexpr int kPfKB = 4;  // blocks staged per tile (64 keys)
constexpr int kPfWindow = kPfThreads;  // block-table entries compacted per pass
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

__device__ __forceinline__ int find_request(const int32_t* __restrict__ q_indptr, int B,
                                            int64_t t) {
  int lo = 0, hi = B - 1;  // last b with q_indptr[b] <= t
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (q_indptr[mid] <= t) lo = mid;
    else hi = mid - 1;
  }
  return lo;
}

// One workgroup per chunk row: write its K and V for every KV head.
template <int D>
__global__ __launch_bounds__(256) void prefill_append_kernel(PrefillArgs a) {
  const int64_t t = blockIdx.x;
  int b = find_request(a.q_indptr, a.B, t);
  while (b + 1 < a.B && a.q_indptr[b + 1] <= t) ++b;  // skip empty requests
  const int n_b = a.q_indptr[b + 1] - a.q_indptr[b];
  const int pos = a.ctx_lens[b] - n_b + static_cast<int>(t - a.q_indptr[b]);
  // positions without a block, or blocks with an id outside the pool, are
  // not written
  if (pos < 0 || pos / kBlockSize >= a.max_blocks) return;
  const int p = a.block_table[static_cast<int64_t>(b) * a.max_blocks + pos / kBlockSize];
  if (!id_ok(p, a.num_blocks)) return;
  const int slot = pos % kBlockSize;
  const int n16 = a.Hkv * (D / 8);
  for (int e = threadIdx.x; e < n16; e += blockDim.x) {
    const int g = e / (D / 8), c = e % (D / 8);
    const int64_t tile = (static_cast<int64_t>(p) * a.Hkv + g) * (kBlockSize * D);
    const u32x4 kv = ld_global<u32x4>(a.k_new + (t * a.Hkv + g) * D + 8 * c);
    *reinterpret_cast<u32x4*>(a.k_cache + tile + c * (kBlockSize * 8) + slot * 8) = kv;
  }
  for (int e = threadIdx.x; e < a.Hkv * D; e += blockDim.x) {
    const int g = e / D, d = e % D;
    const int64_t tile = (static_cast<int64_t>(p) * a.Hkv + g) * (kBlockSize * D);
    a.v_cache[tile + d * kBlockSize + slot] = a.v_new[(t * a.Hkv + g) * D + d];
  }
}

template <int D, int QT>
__global__ __launch_bounds__(kPfThreads) void prefill_attn_kernel(PrefillArgs a) {
  constexpr int KC = D / 32, VT = D / 16;
  constexpr int TILE = kBlockSize * D;          // elements per (block, head) tile
  constexpr int ROWS_PER_WG = kPfWaves * 16 * QT;
  __shared__ __attribute__((aligned(16))) uint16_t k_lds[kPfKB * TILE];
  __shared__ __attribute__((aligned(16))) uint16_t v_lds[kPfKB * TILE];
  __shared__ int list[kPfWindow];
  __shared__ int wave_cnt[kPfWaves];

  const int qtile = blockIdx.x, h = blockIdx.y, b = blockIdx.z;
  const int r0 = a.q_indptr[b], r1 = a.q_indptr[b + 1];
  if (r0 < 0 || r1 > a.T || r1 < r0) return;  // not a row range of q
  const int n_b = r1 - r0;
  const int row0 = qtile * ROWS_PER_WG;
  if (row0 >= n_b) return;
  const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
  const int col = lane % 16, kgrp = lane / 16;
  const int L = a.ctx_lens[b];
  const int P = L - n_b;  // cached prefix
  const int g = h / a.group;
  const int rv = a.req_version[b];
  const int32_t* table = a.block_table + static_cast<int64_t>(b) * a.max_blocks;

  // Query columns of this wave: rows row0 + wave*16*QT + 16*ct + col.
  bf16x8 qv[QT][KC];
  int qpos[QT];
#pragma unroll
  for (int ct = 0; ct < QT; ++ct) {
    const int row = row0 + wave * 16 * QT + 16 * ct + col;
    qpos[ct] = P + row;
#pragma unroll
    for (int c = 0; c < KC; ++c) {
      u32x4 v = {0u, 0u, 0u, 0u};
      if (row < n_b)
        v = ld_global<u32x4>(a.q + (static_cast<int64_t>(r0 + row) * a.Hq + h) * D + 32 * c +
                             8 * kgrp);
      qv[ct][c] = as_bf16x8(v);
    }
  }
  const int wave_last_row = min(row0 + (wave + 1) * 16 * QT, n_b) - 1;
  const int wave_limit = P + wave_last_row;  // largest key position this wave sees
  const int wg_limit = P + min(row0 + ROWS_PER_WG, n_b) - 1;
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

  for (int w0 = 0; w0 < nb_lim; w0 += kPfWindow) {
    // ---- compact the non-stale blocks of this window (in ascending j)
    const int j = w0 + threadIdx.x;
    bool ok = false;
    if (j < nb_lim) {
      const int p = table[j];
      ok = id_ok(p, a.num_blocks) && a.block_version[p] == rv;
    }
    const uint64_t mask = __ballot(ok);
    const int before = __popcll(mask & ((1ull << lane) - 1ull));
    if (lane == 0) wave_cnt[wave] = __popcll(mask);
    __syncthreads();
    int off = 0, cnt = 0;
    for (int w = 0; w < kPfWaves; ++w) {
      if (w < wave) off += wave_cnt[w];
      cnt += wave_cnt[w];
    }
    if (ok) list[off + before] = j;
    __syncthreads();

    for (int t0 = 0; t0 < cnt; t0 += kPfKB) {
      // ---- stage KB blocks (K and V tiles) into LDS
      for (int e = threadIdx.x; e < kPfKB * TILE / 8; e += kPfThreads) {
        const int kb = e / (TILE / 8), piece = e % (TILE / 8);
        u32x4 kv = {0u, 0u, 0u, 0u}, vv = {0u, 0u, 0u, 0u};
        if (t0 + kb < cnt) {
          const int jj = list[t0 + kb];
          const int64_t tile = (static_cast<int64_t>(table[jj]) * a.Hkv + g) * TILE;
          kv = ld_global<u32x4>(a.k_cache + tile + 8 * piece);
          vv = ld_global<u32x4>(a.v_cache + tile + 8 * piece);
          // V piece = 8 slots of one dim: clear slots past the context end
          const int slot0 = (8 * piece) % kBlockSize;
          const int live = L - jj * kBlockSize - slot0;  // live slots in this piece
          if (live < 8) {
            uint32_t w[4] = {vv.x, vv.y, vv.z, vv.w};
#pragma unroll
            for (int e2 = 0; e2 < 8; ++e2)
              if (e2 >= live) w[e2 / 2] &= (e2 & 1) ? 0x0000ffffu : 0xffff0000u;
            vv = u32x4{w[0], w[1], w[2], w[3]};
          }
        }
        *reinterpret_cast<u32x4*>(k_lds + kb * TILE + 8 * piece) = kv;
        *reinterpret_cast<u32x4*>(v_lds + kb * TILE + 8 * piece) = vv;
      }
      __syncthreads();

      const int first_pos = list[t0] * kBlockSize;
      if (first_pos <= wave_limit) {
#pragma unroll
        for (int pr = 0; pr < kPfKB / 2; ++pr) {
          const int kbA = 2 * pr, kbB = 2 * pr + 1;
          const bool hasA = t0 + kbA < cnt, hasB = t0 + kbB < cnt;
          if (!hasA) break;
          const int jA = list[t0 + kbA];
          const int jB = hasB ? list[t0 + kbB] : jA;
          const uint16_t* kA = k_lds + kbA * TILE;
          const uint16_t* kB = k_lds + kbB * TILE;
          bf16x8 kfa[KC], kfb[KC];
#pragma unroll
          for (int c = 0; c < KC; ++c) {
            kfa[c] = as_bf16x8(*reinterpret_cast<const u32x4*>(kA + c * 512 + lane * 8));
            kfb[c] = as_bf16x8(*reinterpret_cast<const u32x4*>(kB + c * 512 + lane * 8));
          }
          bf16x8 vf[VT];
#pragma unroll
          for (int t = 0; t < VT; ++t) {
            const u32x2 va = *reinterpret_cast<const u32x2*>(v_lds + kbA * TILE +
                                                             (16 * t + col) * kBlockSize + 4 * kgrp);
            const u32x2 vb = *reinterpret_cast<const u32x2*>(v_lds + kbB * TILE +
                                                             (16 * t + col) * kBlockSize + 4 * kgrp);
            vf[t] = as_bf16x8(u32x4{va.x, va.y, vb.x, vb.y});
          }
#pragma unroll
          for (int ct = 0; ct < QT; ++ct) {
            f32x4 sA = {0.f, 0.f, 0.f, 0.f}, sB = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int c = 0; c < KC; ++c) {
              sA = mfma16x16x32(kfa[c], qv[ct][c], sA);
              sB = mfma16x16x32(kfb[c], qv[ct][c], sB);
            }
            float s[8];
#pragma unroll
            for (int i = 0; i < 4; ++i) {
              const int posA = jA * kBlockSize + 4 * kgrp + i;
              const int posB = jB * kBlockSize + 4 * kgrp + i;
              s[i] = posA <= qpos[ct] ? sA[i] * a.scale_log2 : -INFINITY;
              s[4 + i] = (hasB && posB <= qpos[ct]) ? sB[i] * a.scale_log2 : -INFINITY;
            }
            float mx = s[0];
#pragma unroll
            for (int i = 1; i < 8; ++i) mx = fmaxf(mx, s[i]);
            mx = fmaxf(mx, __shfl_xor(mx, 16));
            mx = fmaxf(mx, __shfl_xor(mx, 32));
            const float m_new = fmaxf(m_run[ct], mx);
            const float alpha = fast_exp2(m_run[ct] - m_new);
            float psum = 0.f;
            bf16x8 pb;
#pragma unroll
            for (int i = 0; i < 8; ++i) {
              const float p = fast_exp2(s[i] - m_new);
              psum += p;
              pb[i] = static_cast<__bf16>(p);
            }
            l_run[ct] = l_run[ct] * alpha + psum;
            m_run[ct] = m_new;
#pragma unroll
            for (int t = 0; t < VT; ++t) {
              acc[ct][t] *= alpha;
              acc[ct][t] = mfma16x16x32(vf[t], pb, acc[ct][t]);
            }
          }
        }
      }
      __syncthreads();
    }
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
local_status_t launch_prefill(const PrefillArgs& a, int64_t T, int max_rows, hipStream_t s) {
  constexpr int QT = 1;
  if (a.k_new) {
    prefill_append_kernel<D><<<static_cast<unsigned>(T), 256, 0, s>>>(a);
    local_status_t st = local_check_launch("paged_attn_prefill (append)");
    if (st != LOCAL_OK) return st;
  }
  const int rows_per_wg = kPfWaves * 16 * QT;
  dim3 grid((max_rows + rows_per_wg - 1) / rows_per_wg, a.Hq, a.B);
  prefill_attn_kernel<D, QT><<<grid, kPfThreads, 0, s>>>(a);
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
  // A request's chunk is at most T rows and at most its table's width.
  const int max_rows = static_cast<int>(T < 16LL * max_blocks ? T : 16LL * max_blocks);
  hipStream_t s = static_cast<hipStream_t>(stream);
  return D == 64 ? launch_prefill<64>(a, T, max_rows, s) : launch_prefill<128>(a, T, max_rows, s);
}
