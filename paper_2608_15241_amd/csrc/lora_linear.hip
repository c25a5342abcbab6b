// local_lora_linear: y = x W^T + s_t (x A_a^T) B_a^T with a per-token adapter
// a = adapter_idx[t] (§2.2 "LoRA adapters": one frozen base shared by many
// low-rank adapters, every request routed to its own adapter).
//
// Design, SGMV-style but on the matrix cores end to end:
//  * Shrink. U_s[t, a*r_max + j] = bf16(s_t * x_t . A[a,j,:]) for the token's
//    own adapter a and j < rank(a), 0 elsewhere. It is one GEMM of x against
//    all adapters' stacked A (rows a*r_max + j), whose epilogue keeps only the
//    token's own adapter and rank. Its cost is a few percent of the main
//    product; the gather of adapters per token is replaced by masking.
//  * Fused base + expand. The delta is U_s Btilde^T with
//    Btilde[n, a*r_max + j] = B[a, n, j], i.e. extra K-steps of the base
//    product over the columns of U_s. A K-step of 64 such columns is run only
//    if an adapter it covers is used by some token of the tile, and only the
//    columns below each adapter's rank are loaded; everything else is a zero
//    fill that costs no memory traffic.
//  * Tiles are computed transposed, Y^T = W X^T: features are MFMA rows
//    (A operand, W rows), tokens are columns (B operand, x rows), so each
//    lane ends with 4 consecutive features of one token and stores 8 bytes.
//  * One kernel, two tilings. Prefill (many tokens): 128x128 tiles, 2x2
//    waves, LDS double buffer, XCD-aware grouped tile order so each XCD's L2
//    serves an 8x8 block of tiles. Decode (few tokens, HBM-bound on W):
//    one token tile of <=128 rows, 64 features per workgroup, split-K to put
//    >= 256 workgroups in flight, then a reduction kernel.
#include "common.hpp"

namespace localk {
namespace {

constexpr int kGemmThreads = 256;
constexpr int kBK = 64;
constexpr int kLdsK = kBK + 8;          // padded LDS row (144 bytes): conflict-free reads
constexpr int kMaxLoraSteps = 512;      // R <= 256 * 128 columns / 64
constexpr int kNumXcd = 8;

enum GemmMode { kModeMain = 0, kModeShrink = 1 };

struct GemmArgs {
  const uint16_t* x;     // [T][K]
  const uint16_t* w;     // main: W [N][K]; shrink: stacked A [R][K]
  int64_t T, K, N;       // N = output width (R in shrink mode)
  const uint16_t* us;    // U_s [T][R] (main mode, adapters present)
  const uint16_t* bmat;  // B [n_ad][N][r_max]
  const int32_t* ranks;  // [n_ad] or null
  const int32_t* idx;    // [T] or null
  const float* scale;    // [T]
  int n_ad, r_max, R;
  const uint16_t* res;  // optional residual [T][N] added before rounding (main mode)
  uint16_t* y;           // bf16 output [T][N]   (split == 1)
  float* part;           // fp32 partials [split][T][N] (split > 1)
  int mode, split;
  int gm, gn;            // tile grid
  int swizzle;           // XCD-aware grouped order
};

__device__ __forceinline__ int rank_of(const GemmArgs& a, int ad) {
  return a.ranks ? a.ranks[ad] : a.r_max;
}

template <int BM, int BN, int WM, int WN>
__global__ __launch_bounds__(kGemmThreads) void lora_gemm_kernel(GemmArgs a) {
  constexpr int FN = BN / WN / 16;  // 16-row MFMA tiles per wave along features
  constexpr int FM = BM / WM / 16;  // 16-col MFMA tiles per wave along tokens
  constexpr int W_PIECES = BN * (kBK / 8) / kGemmThreads;
  constexpr int X_PIECES = (BM * (kBK / 8) + kGemmThreads - 1) / kGemmThreads;
  static_assert(W_PIECES >= 1 && WM * WN == 4, "tile shape");
  extern __shared__ __attribute__((aligned(16))) uint16_t smem[];
  // LDS: W tiles [2][BN][kLdsK], then x tiles [2][BM][kLdsK]
  auto w_lds = [&](int buf) { return smem + buf * (BN * kLdsK); };
  auto x_lds = [&](int buf) { return smem + 2 * BN * kLdsK + buf * (BM * kLdsK); };
  __shared__ uint64_t present[4];
  __shared__ uint16_t lora_steps[kMaxLoraSteps];
  __shared__ int wave_cnt[4];

  const int tid = threadIdx.x, wave = tid / kWave, lane = tid % kWave;
  const int col = lane % 16, kgrp = lane / 16;

  // ---- tile coordinates
  int mt, nt;
  {
    const int id = blockIdx.x;
    const int total = a.gm * a.gn;
    int lid = id;
    if (a.swizzle && total % kNumXcd == 0) lid = (id % kNumXcd) * (total / kNumXcd) + id / kNumXcd;
    if (a.swizzle) {
      constexpr int GM = 8;
      const int group = lid / (GM * a.gn);
      const int first_m = group * GM;
      const int gsize = min(a.gm - first_m, GM);
      const int r = lid % (GM * a.gn);
      mt = first_m + r % gsize;
      nt = r / gsize;
    } else {
      mt = lid % a.gm;
      nt = lid / a.gm;
    }
  }
  const int64_t m0 = static_cast<int64_t>(mt) * BM;
  const int64_t n0 = static_cast<int64_t>(nt) * BN;
  const int z = blockIdx.y;

  // ---- adapters used by this token tile, and the LoRA K-steps to run
  int n_lora = 0;
  const bool lora = a.mode == kModeMain && a.n_ad > 0 && a.us != nullptr;
  if (lora) {
    if (tid < 4) present[tid] = 0ull;
    __syncthreads();
    for (int t = tid; t < BM; t += kGemmThreads) {
      if (m0 + t < a.T) {
        const int ad = a.idx[m0 + t];
        if (ad >= 0) atomicOr(reinterpret_cast<unsigned long long*>(&present[ad >> 6]),
                              1ull << (ad & 63));
      }
    }
    __syncthreads();
    const int steps = (a.R + kBK - 1) / kBK;
    for (int base = 0; base < steps; base += kGemmThreads) {
      const int l = base + tid;
      bool use = false;
      if (l < steps) {
        const int a_lo = (l * kBK) / a.r_max;
        const int a_hi = min((l * kBK + kBK - 1) / a.r_max, a.n_ad - 1);
        for (int ad = a_lo; ad <= a_hi; ++ad)
          if ((present[ad >> 6] >> (ad & 63)) & 1ull) use = true;
      }
      const uint64_t m = __ballot(use);
      const int before = __popcll(m & ((1ull << lane) - 1ull));
      if (lane == 0) wave_cnt[wave] = __popcll(m);
      __syncthreads();
      int off = n_lora;
      int tot = 0;
      for (int w2 = 0; w2 < 4; ++w2) {
        if (w2 < wave) off += wave_cnt[w2];
        tot += wave_cnt[w2];
      }
      if (use) lora_steps[off + before] = static_cast<uint16_t>(l);
      n_lora += tot;
      __syncthreads();
    }
  }
  // The base K-steps are split evenly; the LoRA steps go to the last split, so
  // the base product is summed in the same order whether or not any adapter
  // is present.
  const int k_main = static_cast<int>(a.K / kBK);
  const int s_begin = static_cast<int>((static_cast<int64_t>(z) * k_main) / a.split);
  const int s_end = z == a.split - 1
                        ? k_main + n_lora
                        : static_cast<int>((static_cast<int64_t>(z + 1) * k_main) / a.split);

  // ---- global -> register loaders for one K-step
  u32x4 wreg[W_PIECES], xreg[X_PIECES];
  auto load_step = [&](int s) {
    if (s < k_main) {
      const int64_t k0 = static_cast<int64_t>(s) * kBK;
#pragma unroll
      for (int i = 0; i < W_PIECES; ++i) {
        const int piece = tid + i * kGemmThreads;
        const int r = piece / 8, kp = piece % 8;
        const int64_t n = n0 + r;
        wreg[i] = n < a.N ? ld_global<u32x4>(a.w + n * a.K + k0 + 8 * kp) : u32x4{0u, 0u, 0u, 0u};
      }
#pragma unroll
      for (int i = 0; i < X_PIECES; ++i) {
        const int piece = tid + i * kGemmThreads;
        const int r = piece / 8, kp = piece % 8;
        const int64_t t = m0 + r;
        xreg[i] = (piece < BM * 8 && t < a.T) ? ld_global<u32x4>(a.x + t * a.K + k0 + 8 * kp)
                                              : u32x4{0u, 0u, 0u, 0u};
      }
    } else {
      const int l = lora_steps[s - k_main];
      const int c0 = l * kBK;
#pragma unroll
      for (int i = 0; i < W_PIECES; ++i) {
        const int piece = tid + i * kGemmThreads;
        const int r = piece / 8, kp = piece % 8;
        const int64_t n = n0 + r;
        const int c = c0 + 8 * kp;
        u32x4 v = {0u, 0u, 0u, 0u};
        if (c < a.R && n < a.N) {
          const int ad = c / a.r_max, j = c % a.r_max;
          const int rk = rank_of(a, ad);
          if (j < rk && ((present[ad >> 6] >> (ad & 63)) & 1ull)) {
            v = ld_global<u32x4>(a.bmat + (static_cast<int64_t>(ad) * a.N + n) * a.r_max + j);
            if (rk - j < 8) {  // clear columns at or past the rank
              uint32_t wv[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
              for (int e = 0; e < 8; ++e)
                if (j + e >= rk) wv[e / 2] &= (e & 1) ? 0x0000ffffu : 0xffff0000u;
              v = u32x4{wv[0], wv[1], wv[2], wv[3]};
            }
          }
        }
        wreg[i] = v;
      }
#pragma unroll
      for (int i = 0; i < X_PIECES; ++i) {
        const int piece = tid + i * kGemmThreads;
        const int r = piece / 8, kp = piece % 8;
        const int64_t t = m0 + r;
        const int c = c0 + 8 * kp;
        xreg[i] = (piece < BM * 8 && t < a.T && c < a.R)
                      ? ld_global<u32x4>(a.us + t * a.R + c)
                      : u32x4{0u, 0u, 0u, 0u};
      }
    }
  };
  auto store_step = [&](int buf) {
#pragma unroll
    for (int i = 0; i < W_PIECES; ++i) {
      const int piece = tid + i * kGemmThreads;
      *reinterpret_cast<u32x4*>(w_lds(buf) + (piece / 8) * kLdsK + 8 * (piece % 8)) = wreg[i];
    }
#pragma unroll
    for (int i = 0; i < X_PIECES; ++i) {
      const int piece = tid + i * kGemmThreads;
      if (piece < BM * 8)
        *reinterpret_cast<u32x4*>(x_lds(buf) + (piece / 8) * kLdsK + 8 * (piece % 8)) = xreg[i];
    }
  };

  f32x4 acc[FN][FM];
#pragma unroll
  for (int i = 0; i < FN; ++i)
#pragma unroll
    for (int j = 0; j < FM; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  const int wn = wave % WN, wm = wave / WN;
  const int wrow0 = wn * (BN / WN);  // this wave's first feature row in the tile
  const int wcol0 = wm * (BM / WM);  // this wave's first token column

  if (s_begin < s_end) {
    load_step(s_begin);
    store_step(0);
    __syncthreads();
    int cur = 0;
    for (int s = s_begin; s < s_end; ++s) {
      const bool more = s + 1 < s_end;
      if (more) load_step(s + 1);
#pragma unroll
      for (int kk = 0; kk < kBK / 32; ++kk) {
        bf16x8 af[FN], bfr[FM];
#pragma unroll
        for (int i = 0; i < FN; ++i)
          af[i] = as_bf16x8(*reinterpret_cast<const u32x4*>(
              w_lds(cur) + (wrow0 + 16 * i + col) * kLdsK + 32 * kk + 8 * kgrp));
#pragma unroll
        for (int j = 0; j < FM; ++j)
          bfr[j] = as_bf16x8(*reinterpret_cast<const u32x4*>(
              x_lds(cur) + (wcol0 + 16 * j + col) * kLdsK + 32 * kk + 8 * kgrp));
#pragma unroll
        for (int i = 0; i < FN; ++i)
#pragma unroll
          for (int j = 0; j < FM; ++j) acc[i][j] = mfma16x16x32(af[i], bfr[j], acc[i][j]);
      }
      if (more) store_step(cur ^ 1);
      __syncthreads();
      cur ^= 1;
    }
  }

  // ---- epilogue: lane holds features n..n+3 (rows) of token t (column)
#pragma unroll
  for (int j = 0; j < FM; ++j) {
    const int64_t t = m0 + wcol0 + 16 * j + col;
    if (t >= a.T) continue;
#pragma unroll
    for (int i = 0; i < FN; ++i) {
      const int64_t n = n0 + wrow0 + 16 * i + 4 * kgrp;
      if (n >= a.N) continue;
      const f32x4 v = acc[i][j];
      if (a.mode == kModeShrink) {
        const int ad = a.idx ? a.idx[t] : -1;
        const float sc = ad >= 0 ? a.scale[t] : 0.f;
        float o[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int r = static_cast<int>(n) + e;
          const int rad = r / a.r_max, rj = r % a.r_max;
          o[e] = (ad >= 0 && rad == ad && rj < rank_of(a, ad)) ? sc * v[e] : 0.f;
        }
        *reinterpret_cast<u32x2*>(a.y + t * a.N + n) =
            u32x2{pack_bf16x2(o[0], o[1]), pack_bf16x2(o[2], o[3])};
      } else if (a.split == 1) {
        f32x4 o = v;
        if (a.res) {
          const u32x2 r = ld_global<u32x2>(a.res + t * a.N + n);
          o[0] += __uint_as_float(r.x << 16);
          o[1] += __uint_as_float(r.x & 0xffff0000u);
          o[2] += __uint_as_float(r.y << 16);
          o[3] += __uint_as_float(r.y & 0xffff0000u);
        }
        *reinterpret_cast<u32x2*>(a.y + t * a.N + n) =
            u32x2{pack_bf16x2(o[0], o[1]), pack_bf16x2(o[2], o[3])};
      } else {
        *reinterpret_cast<f32x4*>(a.part + (static_cast<int64_t>(z) * a.T + t) * a.N + n) = v;
      }
    }
  }
}

// y[t, n..n+3] = bf16(residual + sum over splits of the partials), summed in
// split order.
__global__ __launch_bounds__(256) void splitk_reduce_kernel(const float* __restrict__ part,
                                                            int split, int64_t TN,
                                                            const uint16_t* __restrict__ res,
                                                            uint16_t* __restrict__ y) {
  const int64_t e4 = (static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x) * 4;
  if (e4 >= TN) return;
  f32x4 s = *reinterpret_cast<const f32x4*>(part + e4);
  for (int z = 1; z < split; ++z) s += *reinterpret_cast<const f32x4*>(part + z * TN + e4);
  if (res) {
    const u32x2 r = ld_global<u32x2>(res + e4);
    s[0] += __uint_as_float(r.x << 16);
    s[1] += __uint_as_float(r.x & 0xffff0000u);
    s[2] += __uint_as_float(r.y << 16);
    s[3] += __uint_as_float(r.y & 0xffff0000u);
  }
  *reinterpret_cast<u32x2*>(y + e4) = u32x2{pack_bf16x2(s[0], s[1]), pack_bf16x2(s[2], s[3])};
}

struct Tiling {
  int bm, bn, split;
};

template <int BM, int BN, int WM, int WN>
local_status_t launch_gemm(GemmArgs a, hipStream_t s) {
  a.gm = static_cast<int>((a.T + BM - 1) / BM);
  a.gn = static_cast<int>((a.N + BN - 1) / BN);
  const size_t lds = static_cast<size_t>(2 * (BN + BM) * kLdsK) * sizeof(uint16_t);
  static bool attr_set = false;  // benign race: the attribute value is the same
  if (!attr_set) {
    (void)hipFuncSetAttribute(reinterpret_cast<const void*>(lora_gemm_kernel<BM, BN, WM, WN>),
                        hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(lds));
    attr_set = true;
  }
  dim3 grid(a.gm * a.gn, a.split);
  lora_gemm_kernel<BM, BN, WM, WN><<<grid, kGemmThreads, lds, s>>>(a);
  return local_check_launch("lora_linear (gemm)");
}

// Choose the tile for a product of T tokens x N features over total_steps
// K-steps of 64.
local_status_t run_gemm(GemmArgs a, int total_steps_hint, hipStream_t s) {
  if (a.T > 256) {
    a.split = 1;
    a.swizzle = 1;
    return launch_gemm<128, 128, 2, 2>(a, s);
  }
  a.swizzle = 0;
  const int64_t n_tiles = (a.N + 63) / 64;
  const int64_t m_tiles = (a.T + 127) / 128;
  int split = 1;
  if (a.mode == kModeMain && a.part != nullptr) {
    while (split < 8 && n_tiles * m_tiles * split < 256 && total_steps_hint / (2 * split) >= 4)
      split *= 2;
  }
  a.split = split;
  local_status_t st;
  if (a.T <= 32) st = launch_gemm<32, 64, 1, 4>(a, s);
  else if (a.T <= 64) st = launch_gemm<64, 64, 1, 4>(a, s);
  else st = launch_gemm<128, 64, 1, 4>(a, s);
  if (st != LOCAL_OK || split == 1) return st;
  const int64_t TN = a.T * a.N;
  const int64_t blocks = (TN / 4 + 255) / 256;
  splitk_reduce_kernel<<<static_cast<unsigned>(blocks), 256, 0, s>>>(a.part, split, TN, a.res,
                                                                    a.y);
  return local_check_launch("lora_linear (split-K reduce)");
}

size_t align256(size_t v) { return (v + 255) & ~static_cast<size_t>(255); }

}  // namespace
}  // namespace localk

using namespace localk;

extern "C" local_status_t local_lora_linear(
    const uint16_t* x, int64_t T, int64_t K, const uint16_t* W, int64_t N, const uint16_t* A,
    const uint16_t* B, int32_t n_adapters, int32_t r_max, const int32_t* ranks,
    const int32_t* adapter_idx, const float* scale, const uint16_t* residual, uint16_t* y,
    void* ws, size_t* ws_bytes, void* stream) {
  if (!ws_bytes) return local_fail(LOCAL_ERR_WORKSPACE, "lora_linear: ws_bytes is NULL");
  if (T < 0 || K <= 0 || N <= 0 || n_adapters < 0)
    return local_fail(LOCAL_ERR_SHAPE, "lora_linear: T=%lld K=%lld N=%lld n_adapters=%d",
                      (long long)T, (long long)K, (long long)N, n_adapters);
  if (K % 64 != 0 || N % 64 != 0 || n_adapters > 256 ||
      (n_adapters > 0 && (r_max < 8 || r_max > 128 || r_max % 8 != 0)))
    return local_fail(LOCAL_ERR_UNSUPPORTED,
                      "lora_linear: K=%lld N=%lld n_adapters=%d r_max=%d (need K,N %% 64 == 0, "
                      "n_adapters <= 256, r_max in [8,128] and %% 8 == 0)",
                      (long long)K, (long long)N, n_adapters, r_max);
  const int R = n_adapters > 0 ? n_adapters * r_max : 0;
  // workspace: U_s [T][R] bf16, then split-K partials [8][T][N] fp32 for T <= 256
  const size_t us_bytes = align256(static_cast<size_t>(T) * R * sizeof(uint16_t));
  const size_t part_bytes =
      T <= 256 ? align256(static_cast<size_t>(8) * T * N * sizeof(float)) : 0;
  const size_t need = us_bytes + part_bytes;
  if (!ws) {
    *ws_bytes = need;
    return LOCAL_OK;
  }
  if (*ws_bytes < need)
    return local_fail(LOCAL_ERR_WORKSPACE, "lora_linear: workspace %zu < %zu", *ws_bytes, need);
  if (T == 0) return LOCAL_OK;
  if (!x || !W || !y) return local_fail(LOCAL_ERR_NULL, "lora_linear: NULL x, W or y");
  if (n_adapters > 0 && (!A || !B || !adapter_idx || !scale))
    return local_fail(LOCAL_ERR_NULL, "lora_linear: NULL adapter argument");
  hipStream_t s = static_cast<hipStream_t>(stream);
  uint16_t* us = n_adapters > 0 ? static_cast<uint16_t*>(ws) : nullptr;
  float* part = part_bytes ? reinterpret_cast<float*>(static_cast<char*>(ws) + us_bytes) : nullptr;

  if (n_adapters > 0) {
    GemmArgs sh{};
    sh.x = x;
    sh.w = A;  // [n_ad][r_max][K] == [R][K]
    sh.T = T;
    sh.K = K;
    sh.N = R;
    sh.idx = adapter_idx;
    sh.scale = scale;
    sh.ranks = ranks;
    sh.n_ad = n_adapters;
    sh.r_max = r_max;
    sh.R = R;
    sh.y = us;
    sh.mode = kModeShrink;
    local_status_t st = run_gemm(sh, static_cast<int>(K / 64), s);
    if (st != LOCAL_OK) return st;
  }
  GemmArgs m{};
  m.x = x;
  m.w = W;
  m.T = T;
  m.K = K;
  m.N = N;
  m.us = us;
  m.bmat = B;
  m.ranks = ranks;
  m.idx = adapter_idx;
  m.scale = scale;
  m.n_ad = n_adapters;
  m.r_max = r_max;
  m.R = R;
  m.res = residual;
  m.y = y;
  m.part = part;
  m.mode = kModeMain;
  return run_gemm(m, static_cast<int>(K / 64), s);
}
