// local_lora_linear: y = res + x W^T + s_t (x A_a^T) B_a^T with a per-token
// adapter a = adapter_idx[t] (§2.2 "LoRA adapters": one frozen base shared by
// many low-rank adapters, every request routed to its own adapter).
//
// Design, SGMV-style but on the matrix cores end to end:
//  * Shrink. U_s[t, a*r_max + j] = bf16(s_t * x_t . A[a,j,:]) for the token's
//    own adapter a and j < rank(a), 0 elsewhere. It is one product of x with
//    all adapters' stacked A (rows a*r_max + j) whose epilogue keeps only the
//    token's own adapter and rank: the per-token gather of adapters becomes a
//    mask, at a cost of a few percent of the base product.
//  * Fused base + expand. The delta is U_s Btilde^T with
//    Btilde[n, a*r_max + j] = B[a, n, j], i.e. extra K-steps of the base
//    product over the columns of U_s. A step over U_s columns runs only if an
//    adapter it covers is used by a token of the tile, and only columns below
//    each adapter's rank are loaded; the rest is a zero fill with no traffic.
//  * Every tile is computed transposed, Y^T = W X^T: features are MFMA rows
//    (A operand, rows of W), tokens are columns (B operand, rows of x), so a
//    lane ends with 4 consecutive features of one token (an 8-byte store).
//  * Two kernels for two regimes:
//    - skinny (few tokens, or few features): decode projections are bound by
//      streaming W once. A workgroup owns 16 features x up to 128 tokens and
//      its 8 waves split K; each lane loads its MFMA operand slices straight
//      from global memory several K-steps ahead (no LDS staging, no barrier
//      in the main loop), and the 8 partial tiles are summed once through LDS
//      in a fixed order. Also the shrink of a long prefill chunk.
//    - SGMV shrink (decode sizes): one workgroup per adapter computes the
//      shrink of the tokens routed to it on the matrix cores; each adapter's
//      A is read once and no partial sums leave the workgroup.
//    - tiled (many tokens and features): prefill projections are bound by the
//      matrix cores. 128x128 tiles, 2x2 waves, register prefetch into an LDS
//      double buffer with padded rows, XCD-aware grouped tile order so each
//      XCD's L2 serves an 8x8 block of tiles.
//  Both sum the base K-steps in an order that does not depend on which
//  adapters are present, so a zero up-projection leaves y bit-identical.
#include "common.hpp"

namespace localk {
namespace {

constexpr int kGemmThreads = 256;       // tiled kernel
constexpr int kSkThreads = 512;         // skinny kernel (8 waves)
constexpr int kSkWaves = kSkThreads / kWave;
constexpr int kBK = 64;
constexpr int kLdsK = kBK + 8;          // padded LDS row (144 bytes): conflict-free reads
constexpr int kMaxLoraChunks = 1024;    // R <= 256 * 128 columns, in chunks of 32
constexpr int kNumXcd = 8;

#ifndef LOCAL_SK_U32
#define LOCAL_SK_U32 4     // K-steps of 64 per batch of loads, 32-token tiles
#endif
#ifndef LOCAL_SK_FN32
#define LOCAL_SK_FN32 1    // 16-feature tiles per workgroup at 32 tokens
#endif
#ifndef LOCAL_SK_FN64
#define LOCAL_SK_FN64 1    // 16-feature tiles per workgroup at 64 tokens
#endif
#ifndef LOCAL_SK_FN128
#define LOCAL_SK_FN128 1   // 16-feature tiles per workgroup at 128 tokens
#endif

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
  const uint16_t* res;   // optional residual [T][N] (main mode)
  uint16_t* y;           // bf16 output [T][N] (U_s in shrink mode)
  int ksplit;            // K slices of the skinny kernel (grid.z); 1 = whole K
  int mode;
  int gm, gn;            // tile grid of the tiled kernel
  int swizzle;           // XCD-aware grouped order (tiled kernel)
};

// Rank of adapter ad, clamped to [0, r_max] so that no rank reads past the
// adapter's own rows.
__device__ __forceinline__ int rank_of(const GemmArgs& a, int ad) {
  return a.ranks ? min(max(a.ranks[ad], 0), a.r_max) : a.r_max;
}

__device__ __forceinline__ bool adapter_present(const uint64_t* present, int ad) {
  return (present[ad >> 6] >> (ad & 63)) & 1ull;
}

// Store features n..n+3 of token t (bounds-checked): the shrink mask and
// scale, or the residual, then one rounding to bf16.
__device__ __forceinline__ void store4(const GemmArgs& a, int64_t t, int64_t n, f32x4 v) {
  if (t >= a.T || n >= a.N) return;
  float o[4] = {v[0], v[1], v[2], v[3]};
  if (a.mode == kModeShrink) {
    int ad = a.idx ? a.idx[t] : -1;
    if (ad >= a.n_ad) ad = -1;  // indices outside [0, n_ad) mean no adapter
    const float sc = ad >= 0 ? a.scale[t] : 0.f;
    const int rk = ad >= 0 ? rank_of(a, ad) : 0;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int r = static_cast<int>(n) + e;
      o[e] = (ad >= 0 && r / a.r_max == ad && r % a.r_max < rk) ? sc * o[e] : 0.f;
    }
  } else if (a.res) {
    const u32x2 r = ld_global<u32x2>(a.res + t * a.N + n);
    o[0] += __uint_as_float(r.x << 16);
    o[1] += __uint_as_float(r.x & 0xffff0000u);
    o[2] += __uint_as_float(r.y << 16);
    o[3] += __uint_as_float(r.y & 0xffff0000u);
  }
  *reinterpret_cast<u32x2*>(a.y + t * a.N + n) =
      u32x2{pack_bf16x2(o[0], o[1]), pack_bf16x2(o[2], o[3])};
}

// Marks the adapters used by tokens [t0, t0 + n_tok) and lists, in ascending
// order, the chunks of `chunk` U_s columns that cover at least one of them.
// Returns the number of chunks. All threads of the workgroup must call it.
template <int THREADS>
__device__ int lora_chunk_list(const GemmArgs& a, int64_t t0, int n_tok, int chunk,
                               uint64_t* present, uint16_t* list, int* wave_cnt) {
  constexpr int WAVES = THREADS / kWave;
  const int tid = threadIdx.x, wave = tid / kWave, lane = tid % kWave;
  if (tid < 4) present[tid] = 0ull;
  __syncthreads();
  for (int t = tid; t < n_tok; t += THREADS) {
    if (t0 + t < a.T) {
      const int ad = a.idx[t0 + t];
      if (ad >= 0 && ad < a.n_ad)
        atomicOr(reinterpret_cast<unsigned long long*>(&present[ad >> 6]), 1ull << (ad & 63));
    }
  }
  __syncthreads();
  const int chunks = (a.R + chunk - 1) / chunk;
  int n = 0;
  for (int base = 0; base < chunks; base += THREADS) {
    const int l = base + tid;
    bool use = false;
    if (l < chunks) {
      const int a_lo = (l * chunk) / a.r_max;
      const int a_hi = min((l * chunk + chunk - 1) / a.r_max, a.n_ad - 1);
      for (int ad = a_lo; ad <= a_hi; ++ad) use |= adapter_present(present, ad);
    }
    const uint64_t m = __ballot(use);
    const int before = __popcll(m & ((1ull << lane) - 1ull));
    if (lane == 0) wave_cnt[wave] = __popcll(m);
    __syncthreads();
    int off = n, tot = 0;
    for (int w2 = 0; w2 < WAVES; ++w2) {
      if (w2 < wave) off += wave_cnt[w2];
      tot += wave_cnt[w2];
    }
    if (use) list[off + before] = static_cast<uint16_t>(l);
    n += tot;
    __syncthreads();
  }
  return n;
}

// 16-byte slice of Btilde row n at U_s column c (c % 8 == 0): zero when the
// adapter is absent from the tile or the columns lie at or past its rank.
__device__ __forceinline__ u32x4 load_btilde(const GemmArgs& a, const uint64_t* present,
                                             int64_t n, int c) {
  u32x4 v = {0u, 0u, 0u, 0u};
  if (c >= a.R || n >= a.N) return v;
  const int ad = c / a.r_max, j = c % a.r_max;
  const int rk = rank_of(a, ad);
  if (j >= rk || !adapter_present(present, ad)) return v;
  v = ld_global<u32x4>(a.bmat + (static_cast<int64_t>(ad) * a.N + n) * a.r_max + j);
  if (rk - j < 8) {  // clear columns at or past the rank
    uint32_t wv[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int e = 0; e < 8; ++e)
      if (j + e >= rk) wv[e / 2] &= (e & 1) ? 0x0000ffffu : 0xffff0000u;
    v = u32x4{wv[0], wv[1], wv[2], wv[3]};
  }
  return v;
}

// ------------------------------------------------------------------ skinny
// Workgroup: features [n0, n0 + 16*FN) x tokens [t0, t0 + 16*FM); wave w takes
// a contiguous range of the K/32 base steps (U steps per batch of loads) and
// every 8th U_s chunk; partial tiles are summed through LDS in wave order.
// An 8-wave workgroup runs two waves per SIMD; telling the compiler so lets it
// keep a whole batch of loads in registers instead of interleaving each load
// with the MFMA that consumes it (which leaves one load in flight per wave).
template <int FN, int FM, int U>
__global__ __launch_bounds__(kSkThreads) __attribute__((amdgpu_waves_per_eu(2, 2)))
void lora_skinny_kernel(GemmArgs a) {
  __shared__ uint64_t present[4];
  __shared__ uint16_t chunks[kMaxLoraChunks];
  __shared__ int wave_cnt[kSkWaves];
  extern __shared__ f32x4 red[];  // [waves][FM][FN][64 lanes]

  const int tid = threadIdx.x, wave = tid / kWave, lane = tid % kWave;
  const int col = lane % 16, kgrp = lane / 16;
  const int64_t n0 = static_cast<int64_t>(blockIdx.x) * 16 * FN;
  const int64_t t0 = static_cast<int64_t>(blockIdx.y) * 16 * FM;

  int n_chunks = 0;
  if (a.mode == kModeMain && a.n_ad > 0 && a.us != nullptr)
    n_chunks = lora_chunk_list<kSkThreads>(a, t0, 16 * FM, 32, present, chunks, wave_cnt);

  f32x4 acc[FN][FM];
#pragma unroll
  for (int i = 0; i < FN; ++i)
#pragma unroll
    for (int j = 0; j < FM; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  // this lane's rows: feature rows of W, token rows of x
  const uint16_t* wrow[FN];
  bool wok[FN];
#pragma unroll
  for (int i = 0; i < FN; ++i) {
    const int64_t n = n0 + 16 * i + col;
    wok[i] = n < a.N;
    wrow[i] = a.w + (wok[i] ? n : 0) * a.K;
  }
  const uint16_t* xrow[FM];
  bool xok[FM];
#pragma unroll
  for (int j = 0; j < FM; ++j) {
    const int64_t t = t0 + 16 * j + col;
    xok[j] = t < a.T;
    xrow[j] = a.x + (xok[j] ? t : 0) * a.K;
  }

  // Loads are unconditional (rows are clamped to a valid one above, steps
  // past the wave's range to its last step) and invalid values are zeroed
  // with selects, so the loop has no branch around a load and each batch of
  // MFMAs waits only for its own loads.
  //
  // A step covers 64 k as two MFMAs. The k order inside a step is permuted
  // (MFMA m, k-group g takes k = 16g + 8m .. +8), which is the same for both
  // operands and so leaves the product unchanged, but lets every lane load 32
  // contiguous bytes: each row of W and x is read as whole 128-byte lines.
  // Every workgroup reads the same rows of x. Each one takes the 8 K ranges
  // of its slice in a rotated order (wave w takes range (w + rot) mod 8), so
  // that workgroups running together read different parts of x and spread
  // over the L2 channels instead of all hitting the same lines at once.
  const int ksteps = static_cast<int>(a.K / 64);
  const int z = blockIdx.z;
  const int z_lo = (z * ksteps) / a.ksplit, z_hi = ((z + 1) * ksteps) / a.ksplit;
  const int rw = (wave + static_cast<int>(blockIdx.x + blockIdx.y)) % kSkWaves;
  const int s_lo = z_lo + (rw * (z_hi - z_lo)) / kSkWaves;
  const int s_hi = z_lo + ((rw + 1) * (z_hi - z_lo)) / kSkWaves;
  const u32x4 zero4 = {0u, 0u, 0u, 0u};
  for (int s = s_lo; s < s_hi; s += U) {
    u32x4 wv[U][FN][2], xv[U][FM][2];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int64_t k = static_cast<int64_t>(min(s + u, s_hi - 1)) * 64 + 16 * kgrp;
#pragma unroll
      for (int i = 0; i < FN; ++i) {
        wv[u][i][0] = ld_global<u32x4>(wrow[i] + k);
        wv[u][i][1] = ld_global<u32x4>(wrow[i] + k + 8);
      }
#pragma unroll
      for (int j = 0; j < FM; ++j) {
        xv[u][j][0] = ld_global<u32x4>(xrow[j] + k);
        xv[u][j][1] = ld_global<u32x4>(xrow[j] + k + 8);
      }
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const bool live = s + u < s_hi;
#pragma unroll
      for (int m = 0; m < 2; ++m) {
#pragma unroll
        for (int i = 0; i < FN; ++i) wv[u][i][m] = (live && wok[i]) ? wv[u][i][m] : zero4;
#pragma unroll
        for (int j = 0; j < FM; ++j) xv[u][j][m] = (live && xok[j]) ? xv[u][j][m] : zero4;
#pragma unroll
        for (int i = 0; i < FN; ++i)
#pragma unroll
          for (int j = 0; j < FM; ++j)
            acc[i][j] = mfma16x16x32(as_bf16x8(wv[u][i][m]), as_bf16x8(xv[u][j][m]), acc[i][j]);
      }
    }
  }
  // adapter up-projection: chunks of 32 U_s columns, round-robin over waves
  for (int q = wave; q < n_chunks; q += kSkWaves) {
    const int c = chunks[q] * 32 + 8 * kgrp;
    bf16x8 bv[FN], uv[FM];
#pragma unroll
    for (int i = 0; i < FN; ++i) bv[i] = as_bf16x8(load_btilde(a, present, n0 + 16 * i + col, c));
#pragma unroll
    for (int j = 0; j < FM; ++j) {
      const int64_t t = t0 + 16 * j + col;
      uv[j] = as_bf16x8((t < a.T && c < a.R) ? ld_global<u32x4>(a.us + t * a.R + c)
                                              : u32x4{0u, 0u, 0u, 0u});
    }
#pragma unroll
    for (int i = 0; i < FN; ++i)
#pragma unroll
      for (int j = 0; j < FM; ++j) acc[i][j] = mfma16x16x32(bv[i], uv[j], acc[i][j]);
  }

  // ---- sum the waves' partial tiles in wave order, then store
#pragma unroll
  for (int j = 0; j < FM; ++j)
#pragma unroll
    for (int i = 0; i < FN; ++i) red[((wave * FM + j) * FN + i) * kWave + lane] = acc[i][j];
  __syncthreads();
  for (int e = tid; e < FM * FN * kWave; e += kSkThreads) {
    const int l = e % kWave, i = (e / kWave) % FN, j = e / (kWave * FN);
    f32x4 s = red[e];
    for (int w = 1; w < kSkWaves; ++w) s += red[w * FM * FN * kWave + e];
    store4(a, t0 + 16 * j + l % 16, n0 + 16 * i + 4 * (l / 16), s);
  }
}

// ------------------------------------------------------------- SGMV shrink
// Decode-size shrink, one workgroup per adapter a (segmented by adapter, as
// in SGMV): the tokens routed to a are compacted (ascending) into groups of
// 16 that become the columns of S^T = A_a X_g^T on the matrix cores, with the
// adapter's rank rows as MFMA rows. The 16 waves split K, each issuing the
// loads of U steps before their MFMAs, and their partial tiles are summed
// through LDS in wave order. The workgroup owns U_s columns
// [a*r_max, (a+1)*r_max) for every token: it first zero-fills them, then
// writes bf16(s_t * u) for its tokens and rows below the rank, so every
// adapter's A is read once and no partial sums leave the workgroup.
constexpr int kSgThreads = 1024;
constexpr int kSgWaves = kSgThreads / kWave;
constexpr int kSgMaxTokens = 256;  // decode sizes only
constexpr int kSgMaxTiles = 8;     // r_max <= 128

template <int RT, int U>  // RT 16-row tiles of the rank dimension (r_max <= 16*RT)
__global__ __launch_bounds__(kSgThreads) void lora_sgmv_shrink_kernel(GemmArgs a) {
  __shared__ int toks[kSgMaxTokens];
  __shared__ int wave_cnt[kSgWaves];
  __shared__ f32x4 red[kSgWaves][kWave];
  const int ad = blockIdx.x;
  const int tid = threadIdx.x, wave = tid / kWave, lane = tid % kWave;
  const int col = lane % 16, kgrp = lane / 16;
  const int rk = rank_of(a, ad);

  // zero-fill this adapter's column block for every token
  uint16_t* ublk = a.y + static_cast<int64_t>(ad) * a.r_max;
  for (int64_t e = tid; e < a.T * a.r_max; e += kSgThreads)
    ublk[(e / a.r_max) * a.R + e % a.r_max] = 0;

  // tokens routed to this adapter, ascending (T <= kSgMaxTokens <= threads)
  const int t = tid;
  const bool mine = t < a.T && a.idx[t] == ad;
  const uint64_t m = __ballot(mine);
  if (lane == 0) wave_cnt[wave] = __popcll(m);
  __syncthreads();  // also orders the zero-fill before the value writes below
  int off = 0, n_tok = 0;
  for (int w = 0; w < kSgWaves; ++w) {
    if (w < wave) off += wave_cnt[w];
    n_tok += wave_cnt[w];
  }
  if (mine) toks[off + __popcll(m & ((1ull << lane) - 1ull))] = t;
  __syncthreads();
  if (n_tok == 0 || rk == 0) return;  // uniform: nothing beyond the zero-fill

  const int ksteps = static_cast<int>(a.K / 32);
  const int s_lo = (wave * ksteps) / kSgWaves, s_hi = ((wave + 1) * ksteps) / kSgWaves;
  const int tiles = (rk + 15) / 16;  // uniform: tiles past the rank are skipped
  const uint16_t* abase = a.w + static_cast<int64_t>(ad) * a.r_max * a.K;
  const u32x4 zero4 = {0u, 0u, 0u, 0u};
  for (int g0 = 0; g0 < n_tok; g0 += 16) {
    // this lane's operand rows: rank row (A) and token (B) of each tile
    const uint16_t* arow[RT];
    bool aok[RT];
#pragma unroll
    for (int i = 0; i < RT; ++i) {
      const int j = 16 * i + col;
      aok[i] = j < rk;
      arow[i] = abase + static_cast<int64_t>(aok[i] ? j : 0) * a.K + 8 * kgrp;
    }
    const bool xok = g0 + col < n_tok;
    const uint16_t* xrow = a.x + static_cast<int64_t>(toks[xok ? g0 + col : g0]) * a.K + 8 * kgrp;
    f32x4 acc[RT];
#pragma unroll
    for (int i = 0; i < RT; ++i) acc[i] = f32x4{0.f, 0.f, 0.f, 0.f};
    for (int s0 = s_lo; s0 < s_hi; s0 += U) {
      // steps past s_hi reload the last step and use a zero token operand
      u32x4 xv[U], av[U][RT];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int64_t k = static_cast<int64_t>(min(s0 + u, s_hi - 1)) * 32;
        xv[u] = ld_global<u32x4>(xrow + k);
#pragma unroll
        for (int i = 0; i < RT; ++i)
          av[u][i] = i < tiles ? ld_global<u32x4>(arow[i] + k) : zero4;
      }
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const u32x4 xb = (xok && s0 + u < s_hi) ? xv[u] : zero4;
#pragma unroll
        for (int i = 0; i < RT; ++i)
          if (i < tiles)
            acc[i] = mfma16x16x32(as_bf16x8(aok[i] ? av[u][i] : zero4), as_bf16x8(xb), acc[i]);
      }
    }
    const int slot = g0 + col;
    const int tok = slot < n_tok ? toks[slot] : 0;
    const float sc = slot < n_tok ? a.scale[tok] : 0.f;
#pragma unroll
    for (int i = 0; i < RT; ++i) {
      if (i >= tiles) break;
      red[wave][lane] = acc[i];
      __syncthreads();
      if (wave == 0) {
        f32x4 v = red[0][lane];
        for (int w = 1; w < kSgWaves; ++w) v += red[w][lane];
        if (slot < n_tok) {
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            const int j = 16 * i + 4 * kgrp + q;  // rank row
            if (j < rk) ublk[static_cast<int64_t>(tok) * a.R + j] = f32_to_bf16(sc * v[q]);
          }
        }
      }
      __syncthreads();
    }
  }
}

// ------------------------------------------------------------------ tiled
template <int BM, int BN, int WM, int WN>
__global__ __launch_bounds__(kGemmThreads) void lora_tiled_kernel(GemmArgs a) {
  constexpr int FN = BN / WN / 16;  // 16-row MFMA tiles per wave along features
  constexpr int FM = BM / WM / 16;  // 16-col MFMA tiles per wave along tokens
  constexpr int W_PIECES = BN * (kBK / 8) / kGemmThreads;
  constexpr int X_PIECES = BM * (kBK / 8) / kGemmThreads;
  static_assert(W_PIECES >= 1 && X_PIECES >= 1 && WM * WN == 4, "tile shape");
  extern __shared__ __attribute__((aligned(16))) uint16_t smem[];
  // LDS: W tiles [2][BN][kLdsK], then x tiles [2][BM][kLdsK]
  auto w_lds = [&](int buf) { return smem + buf * (BN * kLdsK); };
  auto x_lds = [&](int buf) { return smem + 2 * BN * kLdsK + buf * (BM * kLdsK); };
  __shared__ uint64_t present[4];
  __shared__ uint16_t chunks[kMaxLoraChunks];
  __shared__ int wave_cnt[4];

  const int tid = threadIdx.x, wave = tid / kWave, lane = tid % kWave;
  const int col = lane % 16, kgrp = lane / 16;

  // ---- tile coordinates (XCD-aware grouped order)
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

  int n_chunks = 0;
  if (a.mode == kModeMain && a.n_ad > 0 && a.us != nullptr)
    n_chunks = lora_chunk_list<kGemmThreads>(a, m0, BM, kBK, present, chunks, wave_cnt);
  const int k_main = static_cast<int>(a.K / kBK);
  const int s_end = k_main + n_chunks;

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
        xreg[i] = t < a.T ? ld_global<u32x4>(a.x + t * a.K + k0 + 8 * kp) : u32x4{0u, 0u, 0u, 0u};
      }
    } else {
      const int c0 = chunks[s - k_main] * kBK;
#pragma unroll
      for (int i = 0; i < W_PIECES; ++i) {
        const int piece = tid + i * kGemmThreads;
        wreg[i] = load_btilde(a, present, n0 + piece / 8, c0 + 8 * (piece % 8));
      }
#pragma unroll
      for (int i = 0; i < X_PIECES; ++i) {
        const int piece = tid + i * kGemmThreads;
        const int64_t t = m0 + piece / 8;
        const int c = c0 + 8 * (piece % 8);
        xreg[i] = (t < a.T && c < a.R) ? ld_global<u32x4>(a.us + t * a.R + c)
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

  load_step(0);
  store_step(0);
  __syncthreads();
  int cur = 0;
  for (int s = 0; s < s_end; ++s) {
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

#pragma unroll
  for (int j = 0; j < FM; ++j)
#pragma unroll
    for (int i = 0; i < FN; ++i)
      store4(a, m0 + wcol0 + 16 * j + col, n0 + wrow0 + 16 * i + 4 * kgrp, acc[i][j]);
}

template <typename Kernel>
void raise_lds_limit(Kernel k, size_t bytes, bool& done) {
  if (!done) {  // benign race: every caller sets the same value
    (void)hipFuncSetAttribute(reinterpret_cast<const void*>(k),
                              hipFuncAttributeMaxDynamicSharedMemorySize,
                              static_cast<int>(bytes));
    done = true;
  }
}

template <int BM, int BN, int WM, int WN>
local_status_t launch_tiled(GemmArgs a, hipStream_t s) {
  a.gm = static_cast<int>((a.T + BM - 1) / BM);
  a.gn = static_cast<int>((a.N + BN - 1) / BN);
  a.swizzle = 1;
  const size_t lds = static_cast<size_t>(2 * (BN + BM) * kLdsK) * sizeof(uint16_t);
  static bool done = false;
  raise_lds_limit(lora_tiled_kernel<BM, BN, WM, WN>, lds, done);
  lora_tiled_kernel<BM, BN, WM, WN><<<a.gm * a.gn, kGemmThreads, lds, s>>>(a);
  return local_check_launch("lora_linear (tiled)");
}

template <int FN, int FM, int U>
local_status_t launch_skinny(GemmArgs a, hipStream_t s) {
  const size_t lds = static_cast<size_t>(kSkWaves) * FM * FN * kWave * sizeof(f32x4);
  static bool done = false;
  raise_lds_limit(lora_skinny_kernel<FN, FM, U>, lds, done);
  dim3 grid(static_cast<unsigned>((a.N + 16 * FN - 1) / (16 * FN)),
            static_cast<unsigned>((a.T + 16 * FM - 1) / (16 * FM)),
            static_cast<unsigned>(a.ksplit));
  lora_skinny_kernel<FN, FM, U><<<grid, kSkThreads, lds, s>>>(a);
  return local_check_launch("lora_linear (skinny)");
}

template <int FN, int FM, int U>
local_status_t launch_skinny_tiles(GemmArgs a, hipStream_t s) {
  a.ksplit = 1;
  return launch_skinny<FN, FM, U>(a, s);
}

local_status_t run_gemm(const GemmArgs& a, hipStream_t s) {
  if (a.mode == kModeMain && a.T > 256) return launch_tiled<128, 128, 2, 2>(a, s);
  // skinny: one token tile of <= 128 rows for decode; 32-row tiles when a
  // shrink covers many tokens, so that enough workgroups run
  if (a.T <= 16) return launch_skinny_tiles<1, 1, 4>(a, s);
  if (a.mode == kModeShrink && a.T > 128) return launch_skinny_tiles<1, 2, LOCAL_SK_U32>(a, s);
  if (a.T <= 32) return launch_skinny_tiles<LOCAL_SK_FN32, 2, LOCAL_SK_U32>(a, s);
  if (a.T <= 64) return launch_skinny_tiles<LOCAL_SK_FN64, 4, 2>(a, s);
  return launch_skinny_tiles<LOCAL_SK_FN128, 8, 2>(a, s);
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
  // workspace: U_s [T][R] bf16
  const size_t need = align256(static_cast<size_t>(T) * R * sizeof(uint16_t));
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
    local_status_t st;
    if (T <= kSgMaxTokens) {  // decode sizes: one workgroup per adapter
      const int rt = (r_max + 15) / 16;
      const unsigned g = static_cast<unsigned>(n_adapters);
      if (rt <= 1) lora_sgmv_shrink_kernel<1, 8><<<g, kSgThreads, 0, s>>>(sh);
      else if (rt <= 2) lora_sgmv_shrink_kernel<2, 4><<<g, kSgThreads, 0, s>>>(sh);
      else if (rt <= 4) lora_sgmv_shrink_kernel<4, 2><<<g, kSgThreads, 0, s>>>(sh);
      else lora_sgmv_shrink_kernel<kSgMaxTiles, 1><<<g, kSgThreads, 0, s>>>(sh);
      st = local_check_launch("lora_linear (SGMV shrink)");
    } else {
      st = run_gemm(sh, s);
    }
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
  m.mode = kModeMain;
  return run_gemm(m, s);
}
