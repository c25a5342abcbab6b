// local_lora_linear: y = res + x W^T + s_t (x A_a^T) B_a^T with a per-token
// adapter a = adapter_idx[t] (§2.2 "LoRA adapters": one frozen base shared by
// many low-rank adapters, every request routed to its own adapter).
//
// Design, SGMV-style but on the matrix cores end to end. Every tile is
// computed transposed, Y^T = W X^T: features are MFMA rows (A operand, rows
// of W), tokens are columns (B operand, rows of x), so a lane ends with 4
// consecutive features of one token.
//
//  * Decode sizes (T <= 256), none waiting on another kernel's workgroups:
//    - base product split over K, streamed: a workgroup owns 16*FN features
//      x up to 128 tokens of one K slice; its W rows (with the shrink's
//      stacked-A rows as extra row tiles when they fit) and x rows stream
//      through an LDS ring by direct global-to-LDS loads, whole 128-byte rows
//      per load instruction; fp32 partial sums per slice. Wider feature
//      tiles for fewer tokens cut the re-reads of x.
//    - SGMV shrink, when the stacked rows are too many to ride along (more
//      than 4 extra row tiles a workgroup): workgroups per (K slice,
//      adapter, projection) gather the
//      tokens routed to that adapter and compute x_t . A[a,j,:] for j below
//      its rank over their slice of K on the matrix cores; fp32 partial sums
//      per slice.
//    - epilogue: sums the base slices, forms U_s = bf16(s_t * u) for the
//      token's own adapter and rank, adds U_s B_a^T and the residual, and
//      rounds once to bf16.
//  * Long prefill chunks (T > 256), two kernels:
//    - shrink: workgroups of 64 tokens x one K slice compute, for each
//      adapter routed in the tile and every projection of the call,
//      x_t . A[a,j,:] of its tokens on the matrix cores; fp32 partial sums
//      per slice.
//    - main product: 128 tokens x 256 features per workgroup, both operands
//      brought to LDS by direct global-to-LDS loads in a three-stage ring;
//      the delta U_s Btilde^T (U_s[t, a*r_max + j] = bf16(s_t * sum of the
//      slices), zero unless a is t's adapter; Btilde[n, a*r_max + j] =
//      B[a, n, j]) runs as extra K-steps, only over adapters used in the tile
//      and columns below their rank.
//  Both paths sum the base K-steps in an order that does not depend on which
//  adapters are present, so a zero up-projection leaves y bit-identical.
#include "common.hpp"
#include "lora_internal.hpp"

namespace localk {
namespace {

constexpr int kMaxGroup = 4;            // projections sharing x in one grouped call
constexpr int kNumXcd = 8;

struct GemmArgs {
  const uint16_t* x;     // [T][K]
  const uint16_t* w;     // main: W [N][K]; shrink: stacked A [R][K]
  int64_t T, K, N;       // N = output width
  float* pout;           // shrink: fp32 partial sums [up_ks][T][p_stride]
  int up_ks;             // K slices of the shrink partial sums
  float* part;           // partial mode: fp32 base partial sums [ksplit][T][N]
  int xrows;             // stacked-A rows per feature-tile workgroup (0 = none)
  // Skinny kernel and epilogue: G projections that share x, taken as one
  // virtual weight whose rows [gstart[g], gstart[g+1]) are the rows of W_g
  // (N = gstart[G]); their stacked A rows are likewise concatenated, R rows
  // per projection.
  int G;
  int64_t gstart[kMaxGroup + 1];
  const uint16_t* gw[kMaxGroup];     // W_g [N_g][K]
  const uint16_t* ga[kMaxGroup];     // A_g [n_ad][r_max][K]
  const uint16_t* gb[kMaxGroup];     // B_g [n_ad][N_g][r_max]
  const int32_t* granks[kMaxGroup];  // ranks_g [n_ad] or null
  const uint16_t* gres[kMaxGroup];   // residual_g [T][N_g] or null
  uint16_t* gy[kMaxGroup];           // y_g [T][N_g]
  int p_stride;          // row length of the shrink partial sums (R or r_max)
  int p_stacked;         // 1: shrink sums indexed by stacked row a*r_max + j
  const int32_t* ranks;  // [n_ad] or null
  const int32_t* idx;    // [T] or null
  const float* scale;    // [T]
  int n_ad, r_max, R;
  const uint16_t* res;   // optional residual [T][N] (main mode)
  uint16_t* y;           // bf16 output [T][N]
  int ksplit;            // K slices of the decode base product (grid.z)
  int gm, gn;            // tile grid of the long-chunk main product
  uint64_t* tile_present;  // long chunks: bitmap of the adapters routed in each
                           // 64-token tile, [ceil(T/64)][4], written by the shrink
};

// Rank of adapter ad, clamped to [0, r_max] so that no rank reads past the
// adapter's own rows.
__device__ __forceinline__ int rank_of(const GemmArgs& a, int ad) {
  return a.ranks ? min(max(a.ranks[ad], 0), a.r_max) : a.r_max;
}

// Entry g of a per-projection argument array. Compare-and-select over the
// array (instead of indexing it) keeps the by-value argument in registers.
template <typename T>
__device__ __forceinline__ T pick(const T (&v)[kMaxGroup], int g) {
  T r = v[0];
#pragma unroll
  for (int i = 1; i < kMaxGroup; ++i) r = g == i ? v[i] : r;
  return r;
}

// Projection of virtual row n of a grouped call.
__device__ __forceinline__ int group_of(const GemmArgs& a, int64_t n) {
  int g = 0;
#pragma unroll
  for (int i = 1; i < kMaxGroup; ++i) g += (i < a.G && n >= a.gstart[i]) ? 1 : 0;
  return g;
}

// First virtual row of projection g (g may be G: the end of the last one).
__device__ __forceinline__ int64_t gstart_of(const GemmArgs& a, int g) {
  int64_t r = a.gstart[0];
#pragma unroll
  for (int i = 1; i <= kMaxGroup; ++i) r = g == i ? a.gstart[i] : r;
  return r;
}

// Rank of adapter ad of projection g, clamped to [0, r_max].
__device__ __forceinline__ int rank_g(const GemmArgs& a, int g, int ad) {
  const int32_t* r = pick(a.granks, g);
  return r ? min(max(r[ad], 0), a.r_max) : a.r_max;
}

// Adapter of token t, or -1 (past the batch, no adapter, or out of range).
__device__ __forceinline__ int token_adapter(const GemmArgs& a, int64_t t) {
  if (t >= a.T) return -1;
  const int ad = a.idx[t];
  return (ad >= 0 && ad < a.n_ad) ? ad : -1;
}

// s_waitcnt encodings (gfx9 layout): wait until at most N vector memory
// operations are outstanding / until all LDS operations are done.
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

// The first `keep` (clamped to 0..8) of 8 packed bf16 values; the rest zero.
__device__ __forceinline__ u32x4 keep_first8(u32x4 v, int keep) {
  uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
  for (int e = 0; e < 8; ++e)
    if (e >= keep) w[e / 2] &= (e & 1) ? 0x0000ffffu : 0xffff0000u;
  return u32x4{w[0], w[1], w[2], w[3]};
}



// Direct global-to-LDS load of 16 bytes per lane: lane l's bytes land at
// lds + 16 l (lds is the wave's common base). A plain function: the builtin
// called with template-dependent arguments fails the host compilation pass
// of a kernel template.
__device__ __forceinline__ void lds_load16(const void* g, void* lds) {
  __builtin_amdgcn_global_load_lds(g, lds, 16, 0, 0);
}

// ------------------------------------------------------------------ stream
// Decode sizes (T <= 256): the base product, with the shrink's stacked-A rows
// as extra row tiles, of one K slice, streamed through LDS. Workgroup:
// features [n0, n0 + 16 FN) (+ XT tiles of stacked-A rows) x tokens
// [t0, t0 + 16 FM) over the z-th of ksplit K slices. Each 64-k step of the
// slice is one LDS stage holding the tile's W and A rows and its x rows
// (128-byte rows, chunk-swizzled as in the long-chunk product), brought in
// by direct global-to-LDS loads: every load instruction moves 8 whole rows,
// and a ring of S stages keeps S - 2 steps in flight while one is computed.
// Each wave owns every fourth output tile, so there is no reduction across
// waves. Rows past N or T and stacked-A rows past the adapter's rank read
// clamped rows; their outputs are never stored (rows past the rank are
// masked by the epilogue). Workgroups start their slice at different steps
// (by feature tile), so that those running together read different parts
// of x; the order depends on the feature tile only, as with the K slices.
constexpr int kStThreads = 256;
constexpr int kStWaves = kStThreads / kWave;
constexpr int kStLdsMax = 147456;

template <int FN, int FM, int XT>
struct StreamShape {
  static constexpr int FT = FN + XT;                                // W and A row tiles
  static constexpr int ROWS = 16 * (FT + FM);                       // rows of a stage
  static constexpr int DMA = (ROWS / 8 + kStWaves - 1) / kStWaves;  // loads per wave and stage
  static constexpr int STAGE = 8 * DMA * kStWaves * 128;            // bytes, padded
  static constexpr int S = kStLdsMax / STAGE < 8 ? kStLdsMax / STAGE : 8;
  static constexpr int NT = (FT * FM + kStWaves - 1) / kStWaves;    // tiles per wave
  static_assert(S >= 3 && DMA * (S - 2) < 64, "stream ring");
};

template <int FN, int FM, int XT>
__global__ __launch_bounds__(kStThreads) void lora_stream_kernel(GemmArgs a) {
  using SS = StreamShape<FN, FM, XT>;
  constexpr int FT = SS::FT, S = SS::S, D = SS::DMA, NT = SS::NT;
  extern __shared__ __attribute__((aligned(16))) uint8_t st_lds[];

  const int tid = threadIdx.x, lane = tid % kWave;
  const int wave = __builtin_amdgcn_readfirstlane(tid / kWave);
  const int col = lane % 16, kgrp = lane / 16;
  const int64_t n0 = static_cast<int64_t>(blockIdx.x) * 16 * FN;
  const int64_t t0 = static_cast<int64_t>(blockIdx.y) * 16 * FM;
  const int64_t x0 = static_cast<int64_t>(blockIdx.x) * a.xrows;  // first stacked-A row
  const int z = blockIdx.z;
  const int ksteps = static_cast<int>(a.K / 64);
  const int z_lo = (z * ksteps) / a.ksplit, z_hi = ((z + 1) * ksteps) / a.ksplit;
  const int nsteps = z_hi - z_lo;
  const int rot = static_cast<int>(blockIdx.x % static_cast<unsigned>(nsteps));

  // the lane's rows of its loads: stage row 8 (wave + 4q) + lane/8
  const int dchunk = (lane % 8) ^ (lane / 8);
  const uint16_t* src[D];
#pragma unroll
  for (int q = 0; q < D; ++q) {
    const int r = 8 * (wave + kStWaves * q) + lane / 8;
    const uint16_t* p;
    if (r < 16 * FN) {  // W row (a 16-row tile lies in one projection)
      const int g = group_of(a, n0 + 16 * (r / 16));
      const int64_t n = n0 + r;
      p = pick(a.gw, g) + (n < a.N ? n - gstart_of(a, g) : 0) * a.K;
    } else if (r < 16 * FT) {  // stacked-A row
      const int64_t row = x0 + (r - 16 * FN);
      const bool ok = r - 16 * FN < a.xrows && row < static_cast<int64_t>(a.G) * a.R;
      const int g = ok ? static_cast<int>(row / a.R) : 0;
      p = pick(a.ga, g) + (ok ? row % a.R : 0) * a.K;
    } else {  // x row (also the padding rows, never read)
      const int64_t t = t0 + (r < 16 * (FT + FM) ? r - 16 * FT : 0);
      p = a.x + (t < a.T ? t : t0) * a.K;
    }
    src[q] = p + 8 * dchunk;
  }
  // k offset of relative step rs (rotated, clamped into the slice)
  auto step_k = [&](int rs) {
    int as = rs < nsteps ? rs + rot : rot;
    as = z_lo + (as >= nsteps ? as - nsteps : as);
    return static_cast<int64_t>(as) * 64;
  };

  // this wave's tiles (past the last tile: the last tile again, not stored)
  int woff[NT], xoff[NT];
#pragma unroll
  for (int k = 0; k < NT; ++k) {
    const int tl = min(wave + kStWaves * k, FT * FM - 1);
    woff[k] = 16 * (tl / FM) * 128;
    xoff[k] = 16 * (FT + tl % FM) * 128;
  }
  const int rd0 = col * 128 + 16 * (kgrp ^ (col % 8));  // chunk kgrp of row col
  const int rd1 = rd0 ^ 64;                              // chunk 4 + kgrp
  f32x4 acc[NT];
#pragma unroll
  for (int k = 0; k < NT; ++k) acc[k] = f32x4{0.f, 0.f, 0.f, 0.f};

  // Step rs: each wave waits for its own loads of stage rs % S (those of the
  // S - 2 later steps may stay in flight); after the barrier every wave's
  // loads of the step are visible and stage (rs - 1) % S is free for the
  // loads of step rs + S - 1.
#pragma unroll
  for (int p = 0; p < S - 1; ++p) {
    const int64_t k = step_k(p);
#pragma unroll
    for (int q = 0; q < D; ++q)
      lds_load16(src[q] + k, st_lds + p * SS::STAGE + 8 * (wave + kStWaves * q) * 128);
  }
  for (int rs = 0; rs < nsteps; ++rs) {
    const int cur = rs % S;
    wait_vmcnt<D * (S - 2)>();
    wait_lgkm0_barrier();
    {
      const int64_t k = step_k(rs + S - 1);
      uint8_t* st = st_lds + (cur == 0 ? S - 1 : cur - 1) * SS::STAGE;
#pragma unroll
      for (int q = 0; q < D; ++q)
        lds_load16(src[q] + k, st + 8 * (wave + kStWaves * q) * 128);
    }
    const uint8_t* st = st_lds + cur * SS::STAGE;
    u32x4 wv[2][NT], xv[2][NT];
#pragma unroll
    for (int m = 0; m < 2; ++m)
#pragma unroll
      for (int k = 0; k < NT; ++k) {
        wv[m][k] = *reinterpret_cast<const u32x4*>(st + woff[k] + (m ? rd1 : rd0));
        xv[m][k] = *reinterpret_cast<const u32x4*>(st + xoff[k] + (m ? rd1 : rd0));
      }
#pragma unroll
    for (int m = 0; m < 2; ++m)
#pragma unroll
      for (int k = 0; k < NT; ++k)
        acc[k] = mfma16x16x32(as_bf16x8(wv[m][k]), as_bf16x8(xv[m][k]), acc[k]);
  }
  wait_vmcnt<0>();

  // partial sums of the slice: lane holds rows 4 (l/16) .. +4 of tile row i,
  // token column l % 16 of tile j
#pragma unroll
  for (int k = 0; k < NT; ++k) {
    const int tl = wave + kStWaves * k;
    if (tl >= FT * FM) continue;
    const int i = tl / FM, j = tl % FM;
    const int64_t t = t0 + 16 * j + col;
    if (t >= a.T) continue;
    if (i >= FN) {  // stacked-A rows: the shrink's partial sums of this slice
      const int rr = 16 * (i - FN) + 4 * kgrp;
      const int64_t rows = static_cast<int64_t>(a.G) * a.R;
      float* dst = a.pout + (static_cast<int64_t>(z) * a.T + t) * rows + x0 + rr;
#pragma unroll
      for (int q = 0; q < 4; ++q)
        if (rr + q < a.xrows && x0 + rr + q < rows) dst[q] = acc[k][q];
      continue;
    }
    const int64_t n = n0 + 16 * i + 4 * kgrp;
    if (n < a.N)
      *reinterpret_cast<f32x4*>(a.part + (static_cast<int64_t>(z) * a.T + t) * a.N + n) = acc[k];
  }
}

// ------------------------------------------------------------- SGMV shrink
// Decode-size shrink, segmented by adapter as in SGMV. Workgroup (z, a, g)
// takes adapter a of projection g and the z-th of up_ks slices of K: the tokens routed to a are
// compacted (ascending) into groups of 16 that become the columns of
// S^T = A_a X_g^T on the matrix cores, with the adapter's rank rows as MFMA
// rows. Each of the 4 waves holds at most U steps of 32 k, so it loads its
// whole slice of A before it even knows the tokens; the waves' partial tiles
// are summed through LDS in wave order. The result, the unscaled fp32 partial
// sum of slice z, goes to P[z][t][j] for the adapter's tokens t and rows
// j < rank; the main kernel sums the slices in order, scales and rounds.
constexpr int kSgThreads = 256;
constexpr int kSgWaves = kSgThreads / kWave;
constexpr int kSgMaxTokens = 256;  // decode sizes only (one token per thread)
constexpr int kSgMaxTiles = 8;     // r_max <= 128

#ifndef LOCAL_SG_U1
#define LOCAL_SG_U1 4  // K-steps of 32 per wave when r_max <= 16
#endif

template <int RT, int U>  // RT 16-row tiles of the rank dimension (r_max <= 16*RT)
__global__ __launch_bounds__(kSgThreads) void lora_sgmv_shrink_kernel(GemmArgs a) {
  __shared__ int toks[kSgMaxTokens];
  __shared__ int wave_cnt[kSgWaves];
  __shared__ f32x4 red[kSgWaves][RT][kWave];
  const int z = blockIdx.x, ad = blockIdx.y, g = blockIdx.z;  // slice, adapter, projection
  const int tid = threadIdx.x, wave = tid / kWave, lane = tid % kWave;
  const int col = lane % 16, kgrp = lane / 16;
  const int rk = rank_g(a, g, ad);
  if (rk == 0) return;  // uniform: no row of this adapter is used
  const int tiles = (rk + 15) / 16;

  // this wave's steps: [s_lo, s_hi) of 32 k, at most U of them
  const int ksteps = static_cast<int>(a.K / 32);
  const int z_lo = (z * ksteps) / a.up_ks, z_hi = ((z + 1) * ksteps) / a.up_ks;
  const int s_lo = z_lo + (wave * (z_hi - z_lo)) / kSgWaves;
  const int s_hi = z_lo + ((wave + 1) * (z_hi - z_lo)) / kSgWaves;
  const u32x4 zero4 = {0u, 0u, 0u, 0u};

  // A: rank rows 16i + col of the slice, loaded first (rows past the rank
  // read row 0 and are zeroed; steps past s_hi read a valid step and are
  // dropped below)
  const uint16_t* abase = pick(a.ga, g) + static_cast<int64_t>(ad) * a.r_max * a.K + 8 * kgrp;
  bool aok[RT];
  u32x4 av[U][RT];
#pragma unroll
  for (int i = 0; i < RT; ++i) aok[i] = 16 * i + col < rk;
#pragma unroll
  for (int u = 0; u < U; ++u) {
    const int64_t k = static_cast<int64_t>(max(min(s_lo + u, s_hi - 1), 0)) * 32;
#pragma unroll
    for (int i = 0; i < RT; ++i) {
      const int64_t row = aok[i] ? 16 * i + col : 0;
      av[u][i] = i < tiles ? ld_global<u32x4>(abase + row * a.K + k) : zero4;
    }
  }

  // tokens routed to this adapter, ascending
  const bool mine = token_adapter(a, tid) == ad;
  const uint64_t m = __ballot(mine);
  if (lane == 0) wave_cnt[wave] = __popcll(m);
  __syncthreads();
  int off = 0, n_tok = 0;
  for (int w = 0; w < kSgWaves; ++w) {
    if (w < wave) off += wave_cnt[w];
    n_tok += wave_cnt[w];
  }
  if (mine) toks[off + __popcll(m & ((1ull << lane) - 1ull))] = tid;
  __syncthreads();

#pragma unroll
  for (int u = 0; u < U; ++u)
#pragma unroll
    for (int i = 0; i < RT; ++i) av[u][i] = (aok[i] && s_lo + u < s_hi) ? av[u][i] : zero4;

  float* pz = a.pout + static_cast<int64_t>(z) * a.T * a.p_stride + g * a.r_max;
  for (int g0 = 0; g0 < n_tok; g0 += 16) {
    const bool xok = g0 + col < n_tok;
    const uint16_t* xrow = a.x + static_cast<int64_t>(toks[xok ? g0 + col : g0]) * a.K + 8 * kgrp;
    u32x4 xv[U];
#pragma unroll
    for (int u = 0; u < U; ++u)
      xv[u] = ld_global<u32x4>(xrow + static_cast<int64_t>(max(min(s_lo + u, s_hi - 1), 0)) * 32);
    f32x4 acc[RT];
#pragma unroll
    for (int i = 0; i < RT; ++i) acc[i] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const u32x4 xb = xok ? xv[u] : zero4;
#pragma unroll
      for (int i = 0; i < RT; ++i)
        if (i < tiles) acc[i] = mfma16x16x32(as_bf16x8(av[u][i]), as_bf16x8(xb), acc[i]);
    }
#pragma unroll
    for (int i = 0; i < RT; ++i) red[wave][i][lane] = acc[i];
    __syncthreads();
    for (int e = tid; e < tiles * kWave; e += kSgThreads) {
      const int i = e / kWave, l = e % kWave;
      f32x4 v = red[0][i][l];
#pragma unroll
      for (int w = 1; w < kSgWaves; ++w) v += red[w][i][l];
      const int slot = g0 + l % 16;
      const int j = 16 * i + 4 * (l / 16);  // first of 4 rank rows
      if (slot < n_tok && j < rk) {
        float* dst = pz + static_cast<int64_t>(toks[slot]) * a.p_stride + j;
        if (j + 4 <= rk) {
          *reinterpret_cast<f32x4*>(dst) = v;
        } else {
          for (int q = 0; j + q < rk; ++q) dst[q] = v[q];
        }
      }
    }
    __syncthreads();
  }
}

// Launch of the SGMV shrink: U steps per wave for the rank tiles, K cut into
// enough slices that no wave has more than U steps.
template <int RT, int U>
local_status_t launch_sgmv_shrink(GemmArgs a, hipStream_t s) {
  lora_sgmv_shrink_kernel<RT, U><<<dim3(static_cast<unsigned>(a.up_ks), static_cast<unsigned>(a.n_ad),
                                        static_cast<unsigned>(a.G)),
                                   kSgThreads, 0, s>>>(a);
  return local_check_launch("lora_linear (SGMV shrink)");
}

// Steps per wave of the SGMV shrink for a given r_max.
int sgmv_steps_per_wave(int r_max) {
  const int rt = (r_max + 15) / 16;
  return rt <= 1 ? LOCAL_SG_U1 : rt <= 2 ? 8 : rt <= 4 ? 4 : 2;
}

// K slices of the SGMV shrink.
int sgmv_slices(int64_t K, int r_max) {
  const int64_t steps = K / 32;
  const int64_t per = static_cast<int64_t>(kSgWaves) * sgmv_steps_per_wave(r_max);
  return static_cast<int>((steps + per - 1) / per);
}

local_status_t run_sgmv_shrink(const GemmArgs& a, hipStream_t s) {
  const int rt = (a.r_max + 15) / 16;
  const int u = sgmv_steps_per_wave(a.r_max);
  if (rt <= 1 && u == 4) return launch_sgmv_shrink<1, 4>(a, s);
  if (rt <= 1) return launch_sgmv_shrink<1, 8>(a, s);
  if (rt <= 2) return launch_sgmv_shrink<2, 8>(a, s);
  if (rt <= 4) return launch_sgmv_shrink<4, 4>(a, s);
  return launch_sgmv_shrink<kSgMaxTiles, 2>(a, s);
}

// --------------------------------------------------------------- epilogue
// Decode sizes, after the base partial sums and the shrink:
//   y[t, n] = bf16( sum_z part[z][t][n] + sum_j U_s[t][j] B[a_t][n][j] + res[t][n] )
// with U_s[t][j] = bf16(s_t * sum_z P[z][t][c]) for j < rank(a_t), both sums
// in slice order; c = a_t*r_max + j when the shrink ran fused with the base
// product (sums for every stacked row), c = j after the SGMV shrink. Workgroup: 16 tokens x 64 features; U_s of its tokens is
// built once in LDS, then each thread finishes 4 consecutive features of one
// token (16-byte partial loads, an 8-byte store).
constexpr int kEpThreads = 256;
constexpr int kEpTokens = 16;
constexpr int kEpFeatures = 64;

template <int KSB>
__global__ __launch_bounds__(kEpThreads) void lora_epilogue_kernel(GemmArgs a) {
  __shared__ float us[kEpTokens][128 + 1];
  const int tid = threadIdx.x;
  const int tt = tid / (kEpFeatures / 4), ng = tid % (kEpFeatures / 4);
  const int64_t t0 = static_cast<int64_t>(blockIdx.y) * kEpTokens;
  const int64_t nv0 = static_cast<int64_t>(blockIdx.x) * kEpFeatures;  // virtual row
  const int64_t t = t0 + tt, nv = nv0 + 4 * ng;
  const bool live = t < a.T && nv < a.N;
  const bool lora = a.n_ad > 0;  // uniform
  const u32x4 zero4 = {0u, 0u, 0u, 0u};
  // the tile's projection (a 64-row tile lies in one) and its own row index
  const int g = group_of(a, nv0);
  const int64_t Ng = gstart_of(a, g + 1) - gstart_of(a, g);
  const int64_t n = nv - gstart_of(a, g);

  // Every load that needs no other load's result is issued first: the base
  // slices, the residual, this token's adapter; then, needing only the
  // adapter, the first 32 rank columns of its B rows and the shrink slices.
  f32x4 pv[KSB];
#pragma unroll
  for (int z = 0; z < KSB; ++z)
    pv[z] = live ? ld_global<f32x4>(a.part + (static_cast<int64_t>(z) * a.T + t) * a.N + nv)
                 : f32x4{0.f, 0.f, 0.f, 0.f};
  const uint16_t* res = pick(a.gres, g);
  u32x2 rv = {0u, 0u};
  if (live && res) rv = ld_global<u32x2>(res + t * Ng + n);
  const int my_ad = (lora && live) ? token_adapter(a, t) : -1;
  const uint16_t* brow =
      pick(a.gb, g) + (static_cast<int64_t>(my_ad >= 0 ? my_ad : 0) * Ng + n) * a.r_max;
  u32x4 bv[4][4];  // [8-column step][feature]
  if (my_ad >= 0) {
#pragma unroll
    for (int js = 0; js < 4; ++js)
#pragma unroll
      for (int i = 0; i < 4; ++i)
        bv[js][i] = 8 * js < a.r_max ? ld_global<u32x4>(brow + i * a.r_max + 8 * js) : zero4;
  }

  f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int z = 0; z < KSB; ++z) acc += pv[z];

  if (lora) {
    // U_s of the tile's tokens, 4 rank rows per item: bf16(s_t * u), u the
    // sum of the shrink slices in slice order (batches of 8 loads)
    const int quads = a.r_max / 4;
    const int64_t slice = a.T * a.p_stride;
    for (int e = tid; e < kEpTokens * quads; e += kEpThreads) {
      const int et = e / quads, j = 4 * (e % quads);
      const int ad = token_adapter(a, t0 + et);
      f32x4 u = {0.f, 0.f, 0.f, 0.f};
      if (ad >= 0) {
        const float sc = a.scale[t0 + et];
        const int rk = rank_g(a, g, ad);
        const float* p = a.pout + (t0 + et) * a.p_stride +
                         (a.p_stacked ? static_cast<int64_t>(g) * a.R + ad * a.r_max
                                      : static_cast<int64_t>(g) * a.r_max) + j;
        for (int z0 = 0; z0 < a.up_ks; z0 += 8) {
          f32x4 sv[8];
#pragma unroll
          for (int zz = 0; zz < 8; ++zz)
            sv[zz] = z0 + zz < a.up_ks ? ld_global<f32x4>(p + (z0 + zz) * slice)
                                       : f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
          for (int zz = 0; zz < 8; ++zz) u += sv[zz];
        }
#pragma unroll
        for (int q = 0; q < 4; ++q)  // rows at or past the rank are never written
          u[q] = j + q < rk ? bf16_to_f32(f32_to_bf16(sc * u[q])) : 0.f;
      }
#pragma unroll
      for (int q = 0; q < 4; ++q) us[et][j + q] = u[q];
    }
    __syncthreads();
    if (my_ad >= 0) {
      // delta of 4 features over the rank columns, 32 at a time
      const int rk = rank_g(a, g, my_ad);
      for (int j0 = 0; j0 < rk; j0 += 32) {
        if (j0 > 0) {
#pragma unroll
          for (int js = 0; js < 4; ++js)
#pragma unroll
            for (int i = 0; i < 4; ++i)
              bv[js][i] = j0 + 8 * js < rk ? ld_global<u32x4>(brow + i * a.r_max + j0 + 8 * js)
                                           : zero4;
        }
#pragma unroll
        for (int js = 0; js < 4; ++js)
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            const int j = j0 + 8 * js + e;
            if (j < rk) {  // columns at or past the rank are never used
              const float u = us[tt][j];
#pragma unroll
              for (int i = 0; i < 4; ++i) {
                const uint32_t w = bv[js][i][e / 2];
                acc[i] += u * __uint_as_float((e & 1) ? (w & 0xffff0000u) : (w << 16));
              }
            }
          }
      }
    }
  }
  if (!live) return;
  if (res) {
    acc[0] += __uint_as_float(rv.x << 16);
    acc[1] += __uint_as_float(rv.x & 0xffff0000u);
    acc[2] += __uint_as_float(rv.y << 16);
    acc[3] += __uint_as_float(rv.y & 0xffff0000u);
  }
  *reinterpret_cast<u32x2*>(pick(a.gy, g) + t * Ng + n) =
      u32x2{pack_bf16x2(acc[0], acc[1]), pack_bf16x2(acc[2], acc[3])};
}

template <int KSB>
local_status_t launch_epilogue(const GemmArgs& a, hipStream_t s) {
  dim3 grid(static_cast<unsigned>((a.N + kEpFeatures - 1) / kEpFeatures),
            static_cast<unsigned>((a.T + kEpTokens - 1) / kEpTokens));
  lora_epilogue_kernel<KSB><<<grid, kEpThreads, 0, s>>>(a);
  return local_check_launch("lora_linear (epilogue)");
}

local_status_t run_epilogue(const GemmArgs& a, hipStream_t s) {
  switch (a.ksplit) {
    case 1: return launch_epilogue<1>(a, s);
    case 2: return launch_epilogue<2>(a, s);
    case 4: return launch_epilogue<4>(a, s);
    case 8: return launch_epilogue<8>(a, s);
    default: return launch_epilogue<16>(a, s);
  }
}

// ----------------------------------------------------------------- prefill
// Long chunks (T > 256), the fused main product. Workgroup: tokens
// [m0, m0 + 128) x features [n0, n0 + 256); wave w owns features
// n0 + 64w .. +64 for all 128 tokens (4 x 8 MFMA tiles, 128 fp32 accumulators
// per lane). Both operands reach LDS by direct global-to-LDS loads (no
// staging registers, no LDS store instructions): a K-step of 64 is one 48 KB
// stage (x: 128 rows, W: 256 rows, 128 bytes each), three stages in a ring,
// so the loads of step s + 2 are in flight while step s computes. Each load
// instruction moves 8 whole 128-byte rows (64 lanes x 16 bytes), so the
// vector memory path sees fully used lines. Inside a row the eight 16-byte
// chunks are stored XOR-swizzled by the row index (chunk c of row r at
// position c ^ (r % 8)): the MFMA operand reads (16 rows, one chunk column)
// then touch distinct banks. The loads name their own waits (the library
// waits on the load counter itself before each barrier). The LoRA delta
// follows as extra K-steps over the U_s columns of the adapters used in the
// token tile.
constexpr int kPfM = 128;
constexpr int kPfN = 256;
#ifndef LOCAL_PF_WM
#define LOCAL_PF_WM 2      // waves along tokens (x 4 along features)
#endif
constexpr int kPfWM = LOCAL_PF_WM;
constexpr int kPfWN = 4;
constexpr int kPfWaves = kPfWM * kPfWN;
constexpr int kPfThreads = kPfWaves * kWave;
constexpr int kPfFT = kPfN / kPfWN / 16;   // 16-feature MFMA tiles per wave (4)
constexpr int kPfTT = kPfM / kPfWM / 16;   // 16-token MFMA tiles per wave
constexpr int kPfRow = 128;                       // bytes of one row of a stage
constexpr int kPfXBytes = kPfM * kPfRow;          // 16 KB
constexpr int kPfStageBytes = (kPfM + kPfN) * kPfRow;  // 48 KB
constexpr int kPfStages = 3;
constexpr int kPfURow = 80;                       // bytes of a U_s tile row: 32 bf16 + pad
constexpr int kPfUBytes = kPfM * kPfURow;         // 10 KB
constexpr int kPfLdsBytes = kPfStages * kPfStageBytes + kPfUBytes;  // 154 KB
constexpr int kPfOutRow = kPfN * 4 + 16;          // bytes of a token row of the output tile
static_assert(kPfM * kPfOutRow <= kPfLdsBytes, "output tile in LDS");
constexpr int kPfXDma = kPfM / 8 / kPfWaves;      // 1 KB loads of x per wave and step
constexpr int kPfWDma = kPfN / 8 / kPfWaves;      // ... of W
constexpr int kPfDma = kPfXDma + kPfWDma;
constexpr int kPfMfma = kPfFT * kPfTT;            // MFMAs per wave and half step

__global__ __launch_bounds__(kPfThreads, 1) void lora_prefill_kernel(GemmArgs a) {
  extern __shared__ __attribute__((aligned(16))) uint8_t pf_lds[];

  const int tid = threadIdx.x, lane = tid % kWave;
  const int wave = __builtin_amdgcn_readfirstlane(tid / kWave);  // uniform: LDS bases in SGPRs
  const int col = lane % 16, kgrp = lane / 16;

  // ---- tile coordinates: XCD-aware grouped order (the blocks of one XCD
  // take an 8-tall column of tiles, so its L2 serves x and W rows in common)
  int mt, nt;
  {
    const int id = blockIdx.x;
    const int total = a.gm * a.gn;
    int lid = id;
    if (total % kNumXcd == 0) lid = (id % kNumXcd) * (total / kNumXcd) + id / kNumXcd;
    constexpr int GM = 8;
    const int group = lid / (GM * a.gn);
    const int first_m = group * GM;
    const int gsize = min(a.gm - first_m, GM);
    const int r = lid % (GM * a.gn);
    mt = first_m + r % gsize;
    nt = r / gsize;
  }
  const int64_t m0 = static_cast<int64_t>(mt) * kPfM;
  const int64_t n0 = static_cast<int64_t>(nt) * kPfN;
  // projection of the tile (a 256-feature tile lies in one projection) and
  // its operands; feature indices below are virtual rows n0 + ...
  const int gq = group_of(a, n0);
  const int64_t gbase = gstart_of(a, gq), Ng = gstart_of(a, gq + 1) - gbase;
  const uint16_t* Wg = pick(a.gw, gq);
  const uint16_t* Bg = pick(a.gb, gq);
  const int32_t* ranksg = pick(a.granks, gq);
  const float* Pg = a.pout ? a.pout + static_cast<int64_t>(gq) * a.up_ks * a.T * a.r_max : nullptr;
  const int wm = wave / kPfWN, wn = wave % kPfWN;
  const int64_t fw0 = n0 + 16 * kPfFT * wn;  // this wave's first feature
  const int tw0 = 16 * kPfTT * wm;           // ... and first token of the tile

  const bool lora = a.n_ad > 0 && Pg != nullptr && a.tile_present != nullptr;  // uniform

  // ---- direct loads. Wave w moves x rows 32w .. +32 and W rows 64w .. +64
  // (its own features) of every stage; lane l writes 16 bytes at
  // block + 16 l, i.e. row 8q + l/8, position l%8, which holds chunk
  // (l%8) ^ (l/8) of that row. Rows past T (N) repeat row m0 (row 0): their
  // accumulators are never stored.
  const int dchunk = (lane % 8) ^ (lane / 8);
  const uint16_t* xg[kPfXDma];
  const uint16_t* wg[kPfWDma];
#pragma unroll
  for (int q = 0; q < kPfXDma; ++q) {
    const int64_t t = m0 + (kPfM / kPfWaves) * wave + 8 * q + lane / 8;
    xg[q] = a.x + (t < a.T ? t : m0) * a.K + 8 * dchunk;
  }
#pragma unroll
  for (int q = 0; q < kPfWDma; ++q) {
    const int64_t nl = n0 - gbase + (kPfN / kPfWaves) * wave + 8 * q + lane / 8;
    wg[q] = Wg + (nl < Ng ? nl : 0) * a.K + 8 * dchunk;
  }
  // loads of K-step s into stage `stage`
  auto issue = [&](int stage, int s) {
    uint8_t* st = pf_lds + stage * kPfStageBytes;
    const int64_t k = static_cast<int64_t>(s) * 64;
#pragma unroll
    for (int q = 0; q < kPfXDma; ++q)
      __builtin_amdgcn_global_load_lds(xg[q] + k, st + ((kPfM / kPfWaves) * wave + 8 * q) * kPfRow,
                                       16, 0, 0);
#pragma unroll
    for (int q = 0; q < kPfWDma; ++q)
      __builtin_amdgcn_global_load_lds(
          wg[q] + k, st + kPfXBytes + ((kPfN / kPfWaves) * wave + 8 * q) * kPfRow, 16, 0, 0);
  };

  f32x4 acc[kPfFT][kPfTT];
#pragma unroll
  for (int i = 0; i < kPfFT; ++i)
#pragma unroll
    for (int j = 0; j < kPfTT; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  // MFMA operand reads. K-group g of MFMA m holds k = 32m + 8g .. +8 of the
  // step (chunk 4m + g), the same for W and x; chunk c of row r sits at
  // position c ^ (r % 8), and r % 8 = col % 8 for every row a lane reads.
  const int rd0 = col * kPfRow + 16 * (kgrp ^ (col % 8));  // chunk kgrp
  const int rd1 = rd0 ^ 64;                                 // chunk 4 + kgrp
  u32x4 xf[2][kPfTT], wf[2][kPfFT];
  auto read_half = [&](int stage, int m) {
    const uint8_t* st = pf_lds + stage * kPfStageBytes + (m ? rd1 : rd0);
#pragma unroll
    for (int i = 0; i < kPfFT; ++i)
      wf[m][i] = *reinterpret_cast<const u32x4*>(st + kPfXBytes + (16 * kPfFT * wn + 16 * i) * kPfRow);
#pragma unroll
    for (int j = 0; j < kPfTT; ++j)
      xf[m][j] = *reinterpret_cast<const u32x4*>(st + (tw0 + 16 * j) * kPfRow);
  };
  // MFMAs [b, e) of half m, in the order tile (i, j) = (idx / TT, idx % TT)
  auto mfma_range = [&](int m, int b, int e) {
#pragma unroll
    for (int idx = b; idx < e; ++idx) {
      const int i = idx / kPfTT, j = idx % kPfTT;
      acc[i][j] = mfma16x16x32(as_bf16x8(wf[m][i]), as_bf16x8(xf[m][j]), acc[i][j]);
    }
  };
  // instruction-group masks of the scheduler's group barriers, and the
  // group sizes of a step: R operand reads per half, Q MFMAs of the second
  // half before the barrier, the loads paired with MFMAs after the reads
  constexpr int kSgMfma = 0x8, kSgVmem = 0x10, kSgDsRead = 0x100;
  constexpr int kR = kPfFT + kPfTT, kQ = kPfMfma / 4;
  constexpr int kVPair = kPfDma < kPfMfma - kQ - kR ? kPfDma : kPfMfma - kQ - kR;
  static_assert(kPfMfma - kQ >= kR && kVPair >= 0, "step schedule");

  // Step s (stage s % 3), first half: the m = 1 operands are read under the
  // m = 0 MFMAs. Then each wave waits for its own loads of step s + 1 (those
  // of step s + 2 may stay in flight) and for its reads of stage s % 3; after
  // the barrier every wave's loads of step s + 1 are visible and stage s % 3
  // is free, so the loads of step s + 3 refill it. Second half: the m = 0
  // operands of step s + 1 are read under the m = 1 MFMAs of step s. The
  // body has no branch (a branch between the two halves makes the compiler
  // copy the 128 accumulators around it): past the last step the loads
  // repeat the last step into the free stage and the reads fetch operands
  // that are never used, so every wait count holds at every step.
  const int steps = static_cast<int>(a.K / 64);
  const int last = steps - 1;
  // the first three stages' loads go out before anything else waits
  issue(0, 0);
  issue(1, min(1, last));
  issue(2, min(2, last));

  // ---- LoRA delta first, chunk by chunk (32 stacked columns
  // c = a*r_max + j): U_s[t][c] = bf16(s_t * sum_z P[z][t][j]) (slices in
  // order) when a is token t's adapter, else 0, formed by the whole
  // workgroup into an LDS tile; Btilde is zero at or past the rank. Its
  // chain of loads runs while the first stages load. Adding the delta first
  // leaves a zero up-projection's result bit-identical (the MFMAs add +0).
  // The adapters routed in the tile come from the bitmaps the shrink wrote
  // for its two 64-token tiles, read by scalar loads, which do not wait for
  // the stage loads.
  uint64_t pm[4] = {0ull, 0ull, 0ull, 0ull};
  if (lora) {
    const int n64 = static_cast<int>((a.T + 63) / 64);
    using const_u64 = const __attribute__((address_space(4))) uint64_t;  // scalar loads
    const_u64* tp = (const_u64*)a.tile_present;
#pragma unroll
    for (int h = 0; h < 2; ++h)
      if (2 * mt + h < n64)
#pragma unroll
        for (int w = 0; w < 4; ++w) pm[w] |= tp[4 * (2 * mt + h) + w];
  }
  // the first chunk after chunk c that covers a routed adapter, or -1
  auto next_chunk = [&](int c) {
    const int amin = ((c + 1) * 32) / a.r_max;  // adapters with columns past chunk c
    int found = -1;
#pragma unroll
    for (int w = 3; w >= 0; --w) {
      uint64_t m = pm[w];
      if (64 * w + 63 < amin)
        m = 0ull;
      else if (64 * w < amin)
        m &= ~0ull << (amin - 64 * w);
      if (m) found = 64 * w + __builtin_ctzll(m);
    }
    return found < 0 ? -1 : max(c + 1, found * a.r_max / 32);
  };
  auto routed = [&](int ad) {  // per lane: adapter ad is routed in the tile
    const int w = ad >> 6;
    const uint64_t m = w == 0 ? pm[0] : w == 1 ? pm[1] : w == 2 ? pm[2] : pm[3];
    return ((m >> (ad & 63)) & 1ull) != 0ull;
  };
  if (lora) {
    uint8_t* ut = pf_lds + kPfStages * kPfStageBytes;  // [128 tokens][kPfURow]
    // forming: kFTpt threads per token, kFG groups of 8 columns each
    constexpr int kFTpt = kPfThreads / kPfM, kFG = 4 / kFTpt;
    const int ftl = tid / kFTpt, fh = tid % kFTpt;
    const int64_t ft = m0 + ftl;
    const int64_t ftc = ft < a.T ? ft : m0;
    const int fidx = a.idx[ftc];
    const float fscl = a.scale[ftc];
    const int64_t slice = a.T * a.r_max;
    // Every load of a chunk is issued unconditionally (clamped to valid
    // addresses) and masked afterwards, so that all of them are in flight
    // together.
    for (int c = next_chunk(-1); c >= 0; c = next_chunk(c)) {
      const int c0 = c * 32;
      // Btilde operand: features fw0 + 16i + col, columns cb .. cb+8
      const int cb = c0 + 8 * kgrp;
      const int bad = min(cb / a.r_max, a.n_ad - 1), bj = cb % a.r_max;
      const int brk = ranksg ? ranksg[bad] : a.r_max;
      u32x4 bw[kPfFT];
#pragma unroll
      for (int i = 0; i < kPfFT; ++i) {
        const int64_t nl = fw0 - gbase + 16 * i + col;
        bw[i] = ld_global<u32x4>(Bg + (static_cast<int64_t>(bad) * Ng + (nl < Ng ? nl : 0)) *
                                          a.r_max + bj);
      }
      // forming: columns c0 + 8 (kFG fh + g), g < kFG (8 columns of one adapter)
      int frk[kFG];
      int64_t off[kFG];
#pragma unroll
      for (int g = 0; g < kFG; ++g) {
        const int c = c0 + 8 * (kFG * fh + g);
        frk[g] = ranksg ? ranksg[min(c / a.r_max, a.n_ad - 1)] : a.r_max;
        off[g] = (ft < a.T ? ft : m0) * a.r_max + c % a.r_max;
      }
      f32x4 sum[kFG][2] = {};
      constexpr int kZB = 8;  // slices loaded together
      for (int z0 = 0; z0 < a.up_ks; z0 += kZB) {
        f32x4 v[kZB][kFG][2];
#pragma unroll
        for (int dz = 0; dz < kZB; ++dz)
#pragma unroll
          for (int g = 0; g < kFG; ++g) {
            const int64_t o = static_cast<int64_t>(min(z0 + dz, a.up_ks - 1)) * slice + off[g];
            v[dz][g][0] = ld_global<f32x4>(Pg + o);
            v[dz][g][1] = ld_global<f32x4>(Pg + o + 4);
          }
        // every slice's loads are issued before the first sum (the compiler
        // would otherwise move some into the conditional sums below, one
        // memory round trip after the others)
#pragma unroll
        for (int dz = 0; dz < kZB; ++dz)
#pragma unroll
          for (int g = 0; g < kFG; ++g) asm volatile("" : "+v"(v[dz][g][0]), "+v"(v[dz][g][1]));
#pragma unroll
        for (int dz = 0; dz < kZB; ++dz)
          if (z0 + dz < a.up_ks)
#pragma unroll
            for (int g = 0; g < kFG; ++g) {
              sum[g][0] += v[dz][g][0];
              sum[g][1] += v[dz][g][1];
            }
      }
      // U_s: zero unless the columns' adapter is the token's, and at or past
      // its rank (padding rows of A may hold anything). The token's adapter
      // and scale are passed through an empty asm here so that the compiler
      // cannot test them (and wait for their loads, which the stage loads
      // precede) before the chunk's loads are issued.
      int fidx_c = fidx;
      float fscl_c = fscl;
      asm volatile("" : "+v"(fidx_c), "+v"(fscl_c));
      const int fad = (ft < a.T && fidx_c >= 0 && fidx_c < a.n_ad) ? fidx_c : -1;
#pragma unroll
      for (int g = 0; g < kFG; ++g) {
        const int c = c0 + 8 * (kFG * fh + g);
        const bool own = c < a.R && fad == c / a.r_max;
        const int keep = own ? min(max(frk[g], 0), a.r_max) - c % a.r_max : 0;
        float u[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const float sv = e < 4 ? sum[g][0][e] : sum[g][1][e - 4];
          u[e] = e < keep ? fscl_c * sv : 0.f;
        }
        *reinterpret_cast<u32x4*>(ut + ftl * kPfURow + 16 * (kFG * fh + g)) =
            u32x4{pack_bf16x2(u[0], u[1]), pack_bf16x2(u[2], u[3]), pack_bf16x2(u[4], u[5]),
                  pack_bf16x2(u[6], u[7])};
      }
      // Btilde: zero for an adapter not routed in the tile, and at or past
      // the rank
      const int bkeep = (cb < a.R && routed(bad))
                            ? min(max(brk, 0), a.r_max) - bj : 0;
      bf16x8 bv[kPfFT];
#pragma unroll
      for (int i = 0; i < kPfFT; ++i) bv[i] = as_bf16x8(keep_first8(bw[i], bkeep));
      wait_lgkm0_barrier();
      bf16x8 uv[kPfTT];
#pragma unroll
      for (int j = 0; j < kPfTT; ++j)
        uv[j] = as_bf16x8(
            *reinterpret_cast<const u32x4*>(ut + (tw0 + 16 * j + col) * kPfURow + 16 * kgrp));
#pragma unroll
      for (int i = 0; i < kPfFT; ++i)
#pragma unroll
        for (int j = 0; j < kPfTT; ++j) acc[i][j] = mfma16x16x32(bv[i], uv[j], acc[i][j]);
      wait_lgkm0_barrier();  // the tile is rewritten by the next chunk
    }
  }
  wait_vmcnt<0>();
  wait_lgkm0_barrier();
  read_half(0, 0);
  // unrolled over the stage ring so that stage offsets are constants; the
  // tail leaves the loop (a branch out of the loop, not around work in it)
  for (int s0 = 0; s0 < steps; s0 += kPfStages) {
#pragma unroll
    for (int u = 0; u < kPfStages; ++u) {
      const int s = s0 + u;
      if (s >= steps) break;
      // first half: one operand read (m = 1) beside each of the first kR
      // MFMAs (m = 0)
      read_half(u, 1);
      mfma_range(0, 0, kPfMfma);
#pragma unroll
      for (int g = 0; g < kR; ++g) {
        __builtin_amdgcn_sched_group_barrier(kSgMfma, 1, 0);
        __builtin_amdgcn_sched_group_barrier(kSgDsRead, 1, 0);
      }
      __builtin_amdgcn_sched_group_barrier(kSgMfma, kPfMfma - kR, 0);
      __builtin_amdgcn_sched_barrier(0);
      // second half: kQ MFMAs (m = 1) before the barrier, then the operand
      // reads of the next step and the loads of step s + 3 beside the rest
      mfma_range(1, 0, kQ);
      __builtin_amdgcn_sched_barrier(0);
      wait_vmcnt<kPfDma>();
      wait_lgkm0_barrier();
      __builtin_amdgcn_sched_barrier(0);
      read_half((u + 1) % kPfStages, 0);
      issue(u, min(s + 3, last));
      mfma_range(1, kQ, kPfMfma);
#pragma unroll
      for (int g = 0; g < kR; ++g) {
        __builtin_amdgcn_sched_group_barrier(kSgMfma, 1, 1);
        __builtin_amdgcn_sched_group_barrier(kSgDsRead, 1, 1);
      }
#pragma unroll
      for (int g = 0; g < kVPair; ++g) {
        __builtin_amdgcn_sched_group_barrier(kSgMfma, 1, 1);
        __builtin_amdgcn_sched_group_barrier(kSgVmem, 1, 1);
      }
      if (kPfDma > kVPair) __builtin_amdgcn_sched_group_barrier(kSgVmem, kPfDma - kVPair, 1);
      if (kPfMfma - kQ - kR > kVPair)
        __builtin_amdgcn_sched_group_barrier(kSgMfma, kPfMfma - kQ - kR - kVPair, 1);
      __builtin_amdgcn_sched_barrier(0);
    }
  }
  wait_vmcnt<0>();

  // ---- output. The tile's fp32 sums go through LDS (the stages are free once
  // every wave's loads have landed and its reads are done), so that each
  // thread then finishes 8 consecutive features of one token: the residual
  // and the output move as coalesced 16-byte pieces. Token rows are
  // kPfOutRow bytes (1 KB + 16), so the 16 tokens of one MFMA tile written
  // together fall in distinct banks.
  wait_lgkm0_barrier();
#pragma unroll
  for (int j = 0; j < kPfTT; ++j)
#pragma unroll
    for (int i = 0; i < kPfFT; ++i)
      *reinterpret_cast<f32x4*>(pf_lds + (tw0 + 16 * j + col) * kPfOutRow +
                                (16 * kPfFT * wn + 16 * i + 4 * kgrp) * 4) = acc[i][j];
  wait_lgkm0_barrier();
  const uint16_t* res = pick(a.gres, gq);
  uint16_t* y = pick(a.gy, gq);
  constexpr int kGroups = kPfN / 8;                       // 8-feature groups per token
  constexpr int kItems = kPfM * kGroups / kPfThreads;     // per thread
  u32x4 rv[kItems];
#pragma unroll
  for (int e = 0; e < kItems; ++e) {
    const int item = tid + e * kPfThreads, tl = item / kGroups, f = 8 * (item % kGroups);
    const int64_t t = m0 + tl, n = n0 - gbase + f;
    rv[e] = (res && t < a.T && n < Ng) ? ld_global<u32x4>(res + t * Ng + n) : u32x4{0u, 0u, 0u, 0u};
  }
#pragma unroll
  for (int e = 0; e < kItems; ++e) {
    const int item = tid + e * kPfThreads, tl = item / kGroups, f = 8 * (item % kGroups);
    const int64_t t = m0 + tl, n = n0 - gbase + f;
    const uint8_t* src = pf_lds + tl * kPfOutRow + f * 4;
    const f32x4 lo = *reinterpret_cast<const f32x4*>(src);
    const f32x4 hi = *reinterpret_cast<const f32x4*>(src + 16);
    float o[8] = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
    if (res) {
      const uint32_t r[4] = {rv[e].x, rv[e].y, rv[e].z, rv[e].w};
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        o[2 * q] += __uint_as_float(r[q] << 16);
        o[2 * q + 1] += __uint_as_float(r[q] & 0xffff0000u);
      }
    }
    if (t < a.T && n < Ng)
      *reinterpret_cast<u32x4*>(y + t * Ng + n) =
          u32x4{pack_bf16x2(o[0], o[1]), pack_bf16x2(o[2], o[3]), pack_bf16x2(o[4], o[5]),
                pack_bf16x2(o[6], o[7])};
  }
}

// ------------------------------------------------------------ long shrink
// Long chunks (T > 256): the shrink as SGMV partial sums over K slices,
//   P[g][z][t][j] = sum over slice z of x[t][k] A_g[a_t][j][k],   j < r_max,
// for the token's own adapter a_t only and every projection g of the call.
// Workgroup: 64 tokens x one K slice of sps 64-k steps; wave w owns tokens
// 16w .. 16w + 15 over the whole slice, so nothing is reduced across waves.
// The x slice is brought to LDS by direct loads while wave 0 lists the
// adapters routed in the tile; then, adapter by adapter, the A slices of
// every projection (r_max rows padded to 16) follow, in the 128-byte rows and
// chunk swizzle of the main product. x is read once for all projections.
constexpr int kShTok = 64;
constexpr int kShThreads = 256;
constexpr int kShWaves = kShThreads / kWave;
constexpr size_t kShLdsMax = 147456;

struct ShrinkShape {
  int ks;      // K slices (grid.y)
  int sps;     // 64-k steps per slice
  int rpad;    // r_max rounded up to 16
  size_t lds;  // dynamic LDS bytes
};

size_t shrink_lds(int sps, int rpad, int G) {
  return static_cast<size_t>(kShTok + G * rpad) * sps * 128;
}

// Fewest K slices (a divisor of the step count) that fit LDS and give at
// least one workgroup per compute unit, at most kShMaxSlices of them unless
// LDS needs more (the main product sums the slices for every U_s value it
// uses). One slice step always fits: (64 + 4 * 128) rows of 128 bytes.
constexpr int kShMaxSlices = 8;
ShrinkShape shrink_shape(int64_t T, int64_t K, int r_max, int G) {
  const int steps = static_cast<int>(K / 64);
  const int rpad = (r_max + 15) / 16 * 16;
  const int64_t tiles = (T + kShTok - 1) / kShTok;
  ShrinkShape best{steps, 1, rpad, shrink_lds(1, rpad, G)};
  for (int ks = 1; ks <= steps; ++ks) {
    if (steps % ks) continue;
    const int sps = steps / ks;
    const size_t lds = shrink_lds(sps, rpad, G);
    if (lds > kShLdsMax) continue;
    best = ShrinkShape{ks, sps, rpad, lds};
    if (tiles * ks >= 256 || ks >= kShMaxSlices) break;
  }
  return best;
}

template <int RT>
__global__ __launch_bounds__(kShThreads) void lora_shrink_long_kernel(GemmArgs a, int sps) {
  constexpr int rpad = 16 * RT;
  extern __shared__ __attribute__((aligned(16))) uint8_t sh_lds[];
  __shared__ int ad_list[kShTok];
  __shared__ int tok_ad[kShTok];
  __shared__ int n_list;

  const int tid = threadIdx.x, lane = tid % kWave;
  const int wave = __builtin_amdgcn_readfirstlane(tid / kWave);
  const int col = lane % 16, kgrp = lane / 16;
  const int64_t t0 = static_cast<int64_t>(blockIdx.x) * kShTok;
  const int z = blockIdx.y;
  const int G = a.G;
  static_assert(kShTok == kWave, "wave 0 reads one token per lane");
  const int64_t k0 = static_cast<int64_t>(z) * sps * 64;
  uint8_t* xl = sh_lds;                                            // [sps][64][128 B]
  uint8_t* al = sh_lds + static_cast<size_t>(sps) * kShTok * 128;  // [G][sps][rpad][128 B]

  // wave 0 reads the tile's adapters before it issues any x load, so that
  // listing them waits for that load alone; the other waves read theirs from
  // LDS after the list is made
  const int my = wave == 0 ? token_adapter(a, t0 + lane) : -1;
  const int64_t t = t0 + 16 * wave + col;  // this lane's token (MFMA column)

  // direct loads as in the main product: lane l writes 16 bytes at
  // block + 16 l = row 8b + l/8, position l%8, holding chunk (l%8) ^ (l/8);
  // wave w moves rows 8w .. +8 and 32 + 8w .. +8 of every step
  const int dchunk = (lane % 8) ^ (lane / 8);
  auto load_x = [&]() {
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int r0 = 8 * (wave + kShWaves * i);
      const int64_t tr = t0 + r0 + lane / 8;
      const uint16_t* src = a.x + (tr < a.T ? tr : t0) * a.K + k0 + 8 * dchunk;
      for (int st = 0; st < sps; ++st)
        lds_load16(src + 64 * st, xl + (static_cast<size_t>(st) * kShTok + r0) * 128);
    }
  };
  if (wave == 0) {  // adapters routed in the tile, in order of first appearance
    uint64_t pending = __ballot(my >= 0);
    int n = 0;
    uint64_t bits = 0ull;  // lane w < 4: word w of the tile's adapter bitmap
    while (pending) {
      const int ad = __shfl(my, __ffsll(static_cast<long long>(pending)) - 1);
      if (lane == 0) ad_list[n] = ad;
      ++n;
      if (lane == (ad >> 6)) bits |= 1ull << (ad & 63);
      pending &= ~__ballot(my == ad);
    }
    if (lane == 0) n_list = n;
    tok_ad[lane] = my;
    if (z == 0 && lane < 4) a.tile_present[4 * blockIdx.x + lane] = bits;
  }
  load_x();
  wait_lgkm0_barrier();  // the list; the x loads stay in flight
  const int n_ad_tile = n_list;
  const int t_ad = tok_ad[16 * wave + col];

  const int rd0 = col * 128 + 16 * (kgrp ^ (col % 8));
  const int rd1 = rd0 ^ 64;
  const int64_t slice = a.T * a.r_max;
  const int a_blocks = sps * (rpad / 8);  // 8-row load blocks per projection
  for (int q = 0; q < n_ad_tile; ++q) {
    const int ad = ad_list[q];
    if (q > 0) wait_lgkm0_barrier();  // every wave is done with the previous A
    // A rows of the adapter, every projection (rows past r_max repeat its
    // last row: never stored)
    for (int b = wave; b < G * a_blocks; b += kShWaves) {
      const int g = b / a_blocks, st = (b % a_blocks) / (rpad / 8), rb = b % (rpad / 8);
      const int j = min(8 * rb + lane / 8, a.r_max - 1);
      lds_load16(pick(a.ga, g) + (static_cast<int64_t>(ad) * a.r_max + j) * a.K + k0 + 64 * st +
                     8 * dchunk,
                 al + ((static_cast<size_t>(g) * sps + st) * rpad + 8 * rb) * 128);
    }
    wait_vmcnt<0>();
    wait_lgkm0_barrier();

    for (int g = 0; g < G; ++g) {
      f32x4 acc[RT];
#pragma unroll
      for (int rt = 0; rt < RT; ++rt) acc[rt] = f32x4{0.f, 0.f, 0.f, 0.f};
      const uint8_t* ag = al + static_cast<size_t>(g) * sps * rpad * 128;
      for (int st = 0; st < sps; ++st) {
#pragma unroll
        for (int m = 0; m < 2; ++m) {
          const int rd = m ? rd1 : rd0;
          const u32x4 xf =
              *reinterpret_cast<const u32x4*>(xl + (st * kShTok + 16 * wave) * 128 + rd);
          u32x4 af[RT];
#pragma unroll
          for (int rt = 0; rt < RT; ++rt)
            af[rt] = *reinterpret_cast<const u32x4*>(ag + (st * rpad + 16 * rt) * 128 + rd);
#pragma unroll
          for (int rt = 0; rt < RT; ++rt)
            acc[rt] = mfma16x16x32(as_bf16x8(af[rt]), as_bf16x8(xf), acc[rt]);
        }
      }
      // lane l of tile rt holds rank rows 16 rt + 4 (l/16) .. +4 of token t
      if (t_ad == ad) {
        float* Pz = a.pout + (static_cast<int64_t>(g) * a.up_ks + z) * slice + t * a.r_max;
#pragma unroll
        for (int rt = 0; rt < RT; ++rt) {
          const int j = 16 * rt + 4 * kgrp;
          if (j < a.r_max) *reinterpret_cast<f32x4*>(Pz + j) = acc[rt];
        }
      }
    }
  }
  wait_vmcnt<0>();  // no direct load may still be writing LDS when the workgroup ends
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

local_status_t launch_prefill(GemmArgs a, hipStream_t s) {
  a.gm = static_cast<int>((a.T + kPfM - 1) / kPfM);
  a.gn = static_cast<int>((a.N + kPfN - 1) / kPfN);
  static bool done = false;
  raise_lds_limit(lora_prefill_kernel, kPfLdsBytes, done);
  lora_prefill_kernel<<<a.gm * a.gn, kPfThreads, kPfLdsBytes, s>>>(a);
  return local_check_launch("lora_linear (prefill)");
}

template <int RT>
local_status_t launch_shrink_rt(GemmArgs a, const ShrinkShape& sh, hipStream_t s) {
  static bool done = false;
  raise_lds_limit(lora_shrink_long_kernel<RT>, kShLdsMax, done);
  const dim3 grid(static_cast<unsigned>((a.T + kShTok - 1) / kShTok), static_cast<unsigned>(sh.ks));
  lora_shrink_long_kernel<RT><<<grid, kShThreads, sh.lds, s>>>(a, sh.sps);
  return local_check_launch("lora_linear (shrink)");
}

local_status_t launch_shrink_long(const GemmArgs& a, const ShrinkShape& sh, hipStream_t s) {
  switch (sh.rpad / 16) {
    case 1: return launch_shrink_rt<1>(a, sh, s);
    case 2: return launch_shrink_rt<2>(a, sh, s);
    case 3: return launch_shrink_rt<3>(a, sh, s);
    case 4: return launch_shrink_rt<4>(a, sh, s);
    case 5: return launch_shrink_rt<5>(a, sh, s);
    case 6: return launch_shrink_rt<6>(a, sh, s);
    case 7: return launch_shrink_rt<7>(a, sh, s);
    default: return launch_shrink_rt<8>(a, sh, s);
  }
}

template <int FN, int FM, int XT>
local_status_t launch_stream(GemmArgs a, hipStream_t s) {
  using SS = StreamShape<FN, FM, XT>;
  static bool done = false;
  raise_lds_limit(lora_stream_kernel<FN, FM, XT>, kStLdsMax, done);
  dim3 grid(static_cast<unsigned>((a.N + 16 * FN - 1) / (16 * FN)),
            static_cast<unsigned>((a.T + 16 * FM - 1) / (16 * FM)),
            static_cast<unsigned>(a.ksplit));
  lora_stream_kernel<FN, FM, XT><<<grid, kStThreads, SS::S * SS::STAGE, s>>>(a);
  return local_check_launch("lora_linear (stream)");
}

// Decode sizes (T <= 256): base partial sums over K slices. Wider feature
// tiles cut the re-reads of x (every workgroup of a slice reads the slice of
// x for all its tokens); the shape is the widest tile (of 4, 3 or 2 MFMA
// tiles; 2 above 64 tokens) and K split that bring the grid closest to
// LOCAL_P_TARGET_WG workgroups from below.
#ifndef LOCAL_P_TARGET_WG
#define LOCAL_P_TARGET_WG 256  // aim: about one workgroup per compute unit
#endif
#ifndef LOCAL_P_WIDE
#define LOCAL_P_WIDE 6  // widest feature tile (MFMA tiles) up to 32 tokens; 0 = none
#endif

struct PartialShape {
  int fn;   // 16-row MFMA tiles per workgroup
  int ksb;  // K slices
};

int token_tiles(int64_t T) { return T <= 16 ? 1 : T <= 32 ? 2 : T <= 64 ? 4 : 8; }

PartialShape partial_shape(int64_t T, int64_t N, int64_t K, bool allow_wide) {
  const int64_t fm = token_tiles(T);
  const int64_t ttiles = (T + 16 * fm - 1) / (16 * fm);
  PartialShape best{T <= 64 ? 4 : 2, 1};
  int64_t best_wg = -1;
  const int fns[4] = {LOCAL_P_WIDE, 4, 3, 2};
  for (int fn : fns) {
    if (fn == 0 || (T > 64 && fn != 2) || (fn > 4 && (T > 32 || !allow_wide))) continue;
    const int64_t tiles = (N + 16 * fn - 1) / (16 * fn) * ttiles;
    for (int ks = 1; ks <= 8 && ks <= K / 64; ks *= 2) {
      const int64_t wg = tiles * ks;
      if (wg <= LOCAL_P_TARGET_WG && wg > best_wg) {
        best = {fn, ks};
        best_wg = wg;
      }
    }
  }
  return best;
}

// The stream kernel for the planned shape: FM token tiles by batch size
// (16 / 32 / 64 / 256 tokens), only the combinations the planner produces.
template <int FN, int XT>
local_status_t run_partial_fn(const GemmArgs& a, hipStream_t s) {
  if (a.T <= 16) return launch_stream<FN, 1, XT>(a, s);
  if constexpr (FN <= 4) {
    if (a.T <= 32) return launch_stream<FN, 2, XT>(a, s);
    if (a.T <= 64) return launch_stream<FN, 4, XT>(a, s);
    if constexpr (FN == 2 && XT <= 2) return launch_stream<2, 8, XT>(a, s);
  } else if constexpr (XT <= 2) {
    if (a.T <= 32) return launch_stream<FN, 2, XT>(a, s);
  }
  return local_fail(LOCAL_ERR_UNSUPPORTED, "lora_linear: tile of %d features, %d extra row tiles, "
                    "%lld tokens", 16 * FN, XT, static_cast<long long>(a.T));
}

template <int XT>
local_status_t run_partial_xt(const GemmArgs& a, int fn, hipStream_t s) {
#if LOCAL_P_WIDE > 4
  if (fn == LOCAL_P_WIDE) return run_partial_fn<LOCAL_P_WIDE, XT>(a, s);
#endif
  if (fn == 4) return run_partial_fn<4, XT>(a, s);
  if (fn == 3) return run_partial_fn<3, XT>(a, s);
  return run_partial_fn<2, XT>(a, s);
}

// Stacked-A rows each feature-tile workgroup takes with the base product
// (the shrink fused into it), or 0 when that would take more than 4 extra
// row tiles (2 above 64 tokens, where the accumulators of more would not fit
// in registers); then the SGMV shrink runs as its own kernel.
int partial_xrows(int64_t T, int64_t ftiles, int64_t rows) {
  if (rows == 0) return 0;
  const int64_t per = (rows + ftiles - 1) / ftiles;
  return per <= (T <= 64 ? 64 : 32) ? static_cast<int>(per) : 0;
}

local_status_t run_partial(const GemmArgs& a, int fn, hipStream_t s) {
  if (a.xrows == 0) return run_partial_xt<0>(a, fn, s);
  if (a.xrows <= 16) return run_partial_xt<1>(a, fn, s);
  if (a.xrows <= 32) return run_partial_xt<2>(a, fn, s);
  if (a.T <= 64) return run_partial_xt<4>(a, fn, s);
  return local_fail(LOCAL_ERR_UNSUPPORTED, "lora_linear: %d stacked rows per tile", a.xrows);
}

size_t align256(size_t v) { return (v + 255) & ~static_cast<size_t>(255); }

// One projection of a (grouped) call.
struct Proj {
  const uint16_t* W;
  int64_t N;
  const uint16_t* A;
  const uint16_t* B;
  const int32_t* ranks;
  const uint16_t* res;
  uint16_t* y;
};

// Sets the group fields of `a` for projections p[0..G).
void set_groups(GemmArgs& a, int G, const Proj* p) {
  a.G = G;
  int64_t n = 0;
  for (int g = 0; g <= kMaxGroup; ++g) {
    a.gstart[g] = n;
    if (g < G) n += p[g].N;
  }
  for (int g = 0; g < kMaxGroup; ++g) {
    const Proj& q = p[g < G ? g : 0];
    a.gw[g] = q.W;
    a.ga[g] = q.A;
    a.gb[g] = q.B;
    a.granks[g] = q.ranks;
    a.gres[g] = q.res;
    a.gy[g] = q.y;
  }
  a.N = n;
}

// Decode-size plan of a call: tile shape, fused shrink rows, workspace.
struct DecodePlan {
  PartialShape shape;
  int xrows;      // stacked-A rows per workgroup (shrink fused), or 0
  int slices;     // SGMV shrink K slices (shrink not fused), or 0
  bool split;     // a grouped call that runs its projections one by one
  size_t part_bytes, shrink_bytes;
};

DecodePlan plan_decode(int64_t T, int64_t K, int G, const Proj* p, int n_ad, int r_max) {
  DecodePlan d{};
  int64_t n_total = 0;
  for (int g = 0; g < G; ++g) n_total += p[g].N;
  const int64_t R = n_ad > 0 ? static_cast<int64_t>(n_ad) * r_max : 0;
  d.shape = partial_shape(T, n_total, K, true);
  int64_t ftiles = (n_total + 16 * d.shape.fn - 1) / (16 * d.shape.fn);
  d.xrows = partial_xrows(T, ftiles, G * R);
  if (d.shape.fn > 4 && d.xrows > 32) {  // the wide tile takes at most 2 extra row tiles
    d.shape = partial_shape(T, n_total, K, false);
    ftiles = (n_total + 16 * d.shape.fn - 1) / (16 * d.shape.fn);
    d.xrows = partial_xrows(T, ftiles, G * R);
  }
  // (Measured at 64 tokens over 16 adapters padded from ranks 8..64 to 64:
  // taking the shrink out of the base product saves 6.8 us of streaming
  // there, and its own SGMV launch costs 10.3 us; so the shrink rides along
  // whenever it fits.)
  if (n_ad > 0 && d.xrows == 0) {
    if (T > kSgMaxTokens) {
      d.split = true;
      return d;
    }
    d.slices = sgmv_slices(K, r_max);
  }
  d.part_bytes = align256(static_cast<size_t>(d.shape.ksb) * T * n_total * sizeof(float));
  d.shrink_bytes =
      d.xrows > 0 ? align256(static_cast<size_t>(d.shape.ksb) * T * G * R * sizeof(float))
                  : align256(static_cast<size_t>(d.slices) * T * G * r_max * sizeof(float));
  return d;
}

local_status_t lora_impl(const uint16_t* x, int64_t T, int64_t K, int G, const Proj* p,
                         int32_t n_adapters, int32_t r_max, const int32_t* adapter_idx,
                         const float* scale, void* ws, size_t* ws_bytes, hipStream_t s);

// Workspace need of a call that runs projections p[0..G) one after another.
local_status_t one_by_one(const uint16_t* x, int64_t T, int64_t K, int G, const Proj* p,
                          int32_t n_adapters, int32_t r_max, const int32_t* adapter_idx,
                          const float* scale, void* ws, size_t* ws_bytes, hipStream_t s) {
  if (!ws) {
    size_t need = 0;
    for (int g = 0; g < G; ++g) {
      size_t n = 0;
      const local_status_t st = lora_impl(x, T, K, 1, p + g, n_adapters, r_max, adapter_idx,
                                          scale, nullptr, &n, s);
      if (st != LOCAL_OK) return st;
      need = need > n ? need : n;
    }
    *ws_bytes = need;
    return LOCAL_OK;
  }
  for (int g = 0; g < G; ++g) {
    size_t n = *ws_bytes;
    const local_status_t st =
        lora_impl(x, T, K, 1, p + g, n_adapters, r_max, adapter_idx, scale, ws, &n, s);
    if (st != LOCAL_OK) return st;
  }
  return LOCAL_OK;
}

local_status_t lora_impl(const uint16_t* x, int64_t T, int64_t K, int G, const Proj* p,
                         int32_t n_adapters, int32_t r_max, const int32_t* adapter_idx,
                         const float* scale, void* ws, size_t* ws_bytes, hipStream_t s) {
  const int R = n_adapters > 0 ? n_adapters * r_max : 0;
  const bool decode = T <= kSgMaxTokens;
  if (G > 1 && !decode) {  // one launch over all projections when no tile straddles two
    for (int q = 0; q < G; ++q)
      if (p[q].N % kPfN != 0)
        return one_by_one(x, T, K, G, p, n_adapters, r_max, adapter_idx, scale, ws, ws_bytes, s);
  }
  DecodePlan d{};
  if (decode) {
    d = plan_decode(T, K, G, p, n_adapters, r_max);
    if (d.split)
      return one_by_one(x, T, K, G, p, n_adapters, r_max, adapter_idx, scale, ws, ws_bytes, s);
  }
  // Workspace. Decode sizes (T <= kSgMaxTokens): the base partial sums
  // [ksb][T][N] fp32 (N over all projections), then the shrink's partial
  // sums: [ksb][T][G*R] fp32 when the shrink runs inside the base product,
  // [slices][T][r_max] after the SGMV shrink. Above: the long shrink's
  // partial sums [G][ks][T][r_max] fp32, then its adapter bitmaps
  // [ceil(T/64)][4] uint64.
  const ShrinkShape shs = decode ? ShrinkShape{} : shrink_shape(T, K, r_max, G);
  const size_t long_p =
      align256(static_cast<size_t>(G) * shs.ks * T * r_max * sizeof(float));
  const size_t long_bits = align256(static_cast<size_t>((T + 63) / 64) * 4 * sizeof(uint64_t));
  const size_t need = decode ? d.part_bytes + d.shrink_bytes
                             : (n_adapters > 0 ? long_p + long_bits : 0);
  if (!ws) {
    *ws_bytes = need;
    return LOCAL_OK;
  }
  if (*ws_bytes < need)
    return local_fail(LOCAL_ERR_WORKSPACE, "lora_linear: workspace %zu < %zu", *ws_bytes, need);
  if (T == 0) return LOCAL_OK;

  GemmArgs g{};
  g.x = x;
  g.T = T;
  g.K = K;
  g.idx = adapter_idx;
  g.scale = scale;
  g.n_ad = n_adapters;
  g.r_max = r_max;
  g.R = R;
  local_status_t st;

  if (decode) {
    float* part = static_cast<float*>(ws);
    float* sp = reinterpret_cast<float*>(static_cast<char*>(ws) + d.part_bytes);
    const bool fused = d.xrows > 0;
    if (n_adapters > 0 && !fused) {  // SGMV shrink of every projection: partial sums
      GemmArgs sh = g;
      set_groups(sh, G, p);
      sh.pout = sp;
      sh.up_ks = d.slices;
      sh.p_stride = G * r_max;
      if ((st = run_sgmv_shrink(sh, s)) != LOCAL_OK) return st;
    }
    GemmArgs m = g;  // base product (+ fused shrink): partial sums per K slice
    set_groups(m, G, p);
    m.part = part;
    m.ksplit = d.shape.ksb;
    m.xrows = d.xrows;
    m.pout = sp;
    if ((st = run_partial(m, d.shape.fn, s)) != LOCAL_OK) return st;
    m.up_ks = fused ? d.shape.ksb : d.slices;  // epilogue: sums, up-projection, residual
    m.p_stride = fused ? G * R : G * r_max;
    m.p_stacked = fused ? 1 : 0;
    m.ksplit = d.shape.ksb;
    return run_epilogue(m, s);
  }

  // long chunks: the shrink's partial sums [G][ks][T][r_max], then the main
  // product over the projections' tiles
  float* P = n_adapters > 0 ? static_cast<float*>(ws) : nullptr;
  GemmArgs m = g;
  set_groups(m, G, p);
  m.pout = P;
  m.tile_present =
      n_adapters > 0 ? reinterpret_cast<uint64_t*>(static_cast<char*>(ws) + long_p) : nullptr;
  m.up_ks = shs.ks;
  if (n_adapters > 0 && (st = launch_shrink_long(m, shs, s)) != LOCAL_OK) return st;
  return launch_prefill(m, s);
}

// Argument checks shared by the entry points (before any launch).
local_status_t check_args(const char* who, const uint16_t* x, int64_t T, int64_t K, int G,
                          const Proj* p, int32_t n_adapters, int32_t r_max,
                          const int32_t* adapter_idx, const float* scale, size_t* ws_bytes,
                          bool sizes_only) {
  if (!ws_bytes) return local_fail(LOCAL_ERR_WORKSPACE, "%s: ws_bytes is NULL", who);
  if (T < 0 || K <= 0 || n_adapters < 0)
    return local_fail(LOCAL_ERR_SHAPE, "%s: T=%lld K=%lld n_adapters=%d", who, (long long)T,
                      (long long)K, n_adapters);
  for (int g = 0; g < G; ++g)
    if (p[g].N <= 0)
      return local_fail(LOCAL_ERR_SHAPE, "%s: N=%lld (projection %d)", who, (long long)p[g].N, g);
  bool shapes_ok = K % 64 == 0 && n_adapters <= 256 &&
                   (n_adapters == 0 || (r_max >= 8 && r_max <= 128 && r_max % 8 == 0));
  for (int g = 0; g < G; ++g) shapes_ok = shapes_ok && p[g].N % 64 == 0;
  if (!shapes_ok)
    return local_fail(LOCAL_ERR_UNSUPPORTED,
                      "%s: K=%lld n_adapters=%d r_max=%d (need K and every N %% 64 == 0, "
                      "n_adapters <= 256, r_max in [8,128] and %% 8 == 0)",
                      who, (long long)K, n_adapters, r_max);
  if (sizes_only || T == 0) return LOCAL_OK;
  if (!x) return local_fail(LOCAL_ERR_NULL, "%s: NULL x", who);
  for (int g = 0; g < G; ++g) {
    if (!p[g].W || !p[g].y) return local_fail(LOCAL_ERR_NULL, "%s: NULL W or y", who);
    if (n_adapters > 0 && (!p[g].A || !p[g].B))
      return local_fail(LOCAL_ERR_NULL, "%s: NULL adapter argument", who);
  }
  if (n_adapters > 0 && (!adapter_idx || !scale))
    return local_fail(LOCAL_ERR_NULL, "%s: NULL adapter argument", who);
  return LOCAL_OK;
}

}  // namespace

// ---- the long-chunk shrink for other files (declared in lora_internal.hpp)
size_t token_shrink_bytes(int64_t T, int64_t K, int r_max, int G, int* slices) {
  const ShrinkShape sh = shrink_shape(T, K, r_max, G);
  if (slices) *slices = sh.ks;
  return align256(static_cast<size_t>(G) * sh.ks * T * r_max * sizeof(float)) +
         align256(static_cast<size_t>((T + 63) / 64) * 4 * sizeof(uint64_t));
}

local_status_t token_shrink(const uint16_t* x, int64_t T, int64_t K, int G,
                            const uint16_t* const* A, int n_ad, int r_max, const int32_t* idx,
                            void* ws, hipStream_t s) {
  const ShrinkShape sh = shrink_shape(T, K, r_max, G);
  GemmArgs g{};
  g.x = x;
  g.T = T;
  g.K = K;
  g.idx = idx;
  g.n_ad = n_ad;
  g.r_max = r_max;
  g.R = n_ad * r_max;
  g.G = G;
  for (int q = 0; q < G; ++q) g.ga[q] = A[q];
  g.pout = static_cast<float*>(ws);
  g.up_ks = sh.ks;
  g.tile_present = reinterpret_cast<uint64_t*>(
      static_cast<char*>(ws) +
      align256(static_cast<size_t>(G) * sh.ks * T * r_max * sizeof(float)));
  return launch_shrink_long(g, sh, s);
}

}  // namespace localk

using namespace localk;

extern "C" local_status_t local_lora_linear(
    const uint16_t* x, int64_t T, int64_t K, const uint16_t* W, int64_t N, const uint16_t* A,
    const uint16_t* B, int32_t n_adapters, int32_t r_max, const int32_t* ranks,
    const int32_t* adapter_idx, const float* scale, const uint16_t* residual, uint16_t* y,
    void* ws, size_t* ws_bytes, void* stream) {
  const Proj p{W, N, A, B, ranks, residual, y};
  local_status_t st = check_args("lora_linear", x, T, K, 1, &p, n_adapters, r_max, adapter_idx,
                                 scale, ws_bytes, ws == nullptr);
  if (st != LOCAL_OK) return st;
  return lora_impl(x, T, K, 1, &p, n_adapters, r_max, adapter_idx, scale, ws, ws_bytes,
                   static_cast<hipStream_t>(stream));
}

extern "C" local_status_t local_lora_linear_grouped(
    const uint16_t* x, int64_t T, int64_t K, int32_t G, const uint16_t* const* W,
    const int64_t* N, const uint16_t* const* A, const uint16_t* const* B, int32_t n_adapters,
    int32_t r_max, const int32_t* const* ranks, const int32_t* adapter_idx, const float* scale,
    uint16_t* const* y, void* ws, size_t* ws_bytes, void* stream) {
  if (G < 1 || G > kMaxGroup)
    return local_fail(LOCAL_ERR_UNSUPPORTED, "lora_linear_grouped: G=%d (need 1..%d)", G,
                      kMaxGroup);
  if (!W || !N || !y || (n_adapters > 0 && (!A || !B)))
    return local_fail(LOCAL_ERR_NULL, "lora_linear_grouped: NULL argument array");
  Proj p[kMaxGroup];
  for (int g = 0; g < G; ++g)
    p[g] = Proj{W[g], N[g], n_adapters > 0 ? A[g] : nullptr, n_adapters > 0 ? B[g] : nullptr,
                (n_adapters > 0 && ranks) ? ranks[g] : nullptr, nullptr, y[g]};
  local_status_t st = check_args("lora_linear_grouped", x, T, K, G, p, n_adapters, r_max,
                                 adapter_idx, scale, ws_bytes, ws == nullptr);
  if (st != LOCAL_OK) return st;
  return lora_impl(x, T, K, G, p, n_adapters, r_max, adapter_idx, scale, ws, ws_bytes,
                   static_cast<hipStream_t>(stream));
}
