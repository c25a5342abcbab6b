// local_lora_grad, local_lora_grad_input: the backward of the mixed-adapter
// LoRA projection, for the training chunks that update an agent's adapter
// while the frozen base serves (§2.2: adapters on a frozen base model; §4:
// background training in bounded chunks). With u_t = x_t A_a^T and
// g_t = s_t dy_t B_a (a = a_t, both over a's rank):
//   dB_a = sum_{t of a} s_t dy_t^T u_t,  dA_a = sum_{t of a} g_t^T x_t,
//   dx_t = dy_t W + g_t A_a.
//
// Design (HBM-bound for the adapter gradients: 4 T r (K + N) flop, shrinks
// included, against T (K + N) bf16 read), four launches:
//  * set-up: the tokens bucketed by adapter (a stable counting sort in one
//    workgroup, as in SGMV) while the other workgroups transpose B per
//    adapter to [r_max][N];
//  * u = x A^T and dy B from the long-chunk shrink of the forward path, as
//    float32 partial sums over K slices (two launches);
//  * dB and dA as segmented outer products, both in one launch: a workgroup
//    per (64 tokens of one adapter, 256 threads x PT columns of dy or x)
//    forms the tokens' coefficients in LDS (slices summed in order, times
//    s_t, 0 past the rank), then each thread keeps PT x r_max float32 sums
//    over the tokens, each token's row read once, coalesced;
//  * the partial sums of the 64-token units added in unit order by a reduce
//    pass: deterministic, no atomics.
//  dx runs the forward fused projection on the transposed weights: with
//  x := dy, W := W^T, A := B^T and B := A^T, its shrink is dy B and its
//  delta s (dy B) A, so dx needs no kernel of its own.
#include <algorithm>
#include <type_traits>

#include "common.hpp"
#include "lora_internal.hpp"

namespace localk {
namespace {

constexpr int kGrUnit = 64;      // tokens per unit of the segmented products
constexpr int kGrThreads = 256;
constexpr int kGrMaxAdapters = 256;
constexpr int kGrGroup = 4;            // projections of one x in a call
constexpr int kGrJobs = 2 * kGrGroup;  // (dB, dA) per projection

typedef int32_t i32x4 __attribute__((ext_vector_type(4)));

size_t al256(size_t v) { return (v + 255) & ~static_cast<size_t>(255); }

// Inclusive prefix sum over the 64 lanes of a wave.
__device__ __forceinline__ int wave_incl_scan(int v) {
  const int lane = threadIdx.x % kWave;
#pragma unroll
  for (int off = 1; off < kWave; off <<= 1) {
    const int u = __shfl_up(v, off);
    if (lane >= off) v += u;
  }
  return v;
}

// ---- tokens bucketed by adapter, stable: perm[seg[a] .. seg[a+1]) holds the
// tokens of adapter a in ascending order; tokens without one are left out.
// useg[a] = sum over b < a of ceil(T_b / 64): the first 64-token unit of a;
// utab[k] = (adapter, first position in perm, token count) of unit k.
// One workgroup of kPrepThreads: wave w owns a contiguous chunk of the
// tokens. It counts its chunk per adapter (ballots over equal adapters),
// then one prefix over (adapter, wave) gives every wave its own running
// offsets, and each wave places its chunk in order with no further barrier.
constexpr int kPrepThreads = 1024;
constexpr int kPrepWaves = kPrepThreads / kWave;

__device__ void bucket_tokens(const int32_t* __restrict__ idx, int64_t T, int n_ad,
                              int32_t* __restrict__ perm, int32_t* __restrict__ seg,
                              int32_t* __restrict__ useg, i32x4* __restrict__ utab) {
  __shared__ int cnt[kPrepWaves][kGrMaxAdapters];  // per wave: count, then running offset
  __shared__ int tot[kGrMaxAdapters];
  const int tid = threadIdx.x, wave = tid / kWave, lane = tid % kWave;
  const int64_t chunk = (T + kPrepWaves * kWave - 1) / (kPrepWaves * kWave) * kWave;
  const int64_t c0 = wave * chunk, c1 = min(T, c0 + chunk);
  auto adapter_at = [&](int64_t t) {
    const int32_t v = t < c1 ? idx[t] : -1;
    return (v >= 0 && v < n_ad) ? v : -1;
  };
  for (int a = lane; a < n_ad; a += kWave) cnt[wave][a] = 0;
  // 1. counts of the wave's chunk (lane 0 writes the wave's own row)
  for (int64_t t0 = c0; t0 < c1; t0 += kWave) {
    const int my = adapter_at(t0 + lane);
    uint64_t pending = __ballot(my >= 0);
    while (pending) {
      const int ad = __builtin_amdgcn_readlane(my, __ffsll(static_cast<long long>(pending)) - 1);
      const uint64_t m = __ballot(my == ad);
      if (lane == 0) cnt[wave][ad] += __popcll(m);
      pending &= ~m;
    }
  }
  __syncthreads();
  // 2. per adapter totals; prefixes over adapters (wave 0); each wave's
  //    first position per adapter
  for (int a = tid; a < n_ad; a += kPrepThreads) {
    int c = 0;
    for (int w = 0; w < kPrepWaves; ++w) c += cnt[w][a];
    tot[a] = c;
  }
  __syncthreads();
  if (wave == 0) {
    int run = 0, urun = 0;
    for (int a0 = 0; a0 < n_ad; a0 += kWave) {
      const int a = a0 + lane;
      const int c = a < n_ad ? tot[a] : 0;
      const int u = (c + kGrUnit - 1) / kGrUnit;
      const int ic = wave_incl_scan(c), iu = wave_incl_scan(u);
      if (a < n_ad) {
        const int s0 = run + ic - c, u0 = urun + iu - u;
        seg[a] = s0;
        useg[a] = u0;
        tot[a] = s0;
        for (int k = 0; k < u; ++k)
          utab[u0 + k] = i32x4{a, s0 + kGrUnit * k, min(kGrUnit, c - kGrUnit * k), 0};
      }
      run += __shfl(ic, kWave - 1);
      urun += __shfl(iu, kWave - 1);
    }
    if (lane == 0) {
      seg[n_ad] = run;
      useg[n_ad] = urun;
    }
  }
  __syncthreads();
  for (int a = tid; a < n_ad; a += kPrepThreads) {
    int off = tot[a];
    for (int w = 0; w < kPrepWaves; ++w) {
      const int c = cnt[w][a];
      cnt[w][a] = off;
      off += c;
    }
  }
  __syncthreads();
  // 3. the wave places its chunk in order
  for (int64_t t0 = c0; t0 < c1; t0 += kWave) {
    const int my = adapter_at(t0 + lane);
    uint64_t pending = __ballot(my >= 0);
    while (pending) {
      const int ad = __builtin_amdgcn_readlane(my, __ffsll(static_cast<long long>(pending)) - 1);
      const uint64_t m = __ballot(my == ad);
      const int base = cnt[wave][ad];
      if (my == ad) perm[base + __popcll(m & ((1ull << lane) - 1ull))] = static_cast<int32_t>(t0 + lane);
      if (lane == 0) cnt[wave][ad] = base + __popcll(m);
      pending &= ~m;
    }
  }
}

// ---- per-matrix transposes dst[i][c][r] = src[i][r][c] of n matrices of
// R x C bf16 (R and C multiples of 8). A tile of TR x TC (at most 2048
// elements) goes through LDS: 16-byte loads along the source rows, 16-byte
// stores along the destination rows.
struct TransposeJob {
  const uint16_t* src;
  uint16_t* dst;
  int64_t R, C;
  int TR, TC, tiles_c, tiles;
};

TransposeJob transpose_job(const uint16_t* src, uint16_t* dst, int64_t n, int64_t R,
                           int64_t C) {
  TransposeJob j{src, dst, R, C, 0, 0, 0, 0};
  if (R < C) {
    j.TR = static_cast<int>(std::min<int64_t>(R, 64));
    j.TC = 2048 / j.TR / 8 * 8;
  } else {
    j.TC = static_cast<int>(std::min<int64_t>(C, 64));
    j.TR = 2048 / j.TC / 8 * 8;
  }
  j.tiles_c = static_cast<int>((C + j.TC - 1) / j.TC);
  j.tiles = j.tiles_c * static_cast<int>((R + j.TR - 1) / j.TR) * static_cast<int>(n);
  return j;
}

// Tile k of job j (tiles of matrix 0 first, then of matrix 1, ...), by the
// 256 threads of quarter q of the workgroup; every thread of the workgroup
// calls it (the barrier is shared), a quarter without a tile with live false.
__device__ void transpose_tile(const TransposeJob& j, int k, bool live) {
  __shared__ __attribute__((aligned(16))) uint16_t tiles[kPrepThreads / kGrThreads][4096];
  const int q = threadIdx.x / kGrThreads;
  uint16_t* tile = tiles[q];  // TR x (TC + 8)
  const int TR = j.TR, TC = j.TC, ld = TC + 8;
  const int per_mat = j.tiles_c * static_cast<int>((j.R + TR - 1) / TR);
  const int64_t i = live ? k / per_mat : 0;
  const int kk = live ? k % per_mat : 0;
  const int64_t r0 = static_cast<int64_t>(kk / j.tiles_c) * TR;
  const int64_t c0 = static_cast<int64_t>(kk % j.tiles_c) * TC;
  const uint16_t* s = j.src + i * j.R * j.C;
  uint16_t* d = j.dst + i * j.R * j.C;
  const int e8 = (threadIdx.x % kGrThreads) * 8;
  if (live && e8 < TR * TC) {
    const int rr = e8 / TC, cc = e8 % TC;
    if (r0 + rr < j.R && c0 + cc < j.C)
      *reinterpret_cast<u32x4*>(tile + rr * ld + cc) =
          ld_global<u32x4>(s + (r0 + rr) * j.C + c0 + cc);
  }
  __syncthreads();
  if (live && e8 < TR * TC) {
    const int cc = e8 / TR, rr = e8 % TR;
    if (c0 + cc < j.C && r0 + rr < j.R) {
      uint32_t w[4];
#pragma unroll
      for (int h = 0; h < 4; ++h)
        w[h] = static_cast<uint32_t>(tile[(rr + 2 * h) * ld + cc]) |
               (static_cast<uint32_t>(tile[(rr + 2 * h + 1) * ld + cc]) << 16);
      *reinterpret_cast<u32x4*>(d + (c0 + cc) * j.R + r0 + rr) = u32x4{w[0], w[1], w[2], w[3]};
    }
  }
}

// One launch for the set-up work, workgroups of kPrepThreads: workgroup 0
// buckets the tokens (when idx is given); each other workgroup transposes
// four tiles (one per quarter) of one job, the jobs one after another.
struct PrepArgs {
  TransposeJob job[kGrGroup];
  int n_jobs;
  const int32_t* idx;
  int64_t T;
  int n_ad;
  int32_t *perm, *seg, *useg;
  i32x4* utab;
};

__global__ __launch_bounds__(kPrepThreads) void grad_prep_kernel(PrepArgs a) {
  constexpr int per = kPrepThreads / kGrThreads;
  int wg = blockIdx.x;
  if (a.idx) {
    if (wg == 0) {
      bucket_tokens(a.idx, a.T, a.n_ad, a.perm, a.seg, a.useg, a.utab);
      return;
    }
    --wg;
  }
  // the job of this workgroup (each job's tiles fill whole workgroups)
  int q = 0;
  while (q + 1 < a.n_jobs && wg >= (a.job[q].tiles + per - 1) / per) {
    wg -= (a.job[q].tiles + per - 1) / per;
    ++q;
  }
  const int k = wg * per + static_cast<int>(threadIdx.x) / kGrThreads;
  transpose_tile(a.job[q], k, k < a.job[q].tiles);
}

local_status_t run_prep(hipStream_t s, const PrepArgs& a) {
  constexpr int per = kPrepThreads / kGrThreads;
  int wgs = a.idx ? 1 : 0;
  for (int q = 0; q < a.n_jobs; ++q) wgs += (a.job[q].tiles + per - 1) / per;
  if (wgs == 0) return LOCAL_OK;
  grad_prep_kernel<<<static_cast<unsigned>(wgs), kPrepThreads, 0, s>>>(a);
  return local_check_launch("lora_grad (prep)");
}

// Coefficients of a unit's tokens into LDS: cl[i][j] = s_i * (sum over the
// shrink's K slices, in slice order) for j below the rank, 0 elsewhere and
// for i >= nt. Each thread forms 4 consecutive j of one token at a time with
// 16-byte loads, 8 slices in flight (the sum stays in slice order).
template <int RJ>
__device__ __forceinline__ void stage_coefficients(float (*cl)[RJ], const int* tok,
                                                   const float* tsc, const float* S, int ks,
                                                   int64_t T, int r_max, int nt, int rk) {
  for (int e = threadIdx.x; e < kGrUnit * RJ / 4; e += kGrThreads) {
    const int i = e / (RJ / 4), j = 4 * (e % (RJ / 4));
    f32x4 sum{0.f, 0.f, 0.f, 0.f};
    if (i < nt && j < rk) {
      const float* src = S + static_cast<int64_t>(tok[i]) * r_max + j;
      for (int z0 = 0; z0 < ks; z0 += 8) {
        f32x4 v[8];
#pragma unroll
        for (int z = 0; z < 8; ++z)
          v[z] = z0 + z < ks
                     ? *reinterpret_cast<const f32x4*>(src + static_cast<int64_t>(z0 + z) * T * r_max)
                     : f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int z = 0; z < 8; ++z) sum += v[z];
      }
      sum *= tsc[i];
#pragma unroll
      for (int q = 0; q < 4; ++q)
        if (j + q >= rk) sum[q] = 0.f;
    }
    *reinterpret_cast<f32x4*>(&cl[i][j]) = sum;
  }
}

// ---- segmented outer products, every gradient of the call in one launch.
// blockIdx.y = job: 2g = dB of projection g (V = dy_g, P = N_g, coefficients
// s u_g, partials [P][r_max]), 2g + 1 = dA of projection g (V = x, P = K,
// coefficients g_g = s dy_g B_g, partials [r_max][P]).
// Workgroup = (unit, column tile of 256 PT columns). The unit's 64 token
// rows are loaded at once, ahead of everything else, so that a workgroup
// waits for memory about three times (unit table, token ids, rows and
// coefficients together). The coefficients are formed in LDS from the
// shrink's K-slice partial sums (u = x A^T, or dy B): summed over the slices
// in order, times s_t, 0 at or past the adapter's rank. Each thread then
// keeps PT x RJ float32 sums of c_t[j] V_t[p] over the unit's tokens.
struct OuterArgs {
  const uint16_t* V[kGrJobs];
  const float* S[kGrJobs];  // shrink partial sums [ks][T][r_max]
  int ks[kGrJobs];
  float* part[kGrJobs];
  int64_t P[kGrJobs];
  const int32_t* ranks[kGrJobs];  // the projection's ranks, or NULL
};

template <int PT, int RJ>
__global__ __launch_bounds__(kGrThreads) void grad_outer_kernel(
    OuterArgs args, int64_t T, int64_t ptiles, int r_max, const int32_t* __restrict__ perm,
    const int32_t* __restrict__ useg, const i32x4* __restrict__ utab, int n_ad,
    const float* __restrict__ scale) {
  using RowT = typename std::conditional<PT == 2, uint32_t, uint16_t>::type;
  __shared__ __attribute__((aligned(16))) float cl[kGrUnit][RJ];
  __shared__ int tok[kGrUnit];
  __shared__ float tsc[kGrUnit];
  const int job = blockIdx.y;
  const int64_t P = args.P[job];
  const int slot = static_cast<int>(blockIdx.x / ptiles);
  const int64_t p0 = ((blockIdx.x % ptiles) * kGrThreads + threadIdx.x) * PT;
  if ((blockIdx.x % ptiles) * kGrThreads * PT >= P) return;  // the whole tile is past P
  if (slot >= useg[n_ad]) return;                             // past the last unit
  const i32x4 ut = utab[slot];
  const int a = ut.x, first = ut.y, nt = ut.z;
  const uint16_t* V = args.V[job];
  const float* S = args.S[job];
  const int ks = args.ks[job];
  const int tid = threadIdx.x;
  if (tid < nt) {
    const int t = perm[first + tid];
    tok[tid] = t;
    tsc[tid] = scale[t];
  }
  const int32_t* ranks = args.ranks[job];
  const int rk = ranks ? min(max(ranks[a], 0), r_max) : r_max;
  __syncthreads();
  // every row of the unit in flight at once (rows past nt read as zero)
  const bool live = p0 < P;
  RowT raw[kGrUnit];
#pragma unroll
  for (int i = 0; i < kGrUnit; ++i)
    raw[i] = (live && i < nt)
                 ? ld_global<RowT>(V + static_cast<int64_t>(tok[i]) * P + p0)
                 : RowT(0);
  stage_coefficients<RJ>(cl, tok, tsc, S, ks, T, r_max, nt, rk);
  __syncthreads();
  float acc[PT][RJ];
#pragma unroll
  for (int q = 0; q < PT; ++q)
#pragma unroll
    for (int j = 0; j < RJ; ++j) acc[q][j] = 0.f;
#pragma unroll
  for (int i = 0; i < kGrUnit; ++i) {
    float v[PT];
    if constexpr (PT == 2) {
      v[0] = __uint_as_float(static_cast<uint32_t>(raw[i]) << 16);
      v[1] = __uint_as_float(static_cast<uint32_t>(raw[i]) & 0xffff0000u);
    } else {
      v[0] = __uint_as_float(static_cast<uint32_t>(raw[i]) << 16);
    }
#pragma unroll
    for (int j4 = 0; j4 < RJ; j4 += 4) {
      const f32x4 cj = *reinterpret_cast<const f32x4*>(&cl[i][j4]);
#pragma unroll
      for (int q = 0; q < PT; ++q) {
        acc[q][j4] += cj[0] * v[q];
        acc[q][j4 + 1] += cj[1] * v[q];
        acc[q][j4 + 2] += cj[2] * v[q];
        acc[q][j4 + 3] += cj[3] * v[q];
      }
    }
  }
  if (!live) return;
  float* out = args.part[job] + static_cast<int64_t>(slot) * P * r_max;
  if (job & 1) {
#pragma unroll
    for (int q = 0; q < PT; ++q)
#pragma unroll
      for (int j = 0; j < RJ; ++j)
        if (j < r_max) out[static_cast<int64_t>(j) * P + p0 + q] = acc[q][j];
  } else {
#pragma unroll
    for (int q = 0; q < PT; ++q)
#pragma unroll
      for (int j = 0; j < RJ; j += 4)
        if (j < r_max)
          *reinterpret_cast<f32x4*>(out + (p0 + q) * r_max + j) =
              f32x4{acc[q][j], acc[q][j + 1], acc[q][j + 2], acc[q][j + 3]};
  }
}

// ---- the same products on the matrix cores (r_max <= 64), float32 MFMA
// v_mfma_f32_16x16x4_f32: D[16 x 16] += A[16 x 4] B[4 x 16], lane l giving
// A[l%16][l/16] and B[l/16][l%16] and holding D[4(l/16) + i][l%16]. With
// the contraction over 4 tokens, A = the coefficients c[t][j] (j = row) and
// B = the token rows V[t][col] (col = column): both are read along their
// rows, so the token-major inputs need no transpose. A wave owns 128
// columns: lane l loads 8 consecutive columns 8(l%16) .. +7 of token l/16
// (16 bytes, 256 contiguous bytes per token), and MFMA e (e < 8) takes
// element e, i.e. columns 8n + e for D column n. JT tiles of 16 cover
// r_max. The unit's rows are all in flight before the first product.
template <int JT>
__global__ __launch_bounds__(kGrThreads) void grad_outer_mfma_kernel(
    OuterArgs args, int64_t T, int64_t ptiles, int r_max, const int32_t* __restrict__ perm,
    const int32_t* __restrict__ useg, const i32x4* __restrict__ utab, int n_ad,
    const float* __restrict__ scale) {
  constexpr int RJ = 16 * JT;
  constexpr int kSteps = kGrUnit / 4;
  __shared__ __attribute__((aligned(16))) float cl[kGrUnit][RJ];
  __shared__ int tok[kGrUnit];
  __shared__ float tsc[kGrUnit];
  const int job = blockIdx.y;
  const int64_t P = args.P[job];
  const int slot = static_cast<int>(blockIdx.x / ptiles);
  const int tid = threadIdx.x, lane = tid % kWave, wave = tid / kWave;
  const int64_t wcol = ((blockIdx.x % ptiles) * (kGrThreads / kWave) + wave) * 128;
  if ((blockIdx.x % ptiles) * 512 >= P) return;  // the whole tile is past P
  if (slot >= useg[n_ad]) return;                // past the last unit
  const i32x4 ut = utab[slot];
  const int a = ut.x, first = ut.y, nt = ut.z;
  const uint16_t* V = args.V[job];
  const float* S = args.S[job];
  const int ks = args.ks[job];
  if (tid < nt) {
    const int t = perm[first + tid];
    tok[tid] = t;
    tsc[tid] = scale[t];
  }
  const int32_t* ranks = args.ranks[job];
  const int rk = ranks ? min(max(ranks[a], 0), r_max) : r_max;
  __syncthreads();
  const int n = lane % 16, k = lane / 16;
  const int64_t col = wcol + 8 * n;  // this lane's 8 columns
  const bool live = col < P;
  u32x4 raw[kSteps];
#pragma unroll
  for (int st = 0; st < kSteps; ++st) {
    const int i = 4 * st + k;
    raw[st] = (live && i < nt) ? ld_global<u32x4>(V + static_cast<int64_t>(tok[i]) * P + col)
                               : u32x4{0u, 0u, 0u, 0u};
  }
  stage_coefficients<RJ>(cl, tok, tsc, S, ks, T, r_max, nt, rk);
  __syncthreads();
  f32x4 acc[JT][8];
#pragma unroll
  for (int jt = 0; jt < JT; ++jt)
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[jt][e] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int st = 0; st < kSteps; ++st) {
    float v[8];
#pragma unroll
    for (int h = 0; h < 4; ++h) {
      v[2 * h] = __uint_as_float(raw[st][h] << 16);
      v[2 * h + 1] = __uint_as_float(raw[st][h] & 0xffff0000u);
    }
#pragma unroll
    for (int jt = 0; jt < JT; ++jt) {
      const float c = cl[4 * st + k][16 * jt + n];
#pragma unroll
      for (int e = 0; e < 8; ++e)
        acc[jt][e] = __builtin_amdgcn_mfma_f32_16x16x4f32(c, v[e], acc[jt][e], 0, 0, 0);
    }
  }
  if (!live) return;
  float* out = args.part[job] + static_cast<int64_t>(slot) * P * r_max;
#pragma unroll
  for (int jt = 0; jt < JT; ++jt) {
    const int j0 = 16 * jt + 4 * k;  // this lane's rows j0 .. j0 + 3
    if (j0 >= r_max) continue;
    if (job & 1) {  // [r_max][P]: 8 consecutive columns per row
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        float* o = out + static_cast<int64_t>(j0 + i) * P + col;
        *reinterpret_cast<f32x4*>(o) =
            f32x4{acc[jt][0][i], acc[jt][1][i], acc[jt][2][i], acc[jt][3][i]};
        *reinterpret_cast<f32x4*>(o + 4) =
            f32x4{acc[jt][4][i], acc[jt][5][i], acc[jt][6][i], acc[jt][7][i]};
      }
    } else {  // [P][r_max]: 4 consecutive rows per column
#pragma unroll
      for (int e = 0; e < 8; ++e)
        *reinterpret_cast<f32x4*>(out + (col + e) * r_max + j0) = acc[jt][e];
    }
  }
}

// ---- out[a][e .. e+4) = sum of the partial sums of a's units, in unit
// order, for e < E = P * r_max; 0 for an adapter without tokens and at or
// past its rank. blockIdx.z = job as for the outer products.
struct ReduceArgs {
  const float* part[kGrJobs];
  float* out[kGrJobs];
  int64_t P[kGrJobs];
  const int32_t* ranks[kGrJobs];
};

__global__ __launch_bounds__(kGrThreads) void grad_reduce_kernel(
    ReduceArgs args, int r_max, const int32_t* __restrict__ useg) {
  const int job = blockIdx.z;
  const int a = blockIdx.y;
  const int64_t P = args.P[job];
  const int64_t E = P * r_max;
  const int64_t e = (static_cast<int64_t>(blockIdx.x) * kGrThreads + threadIdx.x) * 4;
  if (e >= E) return;
  const int u0 = useg[a], nu = useg[a + 1] - u0;
  const int32_t* ranks = args.ranks[job];
  const int rk = ranks ? min(max(ranks[a], 0), r_max) : r_max;
  const float* part = args.part[job];
  f32x4 sum{0.f, 0.f, 0.f, 0.f};
  int u = 0;
  for (; u + 4 <= nu; u += 4) {  // four loads in flight, added in unit order
    f32x4 v[4];
#pragma unroll
    for (int q = 0; q < 4; ++q)
      v[q] = *reinterpret_cast<const f32x4*>(part + static_cast<int64_t>(u0 + u + q) * E + e);
#pragma unroll
    for (int q = 0; q < 4; ++q) sum += v[q];
  }
  for (; u < nu; ++u)
    sum += *reinterpret_cast<const f32x4*>(part + static_cast<int64_t>(u0 + u) * E + e);
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int j = (job & 1) ? static_cast<int>((e + q) / P) : static_cast<int>((e + q) % r_max);
    if (j >= rk) sum[q] = 0.f;
  }
  *reinterpret_cast<f32x4*>(args.out[job] + static_cast<int64_t>(a) * E + e) = sum;
}

local_status_t launch_outer(const OuterArgs& o, int n_jobs, int64_t T, int r_max,
                            const int32_t* perm, const int32_t* useg, const i32x4* utab,
                            int n_ad, int64_t units, const float* scale, hipStream_t s) {
  int64_t pmax = 0;
  for (int q = 0; q < n_jobs; ++q) pmax = std::max(pmax, o.P[q]);
  auto go = [&](auto kernel, int64_t cols_per_wg) {
    const int64_t ptiles = (pmax + cols_per_wg - 1) / cols_per_wg;
    kernel<<<dim3(static_cast<unsigned>(units * ptiles), static_cast<unsigned>(n_jobs)),
             kGrThreads, 0, s>>>(o, T, ptiles, r_max, perm, useg, utab, n_ad, scale);
    return local_check_launch("lora_grad (outer)");
  };
  if (r_max <= 16) return go(grad_outer_mfma_kernel<1>, 512);
  if (r_max <= 32) return go(grad_outer_mfma_kernel<2>, 512);
  if (r_max <= 64) return go(grad_outer_mfma_kernel<4>, 512);
  return go(grad_outer_kernel<1, 128>, kGrThreads);
}

local_status_t grad_checks(const char* who, int64_t T, int64_t K, int64_t N, int32_t n_ad,
                           int32_t r_max) {
  if (T < 0 || K <= 0 || N <= 0 || n_ad < 1)
    return local_fail(LOCAL_ERR_SHAPE, "%s: T=%lld K=%lld N=%lld n_adapters=%d", who,
                      (long long)T, (long long)K, (long long)N, n_ad);
  if (K % 64 || N % 64 || n_ad > kGrMaxAdapters || r_max < 8 || r_max > 128 || r_max % 8)
    return local_fail(LOCAL_ERR_UNSUPPORTED,
                      "%s: K=%lld N=%lld n_adapters=%d r_max=%d (need K, N %% 64 == 0, "
                      "n_adapters <= 256, r_max in [8,128] and %% 8 == 0)",
                      who, (long long)K, (long long)N, n_ad, r_max);
  return LOCAL_OK;
}

}  // namespace
}  // namespace localk

using namespace localk;

namespace localk {
namespace {

// Adapter gradients of G projections that share x (and the routing).
local_status_t grad_impl(const char* who, const uint16_t* x, int64_t T, int64_t K, int G,
                         const uint16_t* const* dy, const int64_t* N, const uint16_t* const* A,
                         const uint16_t* const* B, int32_t n_adapters, int32_t r_max,
                         const int32_t* const* ranks, const int32_t* adapter_idx,
                         const float* scale, float* const* dA, float* const* dB, void* ws,
                         size_t* ws_bytes, hipStream_t s) {
  if (!ws_bytes) return local_fail(LOCAL_ERR_WORKSPACE, "%s: ws_bytes is NULL", who);
  if (G < 1 || G > kGrGroup)
    return local_fail(LOCAL_ERR_UNSUPPORTED, "%s: G=%d (need 1..%d)", who, G, kGrGroup);
  local_status_t st;
  for (int g = 0; g < G; ++g)
    if ((st = grad_checks(who, T, K, N[g], n_adapters, r_max)) != LOCAL_OK) return st;
  const int64_t Tw = T > 0 ? T : 1;
  const int64_t units = Tw / kGrUnit + n_adapters;  // >= sum over adapters of ceil(T_a / 64)
  int ks_x = 0, ks_dy[kGrGroup] = {};
  const size_t sh_x = token_shrink_bytes(Tw, K, r_max, G, &ks_x);
  // workspace: token order, adapter offsets, unit offsets, unit table, B_g^T,
  // the shrinks' partial sums (x against every A_g, dy_g against B_g^T), the
  // partial products of every job
  size_t o = 0;
  auto take = [&](size_t bytes) {
    const size_t at = o;
    o += al256(bytes);
    return at;
  };
  const size_t o_perm = take(static_cast<size_t>(Tw) * 4);
  const size_t o_seg = take(static_cast<size_t>(n_adapters + 1) * 4);
  const size_t o_useg = take(static_cast<size_t>(n_adapters + 1) * 4);
  const size_t o_utab = take(static_cast<size_t>(units) * 16);
  size_t o_bt[kGrGroup], o_shy[kGrGroup], o_pb[kGrGroup], o_pa[kGrGroup];
  for (int g = 0; g < G; ++g) o_bt[g] = take(static_cast<size_t>(n_adapters) * r_max * N[g] * 2);
  const size_t o_shx = take(sh_x);
  for (int g = 0; g < G; ++g) o_shy[g] = take(token_shrink_bytes(Tw, N[g], r_max, 1, &ks_dy[g]));
  for (int g = 0; g < G; ++g) {
    o_pb[g] = take(static_cast<size_t>(units) * N[g] * r_max * 4);
    o_pa[g] = take(static_cast<size_t>(units) * K * r_max * 4);
  }
  if (!ws) {
    *ws_bytes = o;
    return LOCAL_OK;
  }
  if (*ws_bytes < o)
    return local_fail(LOCAL_ERR_WORKSPACE, "%s: workspace %zu < %zu", who, *ws_bytes, o);
  for (int g = 0; g < G; ++g) {
    if (!dA[g] || !dB[g]) return local_fail(LOCAL_ERR_NULL, "%s: NULL output", who);
    if (T > 0 && (!dy[g] || !A[g] || !B[g]))
      return local_fail(LOCAL_ERR_NULL, "%s: NULL pointer argument", who);
  }
  if (T > 0 && (!x || !adapter_idx || !scale))
    return local_fail(LOCAL_ERR_NULL, "%s: NULL pointer argument", who);
  char* w = static_cast<char*>(ws);
  int32_t* perm = reinterpret_cast<int32_t*>(w + o_perm);
  int32_t* seg = reinterpret_cast<int32_t*>(w + o_seg);
  int32_t* useg = reinterpret_cast<int32_t*>(w + o_useg);
  i32x4* utab = reinterpret_cast<i32x4*>(w + o_utab);
  const uint16_t* Bt[kGrGroup];
  // tokens bucketed by adapter and every B_g transposed per adapter to
  // [r_max][N_g], in one launch. T = 0: every adapter is empty and the
  // reduce pass writes zero gradients (no memset: the call stays capturable)
  PrepArgs pr{};
  pr.n_jobs = T > 0 ? G : 0;
  for (int g = 0; g < G; ++g) {
    uint16_t* bt = reinterpret_cast<uint16_t*>(w + o_bt[g]);
    Bt[g] = bt;
    if (T > 0) pr.job[g] = transpose_job(B[g], bt, n_adapters, N[g], r_max);
  }
  pr.idx = adapter_idx ? adapter_idx : reinterpret_cast<const int32_t*>(w);  // not read if T = 0
  pr.T = T;
  pr.n_ad = n_adapters;
  pr.perm = perm;
  pr.seg = seg;
  pr.useg = useg;
  pr.utab = utab;
  if ((st = run_prep(s, pr)) != LOCAL_OK) return st;
  if (T > 0) {
    // u_g = x A_g^T for every g in one pass over x, then dy_g B_g for each g,
    // as the shrink's K-slice partial sums
    if ((st = token_shrink(x, T, K, G, A, n_adapters, r_max, adapter_idx, w + o_shx, s)) !=
        LOCAL_OK)
      return st;
    for (int g = 0; g < G; ++g)
      if ((st = token_shrink(dy[g], T, N[g], 1, &Bt[g], n_adapters, r_max, adapter_idx,
                             w + o_shy[g], s)) != LOCAL_OK)
        return st;
    // dB_g partials from (dy_g, s u_g), dA_g partials from (x, s dy_g B_g)
    OuterArgs oa{};
    for (int g = 0; g < G; ++g) {
      const int32_t* rg = ranks ? ranks[g] : nullptr;
      oa.V[2 * g] = dy[g];
      oa.S[2 * g] = reinterpret_cast<const float*>(w + o_shx) +
                    static_cast<int64_t>(g) * ks_x * T * r_max;
      oa.ks[2 * g] = ks_x;
      oa.part[2 * g] = reinterpret_cast<float*>(w + o_pb[g]);
      oa.P[2 * g] = N[g];
      oa.ranks[2 * g] = rg;
      oa.V[2 * g + 1] = x;
      oa.S[2 * g + 1] = reinterpret_cast<const float*>(w + o_shy[g]);
      oa.ks[2 * g + 1] = ks_dy[g];
      oa.part[2 * g + 1] = reinterpret_cast<float*>(w + o_pa[g]);
      oa.P[2 * g + 1] = K;
      oa.ranks[2 * g + 1] = rg;
    }
    if ((st = launch_outer(oa, 2 * G, T, r_max, perm, useg, utab, n_adapters, units, scale, s)) !=
        LOCAL_OK)
      return st;
  }
  // dB_g [n_ad][N_g][r_max], dA_g [n_ad][r_max][K]
  ReduceArgs ra{};
  int64_t emax = 0;
  for (int g = 0; g < G; ++g) {
    const int32_t* rg = ranks ? ranks[g] : nullptr;
    ra.part[2 * g] = reinterpret_cast<const float*>(w + o_pb[g]);
    ra.out[2 * g] = dB[g];
    ra.P[2 * g] = N[g];
    ra.ranks[2 * g] = rg;
    ra.part[2 * g + 1] = reinterpret_cast<const float*>(w + o_pa[g]);
    ra.out[2 * g + 1] = dA[g];
    ra.P[2 * g + 1] = K;
    ra.ranks[2 * g + 1] = rg;
    emax = std::max(emax, std::max(N[g], K) * r_max);
  }
  grad_reduce_kernel<<<dim3(static_cast<unsigned>((emax / 4 + kGrThreads - 1) / kGrThreads),
                            static_cast<unsigned>(n_adapters), static_cast<unsigned>(2 * G)),
                       kGrThreads, 0, s>>>(ra, r_max, useg);
  return local_check_launch("lora_grad (reduce)");
}

}  // namespace
}  // namespace localk

extern "C" local_status_t local_lora_grad(
    const uint16_t* x, int64_t T, int64_t K, const uint16_t* dy, int64_t N, const uint16_t* A,
    const uint16_t* B, int32_t n_adapters, int32_t r_max, const int32_t* ranks,
    const int32_t* adapter_idx, const float* scale, float* dA, float* dB, void* ws,
    size_t* ws_bytes, void* stream) {
  return grad_impl("lora_grad", x, T, K, 1, &dy, &N, &A, &B, n_adapters, r_max, &ranks,
                   adapter_idx, scale, &dA, &dB, ws, ws_bytes, static_cast<hipStream_t>(stream));
}

extern "C" local_status_t local_lora_grad_grouped(
    const uint16_t* x, int64_t T, int64_t K, int32_t G, const uint16_t* const* dy,
    const int64_t* N, const uint16_t* const* A, const uint16_t* const* B, int32_t n_adapters,
    int32_t r_max, const int32_t* const* ranks, const int32_t* adapter_idx, const float* scale,
    float* const* dA, float* const* dB, void* ws, size_t* ws_bytes, void* stream) {
  if (G < 1 || G > kGrGroup)
    return local_fail(LOCAL_ERR_UNSUPPORTED, "lora_grad_grouped: G=%d (need 1..%d)", G,
                      kGrGroup);
  if (!dy || !N || !A || !B || !dA || !dB)
    return local_fail(LOCAL_ERR_NULL, "lora_grad_grouped: NULL argument array");
  return grad_impl("lora_grad_grouped", x, T, K, G, dy, N, A, B, n_adapters, r_max, ranks,
                   adapter_idx, scale, dA, dB, ws, ws_bytes, static_cast<hipStream_t>(stream));
}

extern "C" local_status_t local_lora_grad_input(
    const uint16_t* dy, int64_t T, int64_t N, const uint16_t* Wt, int64_t K, const uint16_t* A,
    const uint16_t* B, int32_t n_adapters, int32_t r_max, const int32_t* ranks,
    const int32_t* adapter_idx, const float* scale, uint16_t* dx, void* ws, size_t* ws_bytes,
    void* stream) {
  if (!ws_bytes) return local_fail(LOCAL_ERR_WORKSPACE, "lora_grad_input: ws_bytes is NULL");
  local_status_t st = grad_checks("lora_grad_input", T, K, N, n_adapters, r_max);
  if (st != LOCAL_OK) return st;
  // the forward projection of dy: x := dy [T][N], W := W^T [K][N],
  // A := B^T [n][r_max][N], B := A^T [n][K][r_max]
  const size_t o_bt = 0;
  const size_t o_at = o_bt + al256(static_cast<size_t>(n_adapters) * r_max * N * 2);
  const size_t o_fw = o_at + al256(static_cast<size_t>(n_adapters) * K * r_max * 2);
  size_t fw = 0;
  if ((st = local_lora_linear(nullptr, T, N, nullptr, K, nullptr, nullptr, n_adapters, r_max,
                              nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, &fw,
                              stream)) != LOCAL_OK)
    return st;
  const size_t need = o_fw + fw;
  if (!ws) {
    *ws_bytes = need;
    return LOCAL_OK;
  }
  if (*ws_bytes < need)
    return local_fail(LOCAL_ERR_WORKSPACE, "lora_grad_input: workspace %zu < %zu", *ws_bytes,
                      need);
  if (T == 0) return LOCAL_OK;
  if (!dy || !Wt || !A || !B || !adapter_idx || !scale || !dx)
    return local_fail(LOCAL_ERR_NULL, "lora_grad_input: NULL pointer argument");
  hipStream_t s = static_cast<hipStream_t>(stream);
  char* w = static_cast<char*>(ws);
  uint16_t* Bt = reinterpret_cast<uint16_t*>(w + o_bt);
  uint16_t* At = reinterpret_cast<uint16_t*>(w + o_at);
  PrepArgs pr{};
  pr.job[0] = transpose_job(B, Bt, n_adapters, N, r_max);
  pr.job[1] = transpose_job(A, At, n_adapters, r_max, K);
  pr.n_jobs = 2;
  if ((st = run_prep(s, pr)) != LOCAL_OK) return st;
  size_t rest = *ws_bytes - o_fw;
  return local_lora_linear(dy, T, N, Wt, K, Bt, At, n_adapters, r_max, ranks, adapter_idx,
                           scale, nullptr, dx, w + o_fw, &rest, stream);
}
