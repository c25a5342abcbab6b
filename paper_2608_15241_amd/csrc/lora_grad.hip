// local_lora_grad, local_lora_grad_input: the backward of the mixed-adapter
// LoRA projection, for the training chunks that update an agent's adapter
// while the frozen base serves (§2.2: adapters on a frozen base model; §4:
// background training in bounded chunks). With u_t = x_t A_a^T and
// g_t = s_t dy_t B_a (a = a_t, both over a's rank):
//   dB_a = sum_{t of a} s_t dy_t^T u_t,  dA_a = sum_{t of a} g_t^T x_t,
//   dx_t = dy_t W + g_t A_a.
//
// Design (HBM-bound for the adapter gradients: 2 T r (K + N) flop against
// T (K + N) bf16 read):
//  * The tokens are bucketed by adapter (a stable counting sort in one
//    workgroup), as in SGMV.
//  * u and g come from the long-chunk shrink of the forward path: x against
//    A, and dy against B transposed per adapter (a small transpose), then a
//    pass that sums its K slices in order and scales by s_t (tokens without
//    an adapter, and columns at or past the rank, get 0).
//  * dB and dA are segmented outer products: a workgroup per (64 tokens of
//    one adapter, 256 threads x PT columns of dy or x); each thread keeps
//    PT x r_max float32 sums over its tokens, with the tokens' coefficients
//    broadcast from LDS and each token's row read once, coalesced. Partial
//    sums per 64-token unit are added in unit order by a reduce pass:
//    deterministic, no atomics.
//  * dx runs the forward fused projection on the transposed weights: with
//    x := dy, W := W^T, A := B^T and B := A^T, its shrink is dy B and its
//    delta s (dy B) A, so dx needs no kernel of its own.
#include "common.hpp"
#include "lora_internal.hpp"

namespace localk {
namespace {

constexpr int kGrUnit = 64;      // tokens per unit of the segmented products
constexpr int kGrThreads = 256;
constexpr int kGrMaxAdapters = 256;

size_t al256(size_t v) { return (v + 255) & ~static_cast<size_t>(255); }

// ---- tokens bucketed by adapter, stable: perm[seg[a] .. seg[a+1]) holds the
// tokens of adapter a in ascending order; tokens without one are left out.
// One workgroup; the tokens go in passes of 1024, 64 per wave, in order.
__global__ __launch_bounds__(1024) void grad_bucket_kernel(const int32_t* __restrict__ idx,
                                                           int64_t T, int n_ad,
                                                           int32_t* __restrict__ perm,
                                                           int32_t* __restrict__ seg) {
  __shared__ int base[kGrMaxAdapters];
  __shared__ int wcnt[16][kGrMaxAdapters];  // tokens per adapter in each wave of a pass
  const int tid = threadIdx.x, wave = tid / kWave, lane = tid % kWave;
  for (int a = tid; a < n_ad; a += 1024) base[a] = 0;
  __syncthreads();
  for (int64_t t = tid; t < T; t += 1024) {
    const int a = idx[t];
    if (a >= 0 && a < n_ad) atomicAdd(&base[a], 1);
  }
  __syncthreads();
  if (tid == 0) {  // exclusive prefix (n_ad <= 256)
    int run = 0;
    for (int a = 0; a < n_ad; ++a) {
      const int c = base[a];
      seg[a] = run;
      base[a] = run;
      run += c;
    }
    seg[n_ad] = run;
  }
  __syncthreads();
  for (int64_t t0 = 0; t0 < T; t0 += 1024) {
    const int64_t t = t0 + tid;
    const int a = t < T ? idx[t] : -1;
    const int my = (a >= 0 && a < n_ad) ? a : -1;
    for (int e = lane; e < n_ad; e += kWave) wcnt[wave][e] = 0;
    // rank among the wave's earlier lanes of the same adapter, and the
    // wave's count of each adapter present in it
    int rank = 0;
    uint64_t pending = __ballot(my >= 0);
    while (pending) {
      const int ad = __shfl(my, __ffsll(static_cast<long long>(pending)) - 1);
      const uint64_t m = __ballot(my == ad);
      if (my == ad) rank = __popcll(m & ((1ull << lane) - 1ull));
      if (lane == 0) wcnt[wave][ad] = __popcll(m);
      pending &= ~m;
    }
    __syncthreads();
    if (my >= 0) {
      int before = 0;
      for (int w = 0; w < wave; ++w) before += wcnt[w][my];
      perm[base[my] + before + rank] = static_cast<int32_t>(t);
    }
    __syncthreads();
    for (int a2 = tid; a2 < n_ad; a2 += 1024) {
      int c = 0;
      for (int w = 0; w < 16; ++w) c += wcnt[w][a2];
      base[a2] += c;
    }
    __syncthreads();
  }
}

// ---- dst[i][c][r] = src[i][r][c] for n matrices of R x C bf16 (R and C
// multiples of 8), through 64 x 64 LDS tiles: rows read and written whole.
__global__ __launch_bounds__(kGrThreads) void grad_transpose_kernel(
    const uint16_t* __restrict__ src, int64_t R, int64_t C, uint16_t* __restrict__ dst) {
  __shared__ uint16_t tile[64][64 + 2];
  const int64_t i = blockIdx.z;
  const int64_t r0 = static_cast<int64_t>(blockIdx.y) * 64, c0 = static_cast<int64_t>(blockIdx.x) * 64;
  const uint16_t* s = src + i * R * C;
  uint16_t* d = dst + i * R * C;
  for (int e = threadIdx.x; e < 64 * 64; e += kGrThreads) {
    const int rr = e / 64, cc = e % 64;
    if (r0 + rr < R && c0 + cc < C) tile[rr][cc] = s[(r0 + rr) * C + c0 + cc];
  }
  __syncthreads();
  for (int e = threadIdx.x; e < 64 * 64; e += kGrThreads) {
    const int cc = e / 64, rr = e % 64;
    if (r0 + rr < R && c0 + cc < C) d[(c0 + cc) * R + r0 + rr] = tile[rr][cc];
  }
}

// ---- coefficients c[t][j] = s_t * (sum of the shrink's K slices, in order)
// for j below the rank of t's adapter; 0 elsewhere and for tokens without one.
__global__ __launch_bounds__(kGrThreads) void grad_coef_kernel(
    const float* __restrict__ P, int ks, int64_t T, int r_max, const int32_t* __restrict__ idx,
    const float* __restrict__ scale, const int32_t* __restrict__ ranks, int n_ad,
    float* __restrict__ c) {
  const int64_t e = static_cast<int64_t>(blockIdx.x) * kGrThreads + threadIdx.x;
  if (e >= T * r_max) return;
  const int64_t t = e / r_max;
  const int j = static_cast<int>(e % r_max);
  const int a = idx[t];
  float v = 0.f;
  if (a >= 0 && a < n_ad) {
    const int rk = ranks ? min(max(ranks[a], 0), r_max) : r_max;
    if (j < rk) {
      float sum = 0.f;
      for (int z = 0; z < ks; ++z) sum += P[(static_cast<int64_t>(z) * T + t) * r_max + j];
      v = scale[t] * sum;
    }
  }
  c[e] = v;
}

// Adapter and 64-token unit of unit slot k (adapters ascending, units in
// token order), or -1 past the last unit; every lane returns the same.
__device__ int grad_unit(const int32_t* __restrict__ seg, int n_ad, int k, int* unit) {
  const int lane = threadIdx.x % kWave;
  for (int a0 = 0; a0 < n_ad; a0 += kWave) {
    const int a = a0 + lane;
    const int n = a < n_ad ? (seg[a + 1] - seg[a] + kGrUnit - 1) / kGrUnit : 0;
    int incl = n;
#pragma unroll
    for (int off = 1; off < kWave; off <<= 1) {
      const int v = __shfl_up(incl, off);
      if (lane >= off) incl += v;
    }
    const int total = __shfl(incl, kWave - 1);
    if (k < total) {
      const uint64_t m = __ballot(incl > k);
      const int l0 = __ffsll(static_cast<long long>(m)) - 1;
      *unit = k - __shfl(incl - n, l0);
      return a0 + l0;
    }
    k -= total;
  }
  return -1;
}

// ---- segmented outer products. Workgroup = (unit slot, column tile of
// 256 PT columns): partial sums over the unit's tokens of c_t[j] V_t[p] for
// its PT columns per thread. Written per unit slot, [P][r_max] (dB) or
// [r_max][P] (TRANS, dA).
template <int PT, int RJ, bool TRANS>
__global__ __launch_bounds__(kGrThreads) void grad_outer_kernel(
    const uint16_t* __restrict__ V, int64_t P, const float* __restrict__ C, int r_max,
    const int32_t* __restrict__ perm, const int32_t* __restrict__ seg, int n_ad,
    float* __restrict__ part) {
  __shared__ float cl[kGrUnit][RJ];
  __shared__ int tok[kGrUnit];
  const int64_t ptiles = (P + kGrThreads * PT - 1) / (kGrThreads * PT);
  const int slot = static_cast<int>(blockIdx.x / ptiles);
  const int64_t pt = blockIdx.x % ptiles;
  int unit = 0;
  const int a = grad_unit(seg, n_ad, slot, &unit);
  if (a < 0) return;
  const int first = seg[a] + unit * kGrUnit;
  const int nt = min(kGrUnit, seg[a + 1] - first);
  const int tid = threadIdx.x;
  if (tid < nt) tok[tid] = perm[first + tid];
  __syncthreads();
  for (int e = tid; e < kGrUnit * RJ; e += kGrThreads) {
    const int i = e / RJ, j = e % RJ;
    cl[i][j] = (i < nt && j < r_max) ? C[static_cast<int64_t>(tok[i]) * r_max + j] : 0.f;
  }
  __syncthreads();
  const int64_t p0 = (pt * kGrThreads + tid) * PT;
  float acc[PT][RJ];
#pragma unroll
  for (int q = 0; q < PT; ++q)
#pragma unroll
    for (int j = 0; j < RJ; ++j) acc[q][j] = 0.f;
  if (p0 < P) {
    for (int i = 0; i < nt; ++i) {
      const uint16_t* row = V + static_cast<int64_t>(tok[i]) * P + p0;
      float v[PT];
      if constexpr (PT == 4) {
        const u32x2 w = ld_global<u32x2>(row);
        v[0] = __uint_as_float(w.x << 16);
        v[1] = __uint_as_float(w.x & 0xffff0000u);
        v[2] = __uint_as_float(w.y << 16);
        v[3] = __uint_as_float(w.y & 0xffff0000u);
      } else if constexpr (PT == 2) {
        const uint32_t w = ld_global<uint32_t>(row);
        v[0] = __uint_as_float(w << 16);
        v[1] = __uint_as_float(w & 0xffff0000u);
      } else {
        v[0] = __uint_as_float(static_cast<uint32_t>(row[0]) << 16);
      }
#pragma unroll
      for (int j = 0; j < RJ; ++j) {
        const float cj = cl[i][j];
#pragma unroll
        for (int q = 0; q < PT; ++q) acc[q][j] += cj * v[q];
      }
    }
  }
  if (p0 >= P) return;
  float* out = part + static_cast<int64_t>(slot) * P * r_max;
#pragma unroll
  for (int q = 0; q < PT; ++q)
#pragma unroll
    for (int j = 0; j < RJ; ++j)
      if (j < r_max) {
        if (TRANS)
          out[static_cast<int64_t>(j) * P + p0 + q] = acc[q][j];
        else
          out[(p0 + q) * r_max + j] = acc[q][j];
      }
}

// ---- out[a][e] = sum of the partial sums of a's units, in unit order, for
// e < E = P * r_max; 0 for an adapter without tokens and at or past its rank.
__global__ __launch_bounds__(kGrThreads) void grad_reduce_kernel(
    const float* __restrict__ part, int64_t E, int64_t P, int r_max, bool trans,
    const int32_t* __restrict__ seg, int n_ad, const int32_t* __restrict__ ranks,
    float* __restrict__ out) {
  __shared__ int first_unit;
  const int a = blockIdx.y;
  if (threadIdx.x == 0) {
    int u = 0;
    for (int b = 0; b < a; ++b) u += (seg[b + 1] - seg[b] + kGrUnit - 1) / kGrUnit;
    first_unit = u;
  }
  __syncthreads();
  const int64_t e = static_cast<int64_t>(blockIdx.x) * kGrThreads + threadIdx.x;
  if (e >= E) return;
  const int nu = (seg[a + 1] - seg[a] + kGrUnit - 1) / kGrUnit;
  const int j = trans ? static_cast<int>(e / P) : static_cast<int>(e % r_max);
  const int rk = ranks ? min(max(ranks[a], 0), r_max) : r_max;
  float sum = 0.f;
  if (j < rk)
    for (int u = 0; u < nu; ++u) sum += part[static_cast<int64_t>(first_unit + u) * E + e];
  out[static_cast<int64_t>(a) * E + e] = sum;
}

template <bool TRANS>
local_status_t launch_outer(const uint16_t* V, int64_t P, const float* C, int r_max,
                            const int32_t* perm, const int32_t* seg, int n_ad, int64_t units,
                            float* part, hipStream_t s) {
  auto go = [&](auto kernel, int pt) {
    const int64_t ptiles = (P + kGrThreads * pt - 1) / (kGrThreads * pt);
    kernel<<<static_cast<unsigned>(units * ptiles), kGrThreads, 0, s>>>(V, P, C, r_max, perm,
                                                                         seg, n_ad, part);
    return local_check_launch("lora_grad (outer)");
  };
  if (r_max <= 16) return go(grad_outer_kernel<4, 16, TRANS>, 4);
  if (r_max <= 32) return go(grad_outer_kernel<4, 32, TRANS>, 4);
  if (r_max <= 64) return go(grad_outer_kernel<2, 64, TRANS>, 2);
  return go(grad_outer_kernel<1, 128, TRANS>, 1);
}

local_status_t launch_transpose(const uint16_t* src, int64_t n, int64_t R, int64_t C,
                                uint16_t* dst, hipStream_t s) {
  const dim3 grid(static_cast<unsigned>((C + 63) / 64), static_cast<unsigned>((R + 63) / 64),
                  static_cast<unsigned>(n));
  grad_transpose_kernel<<<grid, kGrThreads, 0, s>>>(src, R, C, dst);
  return local_check_launch("lora_grad (transpose)");
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

extern "C" local_status_t local_lora_grad(
    const uint16_t* x, int64_t T, int64_t K, const uint16_t* dy, int64_t N, const uint16_t* A,
    const uint16_t* B, int32_t n_adapters, int32_t r_max, const int32_t* ranks,
    const int32_t* adapter_idx, const float* scale, float* dA, float* dB, void* ws,
    size_t* ws_bytes, void* stream) {
  if (!ws_bytes) return local_fail(LOCAL_ERR_WORKSPACE, "lora_grad: ws_bytes is NULL");
  local_status_t st = grad_checks("lora_grad", T, K, N, n_adapters, r_max);
  if (st != LOCAL_OK) return st;
  const int64_t Tw = T > 0 ? T : 1;
  const int64_t units = Tw / kGrUnit + n_adapters;  // sum over adapters of ceil(T_a / 64)
  int ks_x = 0, ks_dy = 0;
  const size_t sh = std::max(token_shrink_bytes(Tw, K, r_max, &ks_x),
                             token_shrink_bytes(Tw, N, r_max, &ks_dy));
  const size_t o_perm = 0;
  const size_t o_seg = o_perm + al256(static_cast<size_t>(Tw) * 4);
  const size_t o_bt = o_seg + al256(static_cast<size_t>(n_adapters + 1) * 4);
  const size_t o_sh = o_bt + al256(static_cast<size_t>(n_adapters) * r_max * N * 2);
  const size_t o_cu = o_sh + sh;
  const size_t o_cg = o_cu + al256(static_cast<size_t>(Tw) * r_max * 4);
  const size_t o_part = o_cg + al256(static_cast<size_t>(Tw) * r_max * 4);
  const size_t need =
      o_part + al256(static_cast<size_t>(units) * std::max(K, N) * r_max * 4);
  if (!ws) {
    *ws_bytes = need;
    return LOCAL_OK;
  }
  if (*ws_bytes < need)
    return local_fail(LOCAL_ERR_WORKSPACE, "lora_grad: workspace %zu < %zu", *ws_bytes, need);
  if (!dA || !dB) return local_fail(LOCAL_ERR_NULL, "lora_grad: NULL output");
  hipStream_t s = static_cast<hipStream_t>(stream);
  char* w = static_cast<char*>(ws);
  int32_t* perm = reinterpret_cast<int32_t*>(w + o_perm);
  int32_t* seg = reinterpret_cast<int32_t*>(w + o_seg);
  uint16_t* Bt = reinterpret_cast<uint16_t*>(w + o_bt);
  float* cu = reinterpret_cast<float*>(w + o_cu);
  float* cg = reinterpret_cast<float*>(w + o_cg);
  float* part = reinterpret_cast<float*>(w + o_part);
  const int64_t EdB = N * r_max, EdA = static_cast<int64_t>(r_max) * K;
  if (T > 0 && (!x || !dy || !A || !B || !adapter_idx || !scale))
    return local_fail(LOCAL_ERR_NULL, "lora_grad: NULL pointer argument");
  // T = 0: the bucket pass leaves every adapter empty and the reduce pass
  // writes zero gradients (no memset: the call stays capturable)
  grad_bucket_kernel<<<1, 1024, 0, s>>>(adapter_idx, T, n_adapters, perm, seg);
  if ((st = local_check_launch("lora_grad (bucket)")) != LOCAL_OK) return st;
  if (T > 0) {
    // coefficients of dB: s u, u = x A^T
    if ((st = token_shrink(x, T, K, A, n_adapters, r_max, adapter_idx, w + o_sh, s)) != LOCAL_OK)
      return st;
    const unsigned cgrid = static_cast<unsigned>((T * r_max + kGrThreads - 1) / kGrThreads);
    grad_coef_kernel<<<cgrid, kGrThreads, 0, s>>>(reinterpret_cast<const float*>(w + o_sh), ks_x,
                                                  T, r_max, adapter_idx, scale, ranks,
                                                  n_adapters, cu);
    if ((st = local_check_launch("lora_grad (coef)")) != LOCAL_OK) return st;
    // coefficients of dA: g = s dy B, with B transposed per adapter to [r_max][N]
    if ((st = launch_transpose(B, n_adapters, N, r_max, Bt, s)) != LOCAL_OK) return st;
    if ((st = token_shrink(dy, T, N, Bt, n_adapters, r_max, adapter_idx, w + o_sh, s)) !=
        LOCAL_OK)
      return st;
    grad_coef_kernel<<<cgrid, kGrThreads, 0, s>>>(reinterpret_cast<const float*>(w + o_sh),
                                                  ks_dy, T, r_max, adapter_idx, scale, ranks,
                                                  n_adapters, cg);
    if ((st = local_check_launch("lora_grad (coef)")) != LOCAL_OK) return st;
  }
  // dB [n_ad][N][r_max]
  if (T > 0 &&
      (st = launch_outer<false>(dy, N, cu, r_max, perm, seg, n_adapters, units, part, s)) !=
          LOCAL_OK)
    return st;
  grad_reduce_kernel<<<dim3(static_cast<unsigned>((EdB + kGrThreads - 1) / kGrThreads),
                            static_cast<unsigned>(n_adapters)),
                       kGrThreads, 0, s>>>(part, EdB, N, r_max, false, seg, n_adapters, ranks, dB);
  if ((st = local_check_launch("lora_grad (reduce)")) != LOCAL_OK) return st;
  // dA [n_ad][r_max][K]
  if (T > 0 &&
      (st = launch_outer<true>(x, K, cg, r_max, perm, seg, n_adapters, units, part, s)) !=
          LOCAL_OK)
    return st;
  grad_reduce_kernel<<<dim3(static_cast<unsigned>((EdA + kGrThreads - 1) / kGrThreads),
                            static_cast<unsigned>(n_adapters)),
                       kGrThreads, 0, s>>>(part, EdA, K, r_max, true, seg, n_adapters, ranks, dA);
  return local_check_launch("lora_grad (reduce)");
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
  if ((st = launch_transpose(B, n_adapters, N, r_max, Bt, s)) != LOCAL_OK) return st;
  if ((st = launch_transpose(A, n_adapters, r_max, K, At, s)) != LOCAL_OK) return st;
  size_t rest = *ws_bytes - o_fw;
  return local_lora_linear(dy, T, N, Wt, K, Bt, At, n_adapters, r_max, ranks, adapter_idx,
                           scale, nullptr, dx, w + o_fw, &rest, stream);
}
