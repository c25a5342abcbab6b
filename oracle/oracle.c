/*
 * oracle.c — plain CPU reference of the mixed-adapter LoRA step with
 * version-tagged paged attention.
 *
 * TEST INFRASTRUCTURE ONLY. Only the tests, the smoke check and the CPU
 * baseline leg of the benchmark may load this library. It shares no code,
 * header, table or helper with the GPU library and must never serve as its
 * fallback.
 *
 * Every function writes out the plain definition of what the step computes:
 * straight loops, float64 accumulation, no blocking, no fusion, no
 * reordering. Inputs are the exact bf16 values the GPU consumes (uint16
 * storage), decoded exactly to double. OpenMP only distributes independent
 * output rows across threads; each output element is computed by one thread
 * in the order written.
 *
 * KV pool layout (the one the library's interface documents): for physical
 * block p, KV head g, slot s (0..15), dimension d (D = head dim, D % 8 == 0)
 *     K(p,g,s,d) = k_cache[(((p*Hkv + g)*(D/8) + d/8)*16 + s)*8 + d%8]
 *     V(p,g,s,d) = v_cache[((p*Hkv + g)*D + d)*16 + s]
 *
 * Build:  gcc -O2 -std=c11 -fopenmp -shared -fPIC oracle.c -o liboracle.so -lm
 * (no -ffast-math: every sum is evaluated in the order written).
 */
#include <math.h>
#include <stdint.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

#define ORACLE_BS 16

/* bf16 -> double, exact: the bf16 bits are the upper half of a float32. */
static double bf(uint16_t h) {
  uint32_t u = (uint32_t)h << 16;
  float f;
  memcpy(&f, &u, sizeof f);
  return (double)f;
}

static int64_t k_off(int64_t p, int g, int s, int d, int Hkv, int D) {
  return ((((int64_t)p * Hkv + g) * (D / 8) + d / 8) * ORACLE_BS + s) * 8 + d % 8;
}

static int64_t v_off(int64_t p, int g, int s, int d, int Hkv, int D) {
  return (((int64_t)p * Hkv + g) * D + d) * ORACLE_BS + s;
}

int oracle_num_threads(void) {
#ifdef _OPENMP
  return omp_get_max_threads();
#else
  return 1;
#endif
}

/*
 * LoRA projection with per-token adapter routing (§2.2 "LoRA adapters": a
 * frozen base shared by many low-rank adapters, each request routed to its
 * adapter). For token t with adapter a = adapter_idx[t]:
 *   u_j      = sum_k x[t,k] * A[a,j,k]                    (j < rank(a))
 *   y[t,n]   = sum_k x[t,k] * W[n,k] + scale[t] * sum_j u_j * B[a,n,j]
 *              + res[t,n]
 * a < 0 (or n_adapters == 0) leaves the base term alone; res (the layer's
 * residual stream, optional) is added as given.
 * Shapes: x[T][K], W[N][K], A[n_ad][r_max][K], B[n_ad][N][r_max], res and
 * y [T][N].
 */
void oracle_lora_linear(const uint16_t* x, int64_t T, int64_t K,
                        const uint16_t* W, int64_t N,
                        const uint16_t* A, const uint16_t* B,
                        int32_t n_adapters, int32_t r_max,
                        const int32_t* ranks,
                        const int32_t* adapter_idx, const float* scale,
                        const uint16_t* res, double* y) {
#pragma omp parallel for schedule(dynamic, 1)
  for (int64_t t = 0; t < T; ++t) {
    int a = (n_adapters > 0 && adapter_idx) ? adapter_idx[t] : -1;
    if (a >= n_adapters) a = -1; /* outside [0, n_adapters): no adapter */
    int rank = 0;
    double u[256];
    if (a >= 0) {
      rank = ranks ? ranks[a] : r_max;
      if (rank < 0) rank = 0; /* clamped to [0, r_max] */
      if (rank > r_max) rank = r_max;
      for (int j = 0; j < rank; ++j) {
        double acc = 0.0;
        for (int64_t k = 0; k < K; ++k)
          acc += bf(x[t * K + k]) * bf(A[((int64_t)a * r_max + j) * K + k]);
        u[j] = acc;
      }
    }
    for (int64_t n = 0; n < N; ++n) {
      double base = 0.0;
      for (int64_t k = 0; k < K; ++k)
        base += bf(x[t * K + k]) * bf(W[n * K + k]);
      double delta = 0.0;
      for (int j = 0; j < rank; ++j)
        delta += u[j] * bf(B[((int64_t)a * N + n) * r_max + j]);
      double v = base + (a >= 0 ? (double)scale[t] * delta : 0.0);
      if (res) v += bf(res[t * N + n]);
      y[t * N + n] = v;
    }
  }
}

/* Blocks request b owns: ceil(L/16), at most the table's width. */
static int owned_blocks(int L, int max_blocks) {
  if (L <= 0) return 0;
  int nb = (L + ORACLE_BS - 1) / ORACLE_BS;
  return nb < max_blocks ? nb : max_blocks;
}

/* A block is stale when its id is outside the pool or its tag differs from
 * the request's version (the id is then never used to read anything). */
static int block_stale(int p, int64_t num_blocks, const int32_t* block_version,
                       int32_t rv) {
  return p < 0 || p >= num_blocks || block_version[p] != rv;
}

/*
 * Version check (§5.1: KV is reusable only when its validity key — which
 * includes the adapter and the adapter version — matches the request; §1:
 * stale coverage is rejected at lookup). Logical block j of request b is
 * stale iff block_version[block_table[b][j]] != req_version[b]. Writes
 * valid_tokens[b] (live tokens in non-stale blocks), the first min(n, cap)
 * stale (b, j) pairs in (b, j) order, and returns n.
 */
int64_t oracle_block_version_check(const int32_t* block_table, int32_t Bn,
                                   int32_t max_blocks, const int32_t* ctx_lens,
                                   const int32_t* block_version, int64_t num_blocks,
                                   const int32_t* req_version,
                                   int32_t* stale_pairs, int64_t cap,
                                   int32_t* valid_tokens) {
  int64_t n = 0;
  for (int b = 0; b < Bn; ++b) {
    int L = ctx_lens[b];
    int nb = owned_blocks(L, max_blocks);
    int valid = 0;
    for (int j = 0; j < nb; ++j) {
      int p = block_table[(int64_t)b * max_blocks + j];
      int live = L - j * ORACLE_BS;
      if (live > ORACLE_BS) live = ORACLE_BS;
      if (block_stale(p, num_blocks, block_version, req_version[b])) {
        if (n < cap) {
          stale_pairs[2 * n] = b;
          stale_pairs[2 * n + 1] = j;
        }
        ++n;
      } else {
        valid += live;
      }
    }
    valid_tokens[b] = valid;
  }
  return n;
}

/*
 * KV append (§2.2 "KV cache": the key and value of every processed token are
 * stored for later steps). Request b appends rows [q_indptr[b], q_indptr[b+1])
 * of k_new/v_new ([T][Hkv][D]) at logical positions
 * ctx_lens[b] - n_b + i, i < n_b.
 */
void oracle_kv_append(uint16_t* k_cache, uint16_t* v_cache, int32_t Hkv,
                      int32_t D, const int32_t* block_table,
                      int32_t max_blocks, int64_t num_blocks, int32_t Bn,
                      const int32_t* q_indptr, const int32_t* ctx_lens,
                      const uint16_t* k_new, const uint16_t* v_new) {
  for (int b = 0; b < Bn; ++b) {
    int nb_new = q_indptr[b + 1] - q_indptr[b];
    int start = ctx_lens[b] - nb_new;
    for (int i = 0; i < nb_new; ++i) {
      int pos = start + i;
      /* a position without a block, or an id outside the pool: no write */
      if (pos < 0 || pos / ORACLE_BS >= max_blocks) continue;
      int p = block_table[(int64_t)b * max_blocks + pos / ORACLE_BS];
      if (p < 0 || p >= num_blocks) continue;
      int s = pos % ORACLE_BS;
      int64_t row = q_indptr[b] + i;
      for (int g = 0; g < Hkv; ++g)
        for (int d = 0; d < D; ++d) {
          k_cache[k_off(p, g, s, d, Hkv, D)] = k_new[(row * Hkv + g) * D + d];
          v_cache[v_off(p, g, s, d, Hkv, D)] = v_new[(row * Hkv + g) * D + d];
        }
    }
  }
}

/*
 * Paged attention with the per-block version mask (§2.2 "KV cache and prefix
 * caching"; §5.1 validity key). Query row i of request b sits at position
 * P = ctx_lens[b] - n_b + i and attends over
 *   S = { pi <= P, pi/16 < nb_b : logical block pi/16 of b is not stale }
 * with nb_b = min(ceil(ctx_lens[b]/16), max_blocks)
 * with s_pi = sm_scale * <q, K_pi>, out = sum softmax(s)_pi V_pi and
 * lse = log sum exp(s_pi) (natural log). Empty S gives out = 0, lse = -inf.
 * Query head h reads KV head h / (Hq/Hkv). Decode is the case n_b = 1.
 * q[T][Hq][D] bf16 in; out[T][Hq][D] and lse[T][Hq] double out.
 */
void oracle_paged_attn(const uint16_t* q, const int32_t* q_indptr, int32_t Bn,
                       int32_t Hq, int32_t Hkv, int32_t D,
                       const uint16_t* k_cache, const uint16_t* v_cache,
                       const int32_t* block_table, int32_t max_blocks,
                       int64_t num_blocks, const int32_t* ctx_lens,
                       const int32_t* block_version,
                       const int32_t* req_version, double sm_scale,
                       double* out, double* lse) {
  int64_t T = q_indptr[Bn];
  int group = Hq / Hkv;
#pragma omp parallel for collapse(2) schedule(dynamic, 1)
  for (int64_t t = 0; t < T; ++t) {
    for (int h = 0; h < Hq; ++h) {
      int b = 0;
      while (q_indptr[b + 1] <= t) ++b;
      int n_b = q_indptr[b + 1] - q_indptr[b];
      int P = ctx_lens[b] - n_b + (int)(t - q_indptr[b]);
      int nb = owned_blocks(ctx_lens[b], max_blocks);
      if (P > nb * ORACLE_BS - 1) P = nb * ORACLE_BS - 1;
      int g = h / group;
      const uint16_t* qv = q + (t * Hq + h) * D;
      double* o = out + (t * Hq + h) * D;
      /* pass 1: the maximum score over S */
      double m = -INFINITY;
      int64_t count = 0;
      for (int pi = 0; pi <= P; ++pi) {
        int p = block_table[(int64_t)b * max_blocks + pi / ORACLE_BS];
        if (block_stale(p, num_blocks, block_version, req_version[b])) continue;
        double s = 0.0;
        for (int d = 0; d < D; ++d)
          s += bf(qv[d]) * bf(k_cache[k_off(p, g, pi % ORACLE_BS, d, Hkv, D)]);
        s *= sm_scale;
        if (s > m) m = s;
        ++count;
      }
      for (int d = 0; d < D; ++d) o[d] = 0.0;
      if (count == 0) {
        lse[t * Hq + h] = -INFINITY;
        continue;
      }
      /* pass 2: weights exp(s - m), their sum, and the weighted sum of V */
      double denom = 0.0;
      for (int pi = 0; pi <= P; ++pi) {
        int p = block_table[(int64_t)b * max_blocks + pi / ORACLE_BS];
        if (block_stale(p, num_blocks, block_version, req_version[b])) continue;
        double s = 0.0;
        for (int d = 0; d < D; ++d)
          s += bf(qv[d]) * bf(k_cache[k_off(p, g, pi % ORACLE_BS, d, Hkv, D)]);
        s *= sm_scale;
        double w = exp(s - m);
        denom += w;
        for (int d = 0; d < D; ++d)
          o[d] += w * bf(v_cache[v_off(p, g, pi % ORACLE_BS, d, Hkv, D)]);
      }
      for (int d = 0; d < D; ++d) o[d] /= denom;
      lse[t * Hq + h] = m + log(denom);
    }
  }
}

/* bf16 rounding (nearest even) of a double, through float32. Used by the
 * layer-step chain, where every stage's output is bf16 by definition of the
 * interface. NaN is not expected in the oracle's data. */
uint16_t oracle_to_bf16(double v) {
  float f = (float)v;
  uint32_t u;
  memcpy(&u, &f, sizeof u);
  uint32_t lsb = (u >> 16) & 1u;
  u += 0x7fffu + lsb;
  return (uint16_t)(u >> 16);
}

void oracle_to_bf16_array(const double* v, int64_t n, uint16_t* out) {
  for (int64_t i = 0; i < n; ++i) out[i] = oracle_to_bf16(v[i]);
}
