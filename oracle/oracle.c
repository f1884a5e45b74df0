/*
 * fp64 reference checker for the tree-verification step (TEST INFRASTRUCTURE).
 * See oracle.h for the contract.  Only the test-suite, the smoke check and
 * the benchmark's CPU-baseline leg use this file; the product path never
 * does.  Plain loops in the order of the definitions; OpenMP only spreads
 * independent outputs over threads and never changes any summation order.
 */
#include "oracle.h"

#include <math.h>
#include <stdlib.h>
#include <string.h>

#ifdef _OPENMP
#include <omp.h>
#endif

int oracle_num_threads(void) {
#ifdef _OPENMP
  return omp_get_max_threads();
#else
  return 1;
#endif
}

/* Threads of later parallel regions (timing only: results do not depend on it). */
void oracle_set_num_threads(int n) {
#ifdef _OPENMP
  if (n > 0) omp_set_num_threads(n);
#else
  (void)n;
#endif
}

/* ---------------------------------------------------------------- binary16 */

double oracle_f16_to_f64(uint16_t h) {
  int sign = (h >> 15) & 1;
  int expo = (h >> 10) & 0x1F;
  int frac = h & 0x3FF;
  double mag;
  if (expo == 0x1F) {
    mag = frac ? NAN : INFINITY;
  } else if (expo == 0) {
    mag = (double)frac / 16777216.0; /* frac * 2^-24 */
  } else {
    mag = ldexp(1.0 + (double)frac / 1024.0, expo - 15);
  }
  return sign ? -mag : mag;
}

/* Round a double to binary16, nearest-even, by working on its bit pattern. */
uint16_t oracle_f64_to_f16(double x) {
  uint64_t b;
  memcpy(&b, &x, sizeof b);
  uint16_t sign = (uint16_t)((b >> 48) & 0x8000u);
  int e = (int)((b >> 52) & 0x7FF);
  uint64_t m = b & ((1ULL << 52) - 1);
  if (e == 0x7FF) return sign | (m ? 0x7E00 : 0x7C00);
  if (e == 0) return sign; /* double subnormals are far below binary16 range */
  int E = e - 1023;
  if (E > 15) return sign | 0x7C00;
  uint64_t sig = m | (1ULL << 52); /* 53-bit significand, value = sig * 2^(E-52) */
  int normal = E >= -14;
  int shift = normal ? 42 : 42 + (-14 - E);
  if (shift > 60) return sign;
  uint64_t kept = sig >> shift;
  uint64_t rem = sig & ((1ULL << shift) - 1);
  uint64_t half = 1ULL << (shift - 1);
  if (rem > half || (rem == half && (kept & 1))) kept++;
  if (normal) {
    int be = E + 15;
    if (kept == 2048) { kept = 1024; be++; }
    if (be >= 31) return sign | 0x7C00;
    return sign | (uint16_t)(be << 10) | (uint16_t)(kept - 1024);
  }
  return sign | (uint16_t)kept; /* kept == 1024 encodes the smallest normal */
}

static double* f16_rows_to_f64(const uint16_t* x, int32_t M, int32_t Kc, int32_t ldx) {
  double* out = (double*)malloc(sizeof(double) * (size_t)M * Kc);
  for (int32_t m = 0; m < M; ++m)
    for (int32_t k = 0; k < Kc; ++k) out[(size_t)m * Kc + k] = oracle_f16_to_f64(x[(size_t)m * ldx + k]);
  return out;
}

/* -------------------------------------------------------------------- tree */

int oracle_tree(const int32_t* parent, int32_t T, int32_t* depth, uint8_t* anc) {
  if (T < 1 || parent == NULL) return -1;
  if (parent[0] != -1) return -1;
  for (int32_t i = 1; i < T; ++i)
    if (parent[i] < 0 || parent[i] >= i) return -1;
  for (int32_t i = 0; i < T; ++i) {
    if (anc) memset(anc + (size_t)i * T, 0, (size_t)T);
    int32_t d = 0;
    for (int32_t j = i; j != -1; j = parent[j]) {
      if (anc) anc[(size_t)i * T + j] = 1;
      if (j != i) d++;
    }
    if (depth) depth[i] = d;
  }
  return 0;
}

/* ----------------------------------------------------------------- weights */

double oracle_dequant(const uint8_t* qweight, const uint16_t* scales, const uint8_t* zeros,
                      int32_t K, int32_t n, int32_t k) {
  uint8_t byte = qweight[(size_t)n * (K / 2) + k / 2];
  int qv = (k % 2 == 0) ? (byte & 0x0F) : (byte >> 4);
  size_t gi = (size_t)n * (K / 128) + k / 128;
  double s = oracle_f16_to_f64(scales[gi]);
  return (double)(qv - (int)zeros[gi]) * s;
}

/* y64[m][n] = sum_k x64[m][k] * W'[n][k], summed in increasing k. */
static void w4_matmul_f64(const uint8_t* q, const uint16_t* s, const uint8_t* z, int32_t K,
                          int32_t N, const double* x64, int32_t M, double* y64) {
  /* x transposed so the M independent sums advance together over k */
  double* xT = (double*)malloc(sizeof(double) * (size_t)K * M);
  for (int32_t m = 0; m < M; ++m)
    for (int32_t k = 0; k < K; ++k) xT[(size_t)k * M + m] = x64[(size_t)m * K + k];
#pragma omp parallel
  {
    double* w = (double*)malloc(sizeof(double) * (size_t)K);
    double* acc = (double*)malloc(sizeof(double) * (size_t)M);
#pragma omp for schedule(static)
    for (int32_t n = 0; n < N; ++n) {
      for (int32_t k = 0; k < K; ++k) w[k] = oracle_dequant(q, s, z, K, n, k);
      for (int32_t m = 0; m < M; ++m) acc[m] = 0.0;
      for (int32_t k = 0; k < K; ++k) {
        const double wk = w[k];
        const double* xk = xT + (size_t)k * M;
        for (int32_t m = 0; m < M; ++m) acc[m] += xk[m] * wk;
      }
      for (int32_t m = 0; m < M; ++m) y64[(size_t)m * N + n] = acc[m];
    }
    free(w);
    free(acc);
  }
  free(xT);
}

int oracle_w4a16_gemm(const uint8_t* qweight, const uint16_t* scales, const uint8_t* zeros,
                      int32_t K, int32_t N, const uint16_t* x, int32_t M, int32_t ldx,
                      const uint16_t* residual, int32_t ldr, uint16_t* y, int32_t ldy) {
  if (K <= 0 || K % 128 || N <= 0 || M < 0 || ldx < K || ldy < N) return -1;
  if (M == 0) return 0;
  double* x64 = f16_rows_to_f64(x, M, K, ldx);
  double* y64 = (double*)malloc(sizeof(double) * (size_t)M * N);
  w4_matmul_f64(qweight, scales, zeros, K, N, x64, M, y64);
  for (int32_t m = 0; m < M; ++m)
    for (int32_t n = 0; n < N; ++n) {
      double v = y64[(size_t)m * N + n];
      if (residual) v += oracle_f16_to_f64(residual[(size_t)m * ldr + n]);
      y[(size_t)m * ldy + n] = oracle_f64_to_f16(v);
    }
  free(x64);
  free(y64);
  return 0;
}

static double silu(double g) { return g / (1.0 + exp(-g)); }

int oracle_w4a16_swiglu(const uint8_t* qg, const uint16_t* sg, const uint8_t* zg,
                        const uint8_t* qu, const uint16_t* su, const uint8_t* zu, int32_t K,
                        int32_t N, const uint16_t* x, int32_t M, int32_t ldx, uint16_t* y,
                        int32_t ldy) {
  if (K <= 0 || K % 128 || N <= 0 || M < 0 || ldx < K || ldy < N) return -1;
  if (M == 0) return 0;
  double* x64 = f16_rows_to_f64(x, M, K, ldx);
  double* g64 = (double*)malloc(sizeof(double) * (size_t)M * N);
  double* u64 = (double*)malloc(sizeof(double) * (size_t)M * N);
  w4_matmul_f64(qg, sg, zg, K, N, x64, M, g64);
  w4_matmul_f64(qu, su, zu, K, N, x64, M, u64);
  for (int32_t m = 0; m < M; ++m)
    for (int32_t n = 0; n < N; ++n) {
      size_t i = (size_t)m * N + n;
      y[(size_t)m * ldy + n] = oracle_f64_to_f16(silu(g64[i]) * u64[i]);
    }
  free(x64);
  free(g64);
  free(u64);
  return 0;
}

/* ----------------------------------------------------------------- RMSNorm */

int oracle_rmsnorm(const uint16_t* x, int32_t M, int32_t H, int32_t ldx, const uint16_t* gamma,
                   double eps, uint16_t* out, int32_t ldo) {
  if (H <= 0 || M < 0 || ldx < H || ldo < H) return -1;
  for (int32_t m = 0; m < M; ++m) {
    double ss = 0.0;
    for (int32_t k = 0; k < H; ++k) {
      double v = oracle_f16_to_f64(x[(size_t)m * ldx + k]);
      ss += v * v;
    }
    double inv = 1.0 / sqrt(ss / (double)H + eps);
    for (int32_t k = 0; k < H; ++k) {
      double v = oracle_f16_to_f64(x[(size_t)m * ldx + k]);
      out[(size_t)m * ldo + k] = oracle_f64_to_f16(v * inv * oracle_f16_to_f64(gamma[k]));
    }
  }
  return 0;
}

/* -------------------------------------------------------------------- RoPE */

void oracle_rope(double* vec, int32_t D, int64_t pos, double theta) {
  int32_t half = D / 2;
  for (int32_t d = 0; d < half; ++d) {
    double inv_freq = pow(theta, -2.0 * (double)d / (double)D);
    double ang = (double)pos * inv_freq;
    double c = cos(ang), s = sin(ang);
    double a = vec[d], b = vec[d + half];
    vec[d] = a * c - b * s;
    vec[d + half] = b * c + a * s;
  }
}

/* --------------------------------------------------------------- attention */

int oracle_tree_attention(const uint16_t* q, int32_t ldq, const uint16_t* k, const uint16_t* v,
                          int32_t ldkv, uint16_t* k_cache, uint16_t* v_cache, int32_t S_max,
                          int32_t P, const int32_t* parent, int32_t T, int32_t Hq, int32_t Hkv,
                          int32_t D, double rope_theta, double softmax_scale, uint16_t* out,
                          int32_t ldo) {
  if (T < 1 || Hq < 1 || Hkv < 1 || Hq % Hkv || D < 2 || D % 2 || D > 1024 || P < 0 ||
      P + T > S_max)
    return -1;
  if (ldq < Hq * D || ldkv < Hkv * D || ldo < Hq * D) return -1;
  int32_t* depth = (int32_t*)malloc(sizeof(int32_t) * T);
  uint8_t* anc = (uint8_t*)malloc((size_t)T * T);
  if (oracle_tree(parent, T, depth, anc) != 0) {
    free(depth);
    free(anc);
    return -1;
  }
  /* 1. tree keys and values enter the cache at rows P + i: key rotated at
        position P + depth(i) and rounded to fp16, value copied */
  for (int32_t g = 0; g < Hkv; ++g)
    for (int32_t i = 0; i < T; ++i) {
      double kv[1024];
      for (int32_t d = 0; d < D; ++d) kv[d] = oracle_f16_to_f64(k[(size_t)i * ldkv + g * D + d]);
      oracle_rope(kv, D, (int64_t)P + depth[i], rope_theta);
      size_t row = ((size_t)g * S_max + P + i) * D;
      for (int32_t d = 0; d < D; ++d) {
        k_cache[row + d] = oracle_f64_to_f16(kv[d]);
        v_cache[row + d] = v[(size_t)i * ldkv + g * D + d];
      }
    }
  /* 2. each query (head h, node i) attends to prefix rows [0, P) and to the
        tree rows of its ancestors-or-self */
  const int32_t group = Hq / Hkv;
#pragma omp parallel for collapse(2) schedule(dynamic)
  for (int32_t h = 0; h < Hq; ++h)
    for (int32_t i = 0; i < T; ++i) {
      const int32_t g = h / group;
      double qr[1024];
      for (int32_t d = 0; d < D; ++d) qr[d] = oracle_f16_to_f64(q[(size_t)i * ldq + h * D + d]);
      oracle_rope(qr, D, (int64_t)P + depth[i], rope_theta);
      int32_t nkeys = P + T;
      double* sc = (double*)malloc(sizeof(double) * nkeys);
      char* vis = (char*)malloc(nkeys);
      double mx = -INFINITY;
      for (int32_t r = 0; r < nkeys; ++r) {
        vis[r] = r < P ? 1 : anc[(size_t)i * T + (r - P)];
        if (!vis[r]) continue;
        const uint16_t* kr = k_cache + ((size_t)g * S_max + r) * D;
        double dot = 0.0;
        for (int32_t d = 0; d < D; ++d) dot += qr[d] * oracle_f16_to_f64(kr[d]);
        sc[r] = dot * softmax_scale;
        if (sc[r] > mx) mx = sc[r];
      }
      double l = 0.0;
      double o[1024];
      for (int32_t d = 0; d < D; ++d) o[d] = 0.0;
      for (int32_t r = 0; r < nkeys; ++r) {
        if (!vis[r]) continue;
        double p = exp(sc[r] - mx);
        l += p;
        const uint16_t* vr = v_cache + ((size_t)g * S_max + r) * D;
        for (int32_t d = 0; d < D; ++d) o[d] += p * oracle_f16_to_f64(vr[d]);
      }
      for (int32_t d = 0; d < D; ++d) out[(size_t)i * ldo + h * D + d] = oracle_f64_to_f16(o[d] / l);
      free(sc);
      free(vis);
    }
  free(depth);
  free(anc);
  return 0;
}

/* Draft-model attention with a non-square mask (Sec. 3.1, Fig. 4). */
int oracle_draft_tree_attention(const uint16_t* q, int32_t ldq, const uint16_t* k, const uint16_t* v,
                                int32_t ldkv, uint16_t* k_cache, uint16_t* v_cache, int32_t S_max, int32_t P,
                                const int32_t* cache_parent, int32_t N, const int32_t* leaf_parent, int32_t w,
                                int32_t Hq, int32_t Hkv, int32_t D, double rope_theta, double softmax_scale,
                                uint16_t* out, int32_t ldo) {
  if (w < 1 || N < 0 || Hq < 1 || Hkv < 1 || Hq % Hkv || D < 2 || D % 2 || D > 1024 || P < 0 ||
      P + N + w > S_max)
    return -1;
  if (ldq < Hq * D || ldkv < Hkv * D || ldo < Hq * D) return -1;
  for (int32_t j = 0; j < N; ++j)
    if (cache_parent[j] < -1 || cache_parent[j] >= j) return -1;
  for (int32_t i = 0; i < w; ++i)
    if (leaf_parent[i] < -1 || leaf_parent[i] >= N) return -1;
  /* depth of each cached node (a node below the last prefix token has depth
     0, at position P) and of each new token (one more than its parent's) */
  int32_t* cdepth = (int32_t*)malloc(sizeof(int32_t) * (N > 0 ? N : 1));
  for (int32_t j = 0; j < N; ++j) {
    int32_t d = 0;
    for (int32_t u = cache_parent[j]; u != -1; u = cache_parent[u]) d++;
    cdepth[j] = d;
  }
  int32_t* pos = (int32_t*)malloc(sizeof(int32_t) * w);
  for (int32_t i = 0; i < w; ++i) pos[i] = P + (leaf_parent[i] < 0 ? 0 : cdepth[leaf_parent[i]] + 1);
  /* visibility: new token i sees the prefix, the cached nodes on its
     parent's root path (the parent included) and itself */
  uint8_t* vis_cache = (uint8_t*)calloc((size_t)w * (N > 0 ? N : 1), 1);
  for (int32_t i = 0; i < w; ++i)
    for (int32_t u = leaf_parent[i]; u != -1; u = cache_parent[u]) vis_cache[(size_t)i * N + u] = 1;
  /* 1. the new keys and values enter the cache at rows P + N + i */
  for (int32_t g = 0; g < Hkv; ++g)
    for (int32_t i = 0; i < w; ++i) {
      double kv[1024];
      for (int32_t d = 0; d < D; ++d) kv[d] = oracle_f16_to_f64(k[(size_t)i * ldkv + g * D + d]);
      oracle_rope(kv, D, (int64_t)pos[i], rope_theta);
      size_t row = ((size_t)g * S_max + P + N + i) * D;
      for (int32_t d = 0; d < D; ++d) {
        k_cache[row + d] = oracle_f64_to_f16(kv[d]);
        v_cache[row + d] = v[(size_t)i * ldkv + g * D + d];
      }
    }
  /* 2. masked softmax attention per (head, new token) */
  const int32_t group = Hq / Hkv;
#pragma omp parallel for collapse(2) schedule(dynamic)
  for (int32_t h = 0; h < Hq; ++h)
    for (int32_t i = 0; i < w; ++i) {
      const int32_t g = h / group;
      double qr[1024];
      for (int32_t d = 0; d < D; ++d) qr[d] = oracle_f16_to_f64(q[(size_t)i * ldq + h * D + d]);
      oracle_rope(qr, D, (int64_t)pos[i], rope_theta);
      const int32_t nkeys = P + N + w;
      double* sc = (double*)malloc(sizeof(double) * nkeys);
      char* vis = (char*)malloc(nkeys);
      double mx = -INFINITY;
      for (int32_t r = 0; r < nkeys; ++r) {
        vis[r] = r < P ? 1 : r < P + N ? vis_cache[(size_t)i * N + (r - P)] : (r == P + N + i);
        if (!vis[r]) continue;
        const uint16_t* kr = k_cache + ((size_t)g * S_max + r) * D;
        double dot = 0.0;
        for (int32_t d = 0; d < D; ++d) dot += qr[d] * oracle_f16_to_f64(kr[d]);
        sc[r] = dot * softmax_scale;
        if (sc[r] > mx) mx = sc[r];
      }
      double l = 0.0, o[1024];
      for (int32_t d = 0; d < D; ++d) o[d] = 0.0;
      for (int32_t r = 0; r < nkeys; ++r) {
        if (!vis[r]) continue;
        const double p = exp(sc[r] - mx);
        l += p;
        const uint16_t* vr = v_cache + ((size_t)g * S_max + r) * D;
        for (int32_t d = 0; d < D; ++d) o[d] += p * oracle_f16_to_f64(vr[d]);
      }
      for (int32_t d = 0; d < D; ++d) out[(size_t)i * ldo + h * D + d] = oracle_f64_to_f16(o[d] / l);
      free(sc);
      free(vis);
    }
  free(cdepth);
  free(pos);
  free(vis_cache);
  return 0;
}

/* ------------------------------------------------------------------ commit */

int32_t oracle_kv_commit(uint16_t* k_cache, uint16_t* v_cache, int32_t n_layers,
                         int64_t layer_stride, int32_t Hkv, int32_t S_max, int32_t D, int32_t P,
                         const int32_t* parent, int32_t T, int32_t accepted) {
  if (n_layers < 1 || Hkv < 1 || D < 1 || T < 1 || P < 0 || P + T > S_max) return -1;
  if (accepted < 0 || accepted >= T) return -1;
  if (layer_stride < (int64_t)Hkv * S_max * D) return -1;
  if (oracle_tree(parent, T, NULL, NULL) != 0) return -1;
  /* path root -> accepted, obtained by walking parents upward and reversing */
  int32_t* up = (int32_t*)malloc(sizeof(int32_t) * T);
  int32_t L = 0;
  for (int32_t j = accepted; j != -1; j = parent[j]) up[L++] = j;
  int32_t* path = (int32_t*)malloc(sizeof(int32_t) * L);
  for (int32_t i = 0; i < L; ++i) path[i] = up[L - 1 - i];
  uint16_t* snap = (uint16_t*)malloc(sizeof(uint16_t) * (size_t)T * D);
  for (int32_t layer = 0; layer < n_layers; ++layer)
    for (int32_t which = 0; which < 2; ++which) {
      uint16_t* cache = (which ? v_cache : k_cache) + (size_t)layer * layer_stride;
      for (int32_t g = 0; g < Hkv; ++g) {
        uint16_t* tree_rows = cache + ((size_t)g * S_max + P) * D;
        memcpy(snap, tree_rows, sizeof(uint16_t) * (size_t)T * D);
        for (int32_t i = 0; i < L; ++i)
          memcpy(tree_rows + (size_t)i * D, snap + (size_t)path[i] * D, sizeof(uint16_t) * D);
      }
    }
  free(up);
  free(path);
  free(snap);
  return L;
}

/* ------------------------------------------- draft-side KV reorganisation */

int32_t oracle_kv_reorganize(uint16_t* k_cache, uint16_t* v_cache, int32_t n_layers, int64_t layer_stride,
                             int32_t Hkv, int32_t S_max, int32_t D, int32_t P, const int32_t* parent,
                             int32_t N, int32_t last, int32_t keep, int32_t* new_parent, int32_t* n_kept) {
  if (n_layers < 1 || Hkv < 1 || D < 1 || N < 0 || P < 0 || P + N > S_max) return -1;
  if (layer_stride < (int64_t)Hkv * S_max * D) return -1;
  if (last < -1 || last >= N) return -1;
  for (int32_t i = 0; i < N; ++i)
    if (parent[i] < -1 || parent[i] >= i) return -1;
  /* the verified path inside the forest: its root ... last */
  int32_t* order = (int32_t*)malloc(sizeof(int32_t) * (N > 0 ? N : 1));
  int32_t L = 0;
  for (int32_t j = last; j != -1; j = parent[j]) order[L++] = j;
  for (int32_t i = 0; i < L / 2; ++i) {
    const int32_t t = order[i];
    order[i] = order[L - 1 - i];
    order[L - 1 - i] = t;
  }
  /* the subtree below last, in index order (a node is kept when last is
   * one of its ancestors) */
  int32_t S = 0;
  if (keep && last >= 0)
    for (int32_t c = last + 1; c < N; ++c) {
      int32_t below = 0;
      for (int32_t j = parent[c]; j != -1; j = parent[j])
        if (j == last) below = 1;
      if (below) {
        int32_t pos = -1;
        if (parent[c] != last)
          for (int32_t q = 0; q < S; ++q)
            if (order[L + q] == parent[c]) pos = q;
        new_parent[S] = pos;
        order[L + S++] = c;
      }
    }
  uint16_t* snap = (uint16_t*)malloc(sizeof(uint16_t) * (size_t)(N > 0 ? N : 1) * D);
  for (int32_t layer = 0; layer < n_layers; ++layer)
    for (int32_t which = 0; which < 2; ++which) {
      uint16_t* cache = (which ? v_cache : k_cache) + (size_t)layer * layer_stride;
      for (int32_t g = 0; g < Hkv; ++g) {
        uint16_t* tree_rows = cache + ((size_t)g * S_max + P) * D;
        memcpy(snap, tree_rows, sizeof(uint16_t) * (size_t)N * D);
        for (int32_t i = 0; i < L + S; ++i)
          memcpy(tree_rows + (size_t)i * D, snap + (size_t)order[i] * D, sizeof(uint16_t) * D);
      }
    }
  free(order);
  free(snap);
  *n_kept = S;
  return L;
}

/* -------------------------------------------------------- greedy acceptance */

int32_t oracle_greedy_accept(const uint16_t* logits, int32_t T, int32_t V, int32_t ldl,
                             const int32_t* tokens, const int32_t* parent, int32_t* argmax,
                             int32_t* accepted, int32_t* bonus) {
  if (T < 1 || V < 1 || ldl < V) return -1;
  if (oracle_tree(parent, T, NULL, NULL) != 0) return -1;
  /* the target's greedy choice after each node: the first vocabulary index
   * holding the row's largest logit */
  for (int32_t i = 0; i < T; ++i) {
    const uint16_t* row = logits + (size_t)i * ldl;
    int32_t best = 0;
    double bv = oracle_f16_to_f64(row[0]);
    for (int32_t v = 1; v < V; ++v) {
      const double x = oracle_f16_to_f64(row[v]);
      if (x > bv) {
        bv = x;
        best = v;
      }
    }
    argmax[i] = best;
  }
  /* walk from the root: the next accepted node is the lowest-index child
   * whose draft token is the target's choice after the current node */
  int32_t u = 0, L = 1;
  for (;;) {
    int32_t next = -1;
    for (int32_t c = 1; c < T; ++c)
      if (parent[c] == u && tokens[c] == argmax[u]) {
        next = c;
        break;
      }
    if (next < 0) break;
    u = next;
    ++L;
  }
  *accepted = u;
  *bonus = argmax[u];
  return L;
}

/* ------------------------------------------- draft expansion: top-k children */

int32_t oracle_topk_logprobs(const uint16_t* logits, int32_t n, int32_t V, int32_t ldl, int32_t k,
                             int32_t* tokens, double* logprobs) {
  if (n < 0 || V < 1 || ldl < V || k < 1 || k > V) return -1;
  for (int32_t i = 0; i < n; ++i) {
    const uint16_t* row = logits + (size_t)i * ldl;
    /* log-softmax: x - max - log(sum exp(x - max)) */
    double mx = oracle_f16_to_f64(row[0]);
    for (int32_t v = 1; v < V; ++v) {
      const double x = oracle_f16_to_f64(row[v]);
      if (x > mx) mx = x;
    }
    double se = 0.0;
    for (int32_t v = 0; v < V; ++v) se += exp(oracle_f16_to_f64(row[v]) - mx);
    const double lse = mx + log(se);
    /* the k most probable tokens, one at a time: the largest logit not yet
     * taken, the lower index first among equal logits */
    for (int32_t j = 0; j < k; ++j) {
      int32_t best = -1;
      double bv = 0.0;
      for (int32_t v = 0; v < V; ++v) {
        int taken = 0;
        for (int32_t q = 0; q < j; ++q) taken |= tokens[(size_t)i * k + q] == v;
        if (taken) continue;
        const double x = oracle_f16_to_f64(row[v]);
        if (best < 0 || x > bv) {
          best = v;
          bv = x;
        }
      }
      tokens[(size_t)i * k + j] = best;
      logprobs[(size_t)i * k + j] = bv - lse;
    }
  }
  return 0;
}

/* ------------------------------------------------------------------- layer */

int oracle_verify_layer(const oracle_dims* dims, const uint16_t* attn_norm,
                        const uint16_t* mlp_norm, oracle_w4 wqkv, oracle_w4 wo, oracle_w4 wgate,
                        oracle_w4 wup, oracle_w4 wdown, uint16_t* k_cache, uint16_t* v_cache,
                        uint16_t* hidden, int32_t T, int32_t P, const int32_t* parent) {
  const int32_t H = dims->H, Hq = dims->Hq, Hkv = dims->Hkv, D = dims->D, F = dims->F;
  const int32_t Nqkv = (Hq + 2 * Hkv) * D, Hd = Hq * D;
  if (T < 1 || H % 128 || Hd % 128 || F % 128) return -1;
  int rc = 0;
  uint16_t* xn = (uint16_t*)malloc(sizeof(uint16_t) * (size_t)T * H);
  uint16_t* qkv = (uint16_t*)malloc(sizeof(uint16_t) * (size_t)T * Nqkv);
  uint16_t* o = (uint16_t*)malloc(sizeof(uint16_t) * (size_t)T * Hd);
  uint16_t* h = (uint16_t*)malloc(sizeof(uint16_t) * (size_t)T * H);
  uint16_t* hn = (uint16_t*)malloc(sizeof(uint16_t) * (size_t)T * H);
  uint16_t* m = (uint16_t*)malloc(sizeof(uint16_t) * (size_t)T * F);
  rc |= oracle_rmsnorm(hidden, T, H, H, attn_norm, dims->eps, xn, H);
  rc |= oracle_w4a16_gemm(wqkv.q, wqkv.s, wqkv.z, H, Nqkv, xn, T, H, NULL, 0, qkv, Nqkv);
  if (rc == 0)
    rc |= oracle_tree_attention(qkv, Nqkv, qkv + Hd, qkv + Hd + Hkv * D, Nqkv, k_cache, v_cache,
                                dims->S_max, P, parent, T, Hq, Hkv, D, dims->rope_theta,
                                1.0 / sqrt((double)D), o, Hd);
  if (rc == 0) rc |= oracle_w4a16_gemm(wo.q, wo.s, wo.z, Hd, H, o, T, Hd, hidden, H, h, H);
  if (rc == 0) rc |= oracle_rmsnorm(h, T, H, H, mlp_norm, dims->eps, hn, H);
  if (rc == 0)
    rc |= oracle_w4a16_swiglu(wgate.q, wgate.s, wgate.z, wup.q, wup.s, wup.z, H, F, hn, T, H, m, F);
  if (rc == 0) rc |= oracle_w4a16_gemm(wdown.q, wdown.s, wdown.z, F, H, m, T, F, h, H, hidden, H);
  free(xn);
  free(qkv);
  free(o);
  free(h);
  free(hn);
  free(m);
  return rc ? -1 : 0;
}

/* ----------------------------------------------------------------- LM head */

int oracle_lm_head(const uint16_t* h, int32_t M, int32_t H, const uint16_t* gamma, double eps,
                   const uint16_t* W, int32_t V, uint16_t* logits) {
  if (M < 1 || H < 1 || V < 1) return -1;
  uint16_t* hn = (uint16_t*)malloc(sizeof(uint16_t) * (size_t)M * H);
  oracle_rmsnorm(h, M, H, H, gamma, eps, hn, H);
  double* x64 = f16_rows_to_f64(hn, M, H, H);
#pragma omp parallel
  {
    double* w = (double*)malloc(sizeof(double) * (size_t)H);
#pragma omp for schedule(static)
    for (int32_t r = 0; r < V; ++r) {
      for (int32_t k = 0; k < H; ++k) w[k] = oracle_f16_to_f64(W[(size_t)r * H + k]);
      for (int32_t m = 0; m < M; ++m) {
        double acc = 0.0;
        for (int32_t k = 0; k < H; ++k) acc += x64[(size_t)m * H + k] * w[k];
        logits[(size_t)m * V + r] = oracle_f64_to_f16(acc);
      }
    }
    free(w);
  }
  free(hn);
  free(x64);
  return 0;
}
