/*
 * Seeded synthetic workload generator.
 *
 * This module produces the inputs of the tree-verification step: fp16
 * normal tensors, int4 group-quantised weights, draft-tree parent arrays and
 * accepted paths.  It is shared by the fp64 reference checker and by the GPU
 * path (inputs are generated on the host and uploaded), and it deliberately
 * holds none of the verification arithmetic: no dequantisation, no matmul,
 * no normalisation, no rotary embedding, no attention and no commit.
 *
 * Random numbers come from a counter-based generator: element i of stream
 * `stream` under seed `seed` is derived from splitmix64 (Steele, Lea and
 * Flood, "Fast splittable pseudorandom number generators", OOPSLA 2014) of a
 * 64-bit counter, so any slice of any tensor can be regenerated
 * independently and in parallel.
 *
 * Normal draws use inverse-CDF sampling on a 16-bit uniform: value =
 * fp16(mean + std * Phi^-1((u + 0.5) / 65536)), with Phi^-1 evaluated in
 * fp64 (Acklam's rational approximation refined by one Halley step against
 * erfc).  The 65536-entry fp16 table makes every draw a table lookup, which
 * keeps the 35 GB full-model workload cheap to produce on the host.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#ifdef _OPENMP
#include <omp.h>
#endif

#define GEN_GOLDEN 0x9E3779B97F4A7C15ULL

static inline uint64_t mix64(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ULL;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBULL;
  return z ^ (z >> 31);
}

/* splitmix64 output for counter value `c` (state = c * golden). */
uint64_t gen_splitmix64_at(uint64_t c) { return mix64(c * GEN_GOLDEN); }

/* Key for (seed, stream): a distinct 64-bit base counter per tensor. */
static inline uint64_t stream_key(uint64_t seed, uint64_t stream) {
  return mix64(seed * 0xD1B54A32D192ED03ULL + mix64(stream + 0x632BE59BD9B4E019ULL));
}

/* ---- fp16 encoding (round to nearest even), generator-local ---------------- */
static uint16_t enc_f16(double x) {
  uint16_t sign = 0;
  if (signbit(x)) { sign = 0x8000; x = -x; }
  if (isnan(x)) return 0x7E00;
  if (x >= 65520.0) return sign | 0x7C00; /* rounds to infinity */
  if (x < ldexp(1.0, -25)) {
    /* below half the smallest subnormal: rounds to zero, except exactly
       2^-25 which ties to even (zero). */
    return sign;
  }
  int e;
  double m = frexp(x, &e); /* x = m * 2^e, m in [0.5, 1) */
  int exp16 = e - 1 + 15;  /* biased exponent for 1.f form */
  if (exp16 <= 0) {
    /* subnormal: value = n * 2^-24 */
    double n = nearbyint(ldexp(x, 24));
    return sign | (uint16_t)n; /* n == 1024 becomes the smallest normal */
  }
  /* normal: 11 significant bits */
  double n = nearbyint(ldexp(m, 11)); /* in [1024, 2048] */
  if (n == 2048.0) { n = 1024.0; exp16 += 1; }
  if (exp16 >= 31) return sign | 0x7C00;
  return sign | (uint16_t)(exp16 << 10) | (uint16_t)((int)n - 1024);
}

static double dec_f16(uint16_t h) {
  int s = h >> 15, e = (h >> 10) & 31, f = h & 1023;
  double v;
  if (e == 0) v = ldexp((double)f, -24);
  else if (e == 31) v = f ? NAN : INFINITY;
  else v = ldexp((double)(f + 1024), e - 25);
  return s ? -v : v;
}

uint16_t gen_f16_from_f64(double x) { return enc_f16(x); }
double gen_f64_from_f16(uint16_t h) { return dec_f16(h); }

/* ---- inverse normal CDF ----------------------------------------------------- */
static double acklam(double p) {
  static const double a[6] = {-3.969683028665376e+01, 2.209460984245205e+02,
                              -2.759285104469687e+02, 1.383577518672690e+02,
                              -3.066479806614716e+01, 2.506628277459239e+00};
  static const double b[5] = {-5.447609879822406e+01, 1.615858368580409e+02,
                              -1.556989798598866e+02, 6.680131188771972e+01,
                              -1.328068155288572e+01};
  static const double c[6] = {-7.784894002430293e-03, -3.223964580411365e-01,
                              -2.400758277161838e+00, -2.549732539343734e+00,
                              4.374664141464968e+00, 2.938163982698783e+00};
  static const double d[4] = {7.784695709041462e-03, 3.224671290700398e-01,
                              2.445134137142996e+00, 3.754408661907416e+00};
  const double plow = 0.02425, phigh = 1 - plow;
  double q, r, x;
  if (p < plow) {
    q = sqrt(-2 * log(p));
    x = (((((c[0] * q + c[1]) * q + c[2]) * q + c[3]) * q + c[4]) * q + c[5]) /
        ((((d[0] * q + d[1]) * q + d[2]) * q + d[3]) * q + 1);
  } else if (p <= phigh) {
    q = p - 0.5;
    r = q * q;
    x = (((((a[0] * r + a[1]) * r + a[2]) * r + a[3]) * r + a[4]) * r + a[5]) * q /
        (((((b[0] * r + b[1]) * r + b[2]) * r + b[3]) * r + b[4]) * r + 1);
  } else {
    q = sqrt(-2 * log(1 - p));
    x = -(((((c[0] * q + c[1]) * q + c[2]) * q + c[3]) * q + c[4]) * q + c[5]) /
        ((((d[0] * q + d[1]) * q + d[2]) * q + d[3]) * q + 1);
  }
  /* one Halley refinement step */
  double e = 0.5 * erfc(-x / sqrt(2.0)) - p;
  double u = e * sqrt(2 * M_PI) * exp(x * x / 2);
  x = x - u / (1 + x * u / 2);
  return x;
}

double gen_normal_quantile(double p) { return acklam(p); }

/* 65536-entry fp16 table of mean + std * Phi^-1((u + 0.5) / 65536). */
void gen_normal_table_f16(double mean, double std, uint16_t* table) {
  for (int u = 0; u < 65536; ++u) {
    double z = acklam(((double)u + 0.5) / 65536.0);
    table[u] = enc_f16(mean + std * z);
  }
}

/* Element i of (seed, stream): 16 uniform bits. */
static inline uint32_t u16_at(uint64_t key, uint64_t i) {
  uint64_t r = mix64((key + (i >> 2)) * GEN_GOLDEN + 0x2545F4914F6CDD1DULL);
  return (uint32_t)(r >> (16 * (i & 3))) & 0xFFFFu;
}

/* out[j] = N(mean, std) draw number (offset + j) of (seed, stream), fp16. */
void gen_normal_f16(uint64_t seed, uint64_t stream, uint64_t offset, int64_t n,
                    double mean, double std, uint16_t* out) {
  uint16_t* table = (uint16_t*)malloc(65536 * sizeof(uint16_t));
  gen_normal_table_f16(mean, std, table);
  uint64_t key = stream_key(seed, stream);
#pragma omp parallel for schedule(static)
  for (int64_t j = 0; j < n; ++j) out[j] = table[u16_at(key, offset + (uint64_t)j)];
  free(table);
}

/* ---- int4 group quantiser (min/max asymmetric, group 128) ------------------- */
/* Per (row n, group g): s = fp16((max - min) / 15) (1.0 if zero),
 * z = clamp(rne(-min / s), 0, 15), q = clamp(rne(w / s) + z, 0, 15).
 * Packing: qweight[n][k/2], low nibble = even k, high nibble = odd k.
 * scales[n][K/128] fp16, zeros[n][K/128] u8. */
static void quantize_row(const uint16_t* w, int64_t K, uint8_t* qrow, uint16_t* srow,
                         uint8_t* zrow) {
  int64_t G = K / 128;
  for (int64_t g = 0; g < G; ++g) {
    const uint16_t* wg = w + g * 128;
    double mn = dec_f16(wg[0]), mx = mn;
    for (int i = 1; i < 128; ++i) {
      double v = dec_f16(wg[i]);
      if (v < mn) mn = v;
      if (v > mx) mx = v;
    }
    uint16_t sh = enc_f16((mx - mn) / 15.0);
    double s = dec_f16(sh);
    if (s == 0.0) { sh = 0x3C00; s = 1.0; }
    double zf = nearbyint(-mn / s);
    if (zf < 0) zf = 0;
    if (zf > 15) zf = 15;
    int z = (int)zf;
    srow[g] = sh;
    zrow[g] = (uint8_t)z;
    for (int i = 0; i < 128; i += 2) {
      int qv[2];
      for (int t = 0; t < 2; ++t) {
        double qf = nearbyint(dec_f16(wg[i + t]) / s) + z;
        if (qf < 0) qf = 0;
        if (qf > 15) qf = 15;
        qv[t] = (int)qf;
      }
      qrow[(g * 128 + i) / 2] = (uint8_t)(qv[0] | (qv[1] << 4));
    }
  }
}

/* Quantise an existing fp16 matrix w[N][K] (K % 128 == 0). */
void gen_quantize_w4(const uint16_t* w, int64_t N, int64_t K, uint8_t* qweight,
                     uint16_t* scales, uint8_t* zeros) {
#pragma omp parallel for schedule(static)
  for (int64_t n = 0; n < N; ++n)
    quantize_row(w + n * K, K, qweight + n * (K / 2), scales + n * (K / 128),
                 zeros + n * (K / 128));
}

/* Draw w[N][K] ~ N(0, std) fp16 from (seed, stream) and quantise it row by
 * row without materialising the fp16 matrix.  Row n uses draws
 * [n*K, (n+1)*K) of the stream, so the result equals gen_normal_f16 followed
 * by gen_quantize_w4.  row0/nrows select a slab of rows. */
void gen_w4_random(uint64_t seed, uint64_t stream, int64_t K, double std, int64_t row0,
                   int64_t nrows, uint8_t* qweight, uint16_t* scales, uint8_t* zeros) {
  uint16_t* table = (uint16_t*)malloc(65536 * sizeof(uint16_t));
  gen_normal_table_f16(0.0, std, table);
  uint64_t key = stream_key(seed, stream);
#pragma omp parallel
  {
    uint16_t* row = (uint16_t*)malloc((size_t)K * sizeof(uint16_t));
#pragma omp for schedule(static)
    for (int64_t r = 0; r < nrows; ++r) {
      uint64_t base = (uint64_t)(row0 + r) * (uint64_t)K;
      for (int64_t k = 0; k < K; ++k) row[k] = table[u16_at(key, base + (uint64_t)k)];
      quantize_row(row, K, qweight + r * (K / 2), scales + r * (K / 128), zeros + r * (K / 128));
    }
    free(row);
  }
  free(table);
}

/* ---- draft trees -------------------------------------------------------------- */
typedef struct { uint64_t s; } rng_t;
static inline uint64_t rng_next(rng_t* r) { r->s += GEN_GOLDEN; return mix64(r->s); }
static inline int rng_below(rng_t* r, int n) {
  return (int)(((unsigned __int128)rng_next(r) * (unsigned)n) >> 64);
}

/* Random draft tree with T nodes and exactly `levels` levels (the longest
 * root-to-leaf path has `levels` nodes), at most `branching` children per
 * node.  Build a spine of `levels` nodes, hang the remaining nodes on
 * uniformly chosen eligible parents (level < levels-1, fewer than
 * `branching` children), then relabel in a uniformly random topological
 * order so that parent[0] = -1 and 0 <= parent[i] < i.
 * Returns 0, or -1 if the shape is infeasible. */
int gen_tree(int T, int levels, int branching, uint64_t seed, int32_t* parent_out) {
  if (T < 1 || levels < 1 || levels > T || T > 4096) return -1;
  if (branching < 1 && T > 1) return -1;
  int* par = (int*)malloc(sizeof(int) * T);
  int* lvl = (int*)malloc(sizeof(int) * T);
  int* nch = (int*)calloc(T, sizeof(int));
  int* elig = (int*)malloc(sizeof(int) * T);
  int* order = (int*)malloc(sizeof(int) * T);
  int* newid = (int*)malloc(sizeof(int) * T);
  int* avail = (int*)malloc(sizeof(int) * T);
  rng_t r = {mix64(seed ^ 0x7472656547454E31ULL)};
  int rc = 0;
  for (int i = 0; i < levels; ++i) {
    par[i] = i - 1;
    lvl[i] = i;
    if (i > 0) nch[i - 1]++;
  }
  for (int i = levels; i < T; ++i) {
    int ne = 0;
    for (int j = 0; j < i; ++j)
      if (lvl[j] < levels - 1 && nch[j] < branching) elig[ne++] = j;
    if (ne == 0) { rc = -1; goto done; }
    int p = elig[rng_below(&r, ne)];
    par[i] = p;
    lvl[i] = lvl[p] + 1;
    nch[p]++;
  }
  /* random topological relabelling */
  {
    int na = 0, placed = 0;
    char* done_ = (char*)calloc(T, 1);
    avail[na++] = 0;
    while (na > 0) {
      int pick = rng_below(&r, na);
      int v = avail[pick];
      avail[pick] = avail[--na];
      order[placed] = v;
      newid[v] = placed++;
      done_[v] = 1;
      for (int c = 0; c < T; ++c)
        if (par[c] == v) avail[na++] = c;
    }
    free(done_);
    if (placed != T) { rc = -1; goto done; }
    for (int i = 0; i < T; ++i) {
      int v = order[i];
      parent_out[i] = par[v] < 0 ? -1 : newid[par[v]];
    }
  }
done:
  free(par); free(lvl); free(nch); free(elig); free(order); free(newid); free(avail);
  return rc;
}

/* Pick the accepted node: a uniformly random leaf, or (deepest_only) a
 * uniformly random leaf among those of maximal depth.  Returns the node. */
int gen_accept_leaf(const int32_t* parent, int T, uint64_t seed, int deepest_only) {
  int* depth = (int*)malloc(sizeof(int) * T);
  char* has_child = (char*)calloc(T, 1);
  int* cand = (int*)malloc(sizeof(int) * T);
  int maxd = 0;
  for (int i = 0; i < T; ++i) {
    depth[i] = parent[i] < 0 ? 0 : depth[parent[i]] + 1;
    if (depth[i] > maxd) maxd = depth[i];
    if (parent[i] >= 0) has_child[parent[i]] = 1;
  }
  int nc = 0;
  for (int i = 0; i < T; ++i)
    if (!has_child[i] && (!deepest_only || depth[i] == maxd)) cand[nc++] = i;
  rng_t r = {mix64(seed ^ 0x70617468534545ULL)};
  int leaf = nc ? cand[rng_below(&r, nc)] : 0;
  free(depth); free(has_child); free(cand);
  return leaf;
}

/* Uniform 64-bit words (for tests that need raw random bytes). */
void gen_u64(uint64_t seed, uint64_t stream, uint64_t offset, int64_t n, uint64_t* out) {
  uint64_t key = stream_key(seed, stream);
#pragma omp parallel for schedule(static)
  for (int64_t j = 0; j < n; ++j) out[j] = mix64((key ^ 0xA5A5A5A5ULL) + (offset + (uint64_t)j) * GEN_GOLDEN);
}

int gen_num_threads(void) {
#ifdef _OPENMP
  return omp_get_max_threads();
#else
  return 1;
#endif
}
