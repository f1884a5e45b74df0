// Children of the leaves a draft step expands (Sec. 3.1, maximum-likelihood
// tree expansion): per logits row, the k most probable tokens and their
// log-softmax values.
//
// Each row [V] fp16 is split into S contiguous ranges of 16-byte vectors,
// one 256-thread workgroup each (S = 1024 / n, at most 64: about one vector
// per thread at a 128256-entry vocabulary).  Entries are 64-bit sort keys
// (order-preserving logit bits above the inverted index), so a comparison
// of (value, index) pairs is one unsigned compare.  A thread keeps
//   - a descending list of its kTopK best keys (each vector's 8 keys sorted
//     by a bitonic network and merged in), and
//   - an online softmax normaliser (m, s): s = sum exp(x - m) over its
//     values, rescaled whenever m grows.
// Lists and normalisers are merged by butterflies across lanes (bitonic
// merge of two sorted lists per step, all of a step's shuffles independent):
// the wave's 64, then the workgroup's 4 in wave 0, whose lanes publish the
// list and normaliser to workspace slots with agent-scope stores; the last
// workgroup of a row to draw a ticket merges the row's S slots the same way
// (lane = range) and writes token and x - m - log(s) for the first k
// entries.  Merges follow fixed patterns, so results do not depend on
// arrival order.
#include "ss_device.h"
#include "ss_internal.h"

namespace ss {

constexpr int kTopK = 8;        // list length (k <= kTopK)
constexpr int kExpandVecs = 4;  // 16-byte loads in flight per thread

struct TopkArgs {
  const uint16_t* logits;
  int ldl, n, V, k, S, chunk;  // S workgroups per row, each `chunk` 16-byte vectors
  int32_t* tokens;
  float* logprobs;
  void* ws;
  uint64_t* part;   // [n][S][kTopK] sort keys
  uint64_t* stats;  // [n][S] (s bits << 32 | m bits)
};

// Sort key of (fp16 logit h, index): a larger key is a larger logit, or an
// equal logit at a lower index.  The logit's 16 bits are made order-
// preserving (negative values inverted, non-negative ones offset by the
// sign bit, -0 taken as +0); the index is stored inverted below them.
// Key 0 lies below every finite logit and marks an empty entry.
__device__ __forceinline__ uint64_t make_key(uint32_t h, int idx) {
  uint32_t o = (h & 0x8000u) ? (~h & 0xFFFFu) : (h | 0x8000u);
  if (h == 0x8000u) o = 0x8000u;
  return ((uint64_t)o << 32) | (0xFFFFFFFFu - (uint32_t)idx);
}
__device__ __forceinline__ float key_value(uint64_t key) {
  const uint32_t o = (uint32_t)(key >> 32);
  return h2f((uint16_t)((o & 0x8000u) ? (o & 0x7FFFu) : (~o & 0xFFFFu)));
}
__device__ __forceinline__ int key_index(uint64_t key) { return (int)(0xFFFFFFFFu - (uint32_t)key); }

// compare-exchange: afterwards a >= b
__device__ __forceinline__ void cmpx(uint64_t& a, uint64_t& b) {
  const uint64_t hi = a > b ? a : b, lo = a > b ? b : a;
  a = hi;
  b = lo;
}

// The kTopK best of two descending lists: the elementwise larger of `a` and
// reversed `b` is bitonic and holds exactly that set; three half-cleaner
// stages sort it.  Result in `a`.
__device__ __forceinline__ void merge_top(uint64_t (&a)[kTopK], const uint64_t (&b)[kTopK]) {
#pragma unroll
  for (int j = 0; j < kTopK; ++j) a[j] = a[j] > b[kTopK - 1 - j] ? a[j] : b[kTopK - 1 - j];
#pragma unroll
  for (int d = kTopK / 2; d >= 1; d >>= 1)
#pragma unroll
    for (int j = 0; j < kTopK; ++j)
      if ((j & d) == 0) cmpx(a[j], a[j + d]);
}

// Bitonic sorting network, descending.
__device__ __forceinline__ void sort_desc(uint64_t (&a)[kTopK]) {
#pragma unroll
  for (int k = 2; k <= kTopK; k <<= 1)
#pragma unroll
    for (int j = k >> 1; j > 0; j >>= 1)
#pragma unroll
      for (int i = 0; i < kTopK; ++i) {
        const int l = i ^ j;
        if (l > i) {
          if ((i & k) == 0) cmpx(a[i], a[l]);
          else cmpx(a[l], a[i]);
        }
      }
}

// (m, s) pairs: s = sum exp(x - m); an empty pair is (-inf, 0).  lse_combine
// folds (m2, s2) in after (m, s), lse_combine_into before it, so that two
// lanes combining each other's pairs get bit-identical results.
__device__ __forceinline__ void lse_combine(float& m, float& s, float m2, float s2) {
  const float mm = fmaxf(m, m2);
  if (mm == -INFINITY) return;  // both empty
  s = s * __expf(m - mm) + s2 * __expf(m2 - mm);
  m = mm;
}
__device__ __forceinline__ void lse_combine_into(float& m, float& s, float m2, float s2) {
  const float mm = fmaxf(m, m2);
  if (mm == -INFINITY) return;
  s = s2 * __expf(m2 - mm) + s * __expf(m - mm);
  m = mm;
}

// Butterfly over groups of `width` lanes (a power of two up to 64): after
// step `off` each lane holds the kTopK best of its own and lane ^ off's
// lists, and the combined normaliser.  Every lane of a group ends with the
// group's list and normaliser.
__device__ __forceinline__ void butterfly_merge(uint64_t (&L)[kTopK], float& m, float& s, int width) {
  for (int off = 1; off < width; off <<= 1) {
    uint64_t o[kTopK];
#pragma unroll
    for (int j = 0; j < kTopK; ++j) o[j] = shfl_u64(L[j], lane_id() ^ off);
    const float om = __shfl_xor(m, off, kWave), os = __shfl_xor(s, off, kWave);
    merge_top(L, o);
    if (lane_id() & off) lse_combine_into(m, s, om, os);
    else lse_combine(m, s, om, os);
  }
}

__global__ __launch_bounds__(256) void topk_logprobs_kernel(TopkArgs a) {
  __shared__ uint64_t s_key[4][kTopK];
  __shared__ float s_m[4], s_s[4];
  __shared__ int s_last;
  const int row = blockIdx.x / a.S, sp = blockIdx.x % a.S;
  const int tid = threadIdx.x;
  const int lane = lane_id();
  const int wave = tid >> 6;
  const uint16_t* x = a.logits + (size_t)row * a.ldl;
  uint64_t L[kTopK];
#pragma unroll
  for (int j = 0; j < kTopK; ++j) L[j] = 0;
  float m = -INFINITY, s = 0.f;
  auto stat = [&](float v) {
    if (v > m) {
      s = s * __expf(m - v) + 1.0f;
      m = v;
    } else {
      s += __expf(v - m);
    }
  };
  const int nvec = a.V >> 3;
  const int j_lo = min(nvec, sp * a.chunk), j_hi = min(nvec, j_lo + a.chunk);
  for (int j0 = j_lo + tid; j0 < j_hi; j0 += 256 * kExpandVecs) {
    u32x4 w[kExpandVecs];  // all issued before any is used (past the range: its last vector again)
#pragma unroll
    for (int u = 0; u < kExpandVecs; ++u) {
      const int j = min(j0 + 256 * u, j_hi - 1);
      w[u] = *reinterpret_cast<const u32x4*>(x + (size_t)j * 8);
    }
#pragma unroll
    for (int u = 0; u < kExpandVecs; ++u) {
      const int j = j0 + 256 * u;
      if (j >= j_hi) break;
      // one vector: its 8 keys sorted, then merged into the running list
      uint64_t c[kTopK];
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const uint32_t h = (w[u][e >> 1] >> (16 * (e & 1))) & 0xFFFFu;
        c[e] = make_key(h, 8 * j + e);
        stat(h2f((uint16_t)h));
      }
      sort_desc(c);
      merge_top(L, c);
    }
  }
  if (sp == a.S - 1) {  // the columns past the last whole vector (fewer than 8)
    uint64_t c[kTopK];
#pragma unroll
    for (int e = 0; e < kTopK; ++e) c[e] = 0;
    const int i = 8 * nvec + tid;
    if (i < a.V) {
      c[0] = make_key(x[i], i);
      stat(h2f(x[i]));
    }
    merge_top(L, c);
  }

  // the wave's list and normaliser (every lane), then the workgroup's in wave 0
  butterfly_merge(L, m, s, kWave);
  if (lane == 0) {
#pragma unroll
    for (int r = 0; r < kTopK; ++r) s_key[wave][r] = L[r];
    s_m[wave] = m;
    s_s[wave] = s;
  }
  __syncthreads();
  if (wave == 0) {
    uint64_t W[kTopK];
    float wm = -INFINITY, wsum = 0.f;
#pragma unroll
    for (int r = 0; r < kTopK; ++r) W[r] = lane < 4 ? s_key[lane & 3][r] : 0;
    if (lane < 4) {
      wm = s_m[lane];
      wsum = s_s[lane];
    }
    butterfly_merge(W, wm, wsum, 16);  // lanes 0..15 (4..15 empty) all end with the result
    // lane 0 (which holds the whole list, like every lane) publishes the
    // entries and the normaliser and takes the ticket, so that the ticket's
    // release covers every store of the partial
    if (lane == 0) {
      const size_t slot = (size_t)row * a.S + sp;
#pragma unroll
      for (int r = 0; r < kTopK; ++r)
        __hip_atomic_store(a.part + slot * kTopK + r, W[r], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      __hip_atomic_store(a.stats + slot, ((uint64_t)__float_as_uint(wsum) << 32) | __float_as_uint(wm),
                         __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      uint32_t* row_counter = ws_counters(a.ws) + 16 * (1 + row);  // 64 bytes apart
      const bool last = take_ticket(row_counter) == (uint32_t)(a.S - 1);
      if (last) reset_counter(row_counter);  // for the next launch (stream-ordered)
      s_last = last;
    }
  }
  __syncthreads();
  if (!s_last || wave != 0) return;

  // ---- the row's last workgroup, one wave: lane q holds range q ----
  uint64_t R[kTopK];
  float rm = -INFINITY, rs = 0.f;
#pragma unroll
  for (int r = 0; r < kTopK; ++r)
    R[r] = lane < a.S ? __hip_atomic_load(a.part + ((size_t)row * a.S + lane) * kTopK + r, __ATOMIC_RELAXED,
                                          __HIP_MEMORY_SCOPE_AGENT)
                      : 0;
  if (lane < a.S) {
    const uint64_t st = __hip_atomic_load(a.stats + (size_t)row * a.S + lane, __ATOMIC_RELAXED,
                                          __HIP_MEMORY_SCOPE_AGENT);
    rm = __uint_as_float((uint32_t)st);
    rs = __uint_as_float((uint32_t)(st >> 32));
  }
  butterfly_merge(R, rm, rs, kWave);
  const float lse = rm + __logf(rs);
  if (lane < a.k) {
    uint64_t key = R[0];
#pragma unroll
    for (int r = 1; r < kTopK; ++r)
      if (lane == r) key = R[r];
    a.tokens[(size_t)row * a.k + lane] = key_index(key);
    a.logprobs[(size_t)row * a.k + lane] = key_value(key) - lse;
  }
}

int topk_logprobs_splits(int n) {
  int S = 1024 / n;
  return S < 1 ? 1 : S > 64 ? 64 : S;
}

size_t topk_logprobs_part_bytes(int n) {
  return (size_t)n * topk_logprobs_splits(n) * (kTopK + 1) * 8;
}

void launch_topk_logprobs(const uint16_t* logits, int ldl, int n, int V, int k, int32_t* tokens, float* logprobs,
                          void* ws, void* part, hipStream_t st) {
  const int S = topk_logprobs_splits(n);
  const int nvec = V >> 3;
  uint64_t* p = reinterpret_cast<uint64_t*>(part);
  TopkArgs a{logits, ldl, n, V, k, S, (nvec + S - 1) / S, tokens, logprobs, ws, p, p + (size_t)n * S * kTopK};
  hipLaunchKernelGGL(topk_logprobs_kernel, dim3(n * S), dim3(256), 0, st, a);
}

}  // namespace ss
