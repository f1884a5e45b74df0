// Greedy acceptance of a verified draft tree on the device, closing the
// verification step without a host round trip (target-side verification
// with the target's greedy choice: Sec. 3.1 and the Fig. 3 walk-through,
// where each iteration's output is the accepted root path followed by one
// token the target produced after it).
//
// Each logits row [V] fp16 is split into S contiguous ranges of 16-byte
// vectors, one 256-thread workgroup each (S = 1024 / T: about a thousand
// workgroups for any tree size; 8 loads in flight per thread).  A thread
// keeps (value, index) over increasing indices; the wave and the workgroup
// combine pairs (larger value; on equal values the lower index), and the
// pair goes to a workspace slot with an agent-scope store.  Tickets come in
// two levels: the workgroup that draws the last ticket of its row combines
// the row's S pairs in range order (agent-scope loads, so every slot is
// visible whichever XCD wrote it), which gives the first index of the row's
// largest value -- the target's choice after that node -- and takes a ticket
// on the step's counter; the last row to finish walks the tree in one
// wavefront (lane = node): from the root, the next node is the lowest-index
// child whose draft token equals the current node's choice (one ballot per
// step, at most T - 1 steps, each to a higher index), and the node where no
// child matches is accepted; its choice is the bonus token.  At the
// 80-layer shape (T = 64, V = 128256): 10.5 us; one workgroup per row took
// 41 us and a single counter for all 1024 workgroups 19.6 us (the atomics on
// one address serialise).
#include "ss_device.h"
#include "ss_internal.h"

namespace ss {

struct AcceptArgs {
  const uint16_t* logits;
  int ldl, T, V, S, chunk;  // S workgroups per row, each `chunk` 16-byte vectors
  const int32_t* tokens;
  const int32_t* parent;
  int32_t* argmax;
  int32_t* accepted;
  int32_t* bonus;
  int32_t* path_len;
  void* ws;
  uint64_t* part;  // [T][S] (index << 32 | value bits) per workgroup
};

// (v, i) beats (bv, bi): larger value, or equal value at a lower index
__device__ __forceinline__ bool beats(float v, int i, float bv, int bi) { return v > bv || (v == bv && i < bi); }

constexpr int kAcceptVecs = 8;  // 16-byte loads in flight per thread

__global__ __launch_bounds__(256) void greedy_accept_kernel(AcceptArgs a) {
  __shared__ float s_v[4];
  __shared__ int s_i[4];
  __shared__ int s_ticket;
  const int row = blockIdx.x / a.S, sp = blockIdx.x % a.S;
  const int tid = threadIdx.x;
  const int lane = lane_id();
  const int wave = tid >> 6;
  const uint16_t* x = a.logits + (size_t)row * a.ldl;
  float bv = -INFINITY;
  int bi = a.V;
  const int nvec = a.V >> 3;
  const int j_lo = min(nvec, sp * a.chunk), j_hi = min(nvec, j_lo + a.chunk);
  for (int j0 = j_lo + tid; j0 < j_hi; j0 += 256 * kAcceptVecs) {
    u32x4 w[kAcceptVecs];  // all issued before any is used (past the range: its last vector again)
#pragma unroll
    for (int u = 0; u < kAcceptVecs; ++u) {
      const int j = min(j0 + 256 * u, j_hi - 1);
      w[u] = *reinterpret_cast<const u32x4*>(x + (size_t)j * 8);
    }
#pragma unroll
    for (int u = 0; u < kAcceptVecs; ++u) {
      const int j = j0 + 256 * u;
      if (j >= j_hi) break;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float v = h2f((uint16_t)(w[u][e >> 1] >> (16 * (e & 1))));
        if (beats(v, 8 * j + e, bv, bi)) {
          bv = v;
          bi = 8 * j + e;
        }
      }
    }
  }
  if (sp == a.S - 1) {  // the columns past the last whole vector
    for (int i = 8 * nvec + tid; i < a.V; i += 256) {
      const float v = h2f(x[i]);
      if (beats(v, i, bv, bi)) {
        bv = v;
        bi = i;
      }
    }
  }
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) {
    const float ov = __shfl_xor(bv, off, kWave);
    const int oi = __shfl_xor(bi, off, kWave);
    if (beats(ov, oi, bv, bi)) {
      bv = ov;
      bi = oi;
    }
  }
  if (lane == 0) {
    s_v[wave] = bv;
    s_i[wave] = bi;
  }
  __syncthreads();
  if (tid == 0) {
#pragma unroll
    for (int w = 1; w < 4; ++w)
      if (beats(s_v[w], s_i[w], bv, bi)) {
        bv = s_v[w];
        bi = s_i[w];
      }
    __hip_atomic_store(a.part + blockIdx.x, ((uint64_t)(uint32_t)bi << 32) | __float_as_uint(bv), __ATOMIC_RELAXED,
                       __HIP_MEMORY_SCOPE_AGENT);
    // tickets in two levels, so that no counter takes more than max(S, T)
    // atomics: the last workgroup of a row combines the row, the last row
    // to finish walks the tree
    uint32_t* row_counter = ws_counters(a.ws) + 16 * (1 + row);  // 64 bytes apart
    int last = 0;
    if (take_ticket(row_counter) == (uint32_t)(a.S - 1)) {
      reset_counter(row_counter);
      float cv = -INFINITY;
      int ci = a.V;
      for (int q = 0; q < a.S; ++q) {  // the row's ranges in order
        const uint64_t pq =
            __hip_atomic_load(a.part + (size_t)row * a.S + q, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        const float v = __uint_as_float((uint32_t)pq);
        const int i = (int)(pq >> 32);
        if (beats(v, i, cv, ci)) {
          cv = v;
          ci = i;
        }
      }
      // a row of NaNs alone keeps the sentinel: report index 0
      __hip_atomic_store(a.argmax + row, ci < a.V ? ci : 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      last = take_ticket(ws_counters(a.ws)) == (uint32_t)(a.T - 1);
    }
    s_ticket = last;
  }
  __syncthreads();
  if (!s_ticket || wave != 0) return;

  // ---- the last row to finish, one wavefront (lane = node): validate the
  // tree and walk it ----
  if (lane == 0) reset_counter(ws_counters(a.ws));  // for the next launch (stream-ordered)
  const bool in = lane < a.T;
  const int choice = in ? __hip_atomic_load(a.argmax + lane, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) : 0;
  const int p = in ? a.parent[lane] : -1;
  const bool ok = !in || (lane == 0 ? p == -1 : (p >= 0 && p < lane));
  if (!__all(ok)) {
    if (lane == 0) report_error(a.ws, SWIFTSPEC_DEVERR_BAD_TREE);
    return;
  }
  const int tok = in ? a.tokens[lane] : 0;
  int u = 0, L = 1;
  for (int step = 1; step < a.T; ++step) {  // each step moves to a higher index: at most T - 1
    const int want = __shfl(choice, u, kWave);
    const uint64_t cand = __ballot(in && lane > 0 && p == u && tok == want);
    if (cand == 0) break;
    u = (int)__builtin_ctzll(cand);
    ++L;
  }
  const int b = __shfl(choice, u, kWave);
  if (lane == 0) {
    *a.accepted = u;
    *a.bonus = b;
    if (a.path_len) *a.path_len = L;
  }
}

int greedy_accept_splits(int T) {
  int S = 1024 / T;
  return S < 1 ? 1 : S > 64 ? 64 : S;
}

void launch_greedy_accept(const uint16_t* logits, int ldl, int T, int V, const int32_t* tokens,
                          const int32_t* parent, int32_t* argmax, int32_t* accepted, int32_t* bonus,
                          int32_t* path_len, void* ws, void* part, hipStream_t st) {
  const int S = greedy_accept_splits(T);
  const int nvec = V >> 3;
  AcceptArgs a{logits, ldl, T, V, S, (nvec + S - 1) / S, tokens, parent, argmax, accepted, bonus, path_len, ws,
               reinterpret_cast<uint64_t*>(part)};
  hipLaunchKernelGGL(greedy_accept_kernel, dim3(T * S), dim3(256), 0, st, a);
}

}  // namespace ss
