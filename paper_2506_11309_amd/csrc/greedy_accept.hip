// Greedy acceptance of a verified draft tree on the device, closing the
// verification step without a host round trip (target-side verification
// with the target's greedy choice: Sec. 3.1 and the Fig. 3 walk-through,
// where each iteration's output is the accepted root path followed by one
// token the target produced after it).
//
// One workgroup per tree node reads that node's logits row [V] fp16
// (16-byte loads strided over 256 threads, 16 in flight per thread) and
// finds its first maximum:
// each thread keeps (value, index) over increasing indices, then the wave
// and the workgroup combine pairs (larger value; on equal values the lower
// index), so the result is the first index of the row's largest value.  The
// choice goes to argmax[node] with an agent-scope store; the workgroup then
// takes a ticket, and the one that draws the last ticket walks the tree in
// one wavefront (lane = node): from the root, the next node is the
// lowest-index child whose draft token equals the current node's choice
// (one ballot per step, at most T - 1 steps, each to a higher index), and
// the node where no child matches is accepted; its choice is the bonus
// token.  The walk reads the choices with agent-scope loads, so every
// workgroup's store is visible whichever XCD ran it.
#include "ss_device.h"
#include "ss_internal.h"

namespace ss {

struct AcceptArgs {
  const uint16_t* logits;
  int ldl, T, V;
  const int32_t* tokens;
  const int32_t* parent;
  int32_t* argmax;
  int32_t* accepted;
  int32_t* bonus;
  int32_t* path_len;
  void* ws;
};

// (v, i) beats (bv, bi): larger value, or equal value at a lower index
__device__ __forceinline__ bool beats(float v, int i, float bv, int bi) { return v > bv || (v == bv && i < bi); }

__global__ __launch_bounds__(256) void greedy_accept_kernel(AcceptArgs a) {
  __shared__ float s_v[4];
  __shared__ int s_i[4];
  __shared__ int s_ticket;
  const int row = blockIdx.x;
  const int tid = threadIdx.x;
  const int lane = lane_id();
  const int wave = tid >> 6;
  const uint16_t* x = a.logits + (size_t)row * a.ldl;
  float bv = -INFINITY;
  int bi = a.V;
  const int nvec = a.V >> 3;
  constexpr int kBatch = 16;  // 16-byte loads in flight per thread
  for (int j0 = tid; j0 < nvec; j0 += 256 * kBatch) {
    u32x4 w[kBatch];  // all issued before any is used (past the row: its last vector again)
#pragma unroll
    for (int u = 0; u < kBatch; ++u) {
      const int j = min(j0 + 256 * u, nvec - 1);
      w[u] = *reinterpret_cast<const u32x4*>(x + (size_t)j * 8);
    }
#pragma unroll
    for (int u = 0; u < kBatch; ++u) {
      const int j = j0 + 256 * u;
      if (j >= nvec) break;
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
  for (int i = 8 * nvec + tid; i < a.V; i += 256) {
    const float v = h2f(x[i]);
    if (beats(v, i, bv, bi)) {
      bv = v;
      bi = i;
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
    // a row of NaNs alone keeps the sentinel; report index 0 for it
    __hip_atomic_store(a.argmax + row, bi < a.V ? bi : 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    wait_all_memory();
    s_ticket = (int)take_ticket(ws_counters(a.ws));
  }
  __syncthreads();
  if (s_ticket != a.T - 1 || wave != 0) return;

  // ---- last workgroup, one wavefront: validate the tree and walk it ----
  if (lane == 0) reset_counter(ws_counters(a.ws));  // for the next launch (stream-ordered)
  const bool in = lane < a.T;
  const int p = in ? a.parent[lane] : -1;
  const bool ok = !in || (lane == 0 ? p == -1 : (p >= 0 && p < lane));
  if (!__all(ok)) {
    if (lane == 0) report_error(a.ws, SWIFTSPEC_DEVERR_BAD_TREE);
    return;
  }
  const int choice = in ? __hip_atomic_load(a.argmax + lane, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) : 0;
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

void launch_greedy_accept(const uint16_t* logits, int ldl, int T, int V, const int32_t* tokens,
                          const int32_t* parent, int32_t* argmax, int32_t* accepted, int32_t* bonus,
                          int32_t* path_len, void* ws, hipStream_t st) {
  AcceptArgs a{logits, ldl, T, V, tokens, parent, argmax, accepted, bonus, path_len, ws};
  hipLaunchKernelGGL(greedy_accept_kernel, dim3(T), dim3(256), 0, st, a);
}

}  // namespace ss
