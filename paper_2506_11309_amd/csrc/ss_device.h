// Device-side helpers shared by the swiftspec HIP kernels (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/swiftspec.h"

namespace ss {

typedef _Float16 half8 __attribute__((ext_vector_type(8)));
typedef _Float16 half2v __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

constexpr int kWave = 64;

// Workspace header: error word at byte 0, ticket counters from byte 256.
constexpr uint32_t kWsHeaderBytes = 65536u;
constexpr uint32_t kWsCounterOffset = 256u;
constexpr uint32_t kWsMaxCounters = (kWsHeaderBytes - kWsCounterOffset) / 4u;

__device__ __forceinline__ uint32_t* ws_error_word(void* ws) { return reinterpret_cast<uint32_t*>(ws); }
__device__ __forceinline__ uint32_t* ws_counters(void* ws) {
  return reinterpret_cast<uint32_t*>(reinterpret_cast<char*>(ws) + kWsCounterOffset);
}

__device__ __forceinline__ void report_error(void* ws, uint32_t bits) {
  if (ws) __hip_atomic_fetch_or(ws_error_word(ws), bits, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__device__ __forceinline__ int lane_id() { return __lane_id(); }

__device__ __forceinline__ uint64_t shfl_u64(uint64_t v, int src) {
  uint32_t lo = __shfl((int)(uint32_t)v, src, kWave);
  uint32_t hi = __shfl((int)(uint32_t)(v >> 32), src, kWave);
  return ((uint64_t)hi << 32) | lo;
}

// Ancestor-or-self bitmask and depth of node `lane` (lane < T <= 64) for the
// parent array `parent` (global memory), computed by one full wavefront with
// pointer jumping: after round r every lane holds the 2^r nearest nodes of
// its root path, so 6 rounds cover any depth below 64.  Must be called by
// all 64 lanes of a wave.  Returns false (for every lane) if the array is
// not a valid increasing tree; then anc = own bit and depth = 0.
// kForest: any node may be a root (parent -1), as in a draft model's tree
// cache below its last prefix token; otherwise node 0 is the only root.
// tree_masks_from: the same from the parent value p of node `lane` (-1 for
// lanes >= T), already loaded by the caller.
template <bool kForest = false>
__device__ __forceinline__ bool tree_masks_from(int p, int T, uint64_t& anc, int& depth) {
  const int lane = lane_id();
  bool ok = lane >= T || (kForest ? (p >= -1 && p < lane) : (lane == 0 ? p == -1 : (p >= 0 && p < lane)));
  const bool all_ok = __all(ok);
  uint64_t a = lane < T ? (1ull << lane) : 0ull;
  if (!all_ok) {
    anc = a;
    depth = 0;
    return false;
  }
  int up = lane < T ? p : -1;
#pragma unroll
  for (int r = 0; r < 6; ++r) {
    const int src = up >= 0 ? up : lane;
    const uint64_t a_up = shfl_u64(a, src);
    const int up_up = __shfl(up, src, kWave);
    if (up >= 0) {
      a |= a_up;
      up = up_up;
    }
  }
  anc = a;
  depth = __popcll(a) - 1;
  return true;
}
template <bool kForest = false>
__device__ __forceinline__ bool tree_masks_wave(const int32_t* __restrict__ parent, int T,
                                                uint64_t& anc, int& depth) {
  const int lane = lane_id();
  return tree_masks_from<kForest>(lane < T ? parent[lane] : -1, T, anc, depth);
}

// fp16 bit helpers
__device__ __forceinline__ float h2f(uint16_t h) {
  _Float16 v;
  __builtin_memcpy(&v, &h, 2);
  return (float)v;
}
__device__ __forceinline__ uint16_t f2h(float f) {
  _Float16 v = (_Float16)f;  // round to nearest even
  uint16_t h;
  __builtin_memcpy(&h, &v, 2);
  return h;
}

template <typename V, typename S>
__device__ __forceinline__ V bitcast(const S& s) {
  static_assert(sizeof(V) == sizeof(S), "size mismatch");
  V v;
  __builtin_memcpy(&v, &s, sizeof(V));
  return v;
}

// Agent-scope (cross-XCD) coherent 8-byte store / load for split partials.
__device__ __forceinline__ void store_agent_u64(void* p, uint64_t v) {
  __hip_atomic_store(reinterpret_cast<uint64_t*>(p), v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ uint64_t load_agent_u64(const void* p) {
  return __hip_atomic_load(reinterpret_cast<const uint64_t*>(p), __ATOMIC_RELAXED,
                           __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void store_agent_f32x4(float* p, f32x4 v) {
  store_agent_u64(p, bitcast<uint64_t>(f32x2{v[0], v[1]}));
  store_agent_u64(p + 2, bitcast<uint64_t>(f32x2{v[2], v[3]}));
}
__device__ __forceinline__ f32x4 load_agent_f32x4(const float* p) {
  f32x2 a = bitcast<f32x2>(load_agent_u64(p));
  f32x2 b = bitcast<f32x2>(load_agent_u64(p + 2));
  return f32x4{a[0], a[1], b[0], b[1]};
}

// Workgroup barrier without a memory fence: s_barrier after the wave's own
// LDS traffic has completed.  __syncthreads() would also wait for every
// outstanding global load (prefetched tiles); the empty asm statements
// with a memory clobber keep the compiler from moving LDS accesses across.
__device__ __forceinline__ void lds_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// Raw buffer resource over [p, p + bytes) (stride 0; dword 3 = the CDNA
// raw-buffer format), and 16- / 4-byte loads at voffset + soffset from it.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t buffer_rsrc(const void* p, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), (short)0, (int)bytes, 0x00020000);
}
__device__ __forceinline__ u32x4 buffer_load_x4(__amdgpu_buffer_rsrc_t r, uint32_t voffset, uint32_t soffset) {
  return __builtin_amdgcn_raw_buffer_load_b128(r, voffset, soffset, 0);
}
__device__ __forceinline__ uint32_t buffer_load_x1(__amdgpu_buffer_rsrc_t r, uint32_t voffset, uint32_t soffset) {
  return __builtin_amdgcn_raw_buffer_load_b32(r, voffset, soffset, 0);
}

// 16-byte buffer load of every lane straight into LDS: lane l's 16 bytes
// (at voff + soff of the buffer) land at LDS address lds_addr + 16 l.  M0,
// which holds the LDS base of such loads, is saved and restored around the
// load (one wait state after setting it), so the compiler's own use of M0 is
// untouched.  The compiler does not see the LDS write: the caller waits for
// it with vmcnt and orders it against LDS reads with barriers.
typedef int i32x4 __attribute__((ext_vector_type(4)));
__device__ __forceinline__ i32x4 raw_rsrc(const void* base, uint32_t bytes) {
  const uint64_t b = (uint64_t)(uintptr_t)base;
  return i32x4{(int)(uint32_t)b, (int)(uint32_t)(b >> 32), (int)bytes, 0x00020000};
}
__device__ __forceinline__ void buffer_load_lds16(i32x4 rsrc, uint32_t voff, uint32_t soff, uint32_t lds_addr) {
  uint32_t saved;
  asm volatile(
      "s_mov_b32 %0, m0\n\ts_mov_b32 m0, %4\n\ts_nop 0\n\t"
      "buffer_load_dwordx4 %1, %2, %3 offen lds\n\ts_mov_b32 m0, %0"
      : "=&s"(saved)
      : "v"(voff), "s"(rsrc), "s"(soff), "s"(lds_addr)
      : "memory");
}
__device__ __forceinline__ uint32_t lds_address(const void* p) {
  return (uint32_t)(uintptr_t)(__attribute__((address_space(3))) const void*)p;
}

// Wait until at most N vector-memory operations of this wave are outstanding;
// expcnt and lgkmcnt are left alone.
template <int N>
__device__ __forceinline__ void vm_wait() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (0x7 << 4) | (0xF << 8));
}
// Ticket for the deterministic "last arriving workgroup combines" pattern,
// taken by the lane that stored the workgroup's partial.  Acquire-release at
// agent scope: the release publishes that lane's earlier stores (every
// later ticket holder reads the counter through the release sequence of
// these read-modify-writes), and the acquire lets the last holder read
// every earlier holder's stores; other lanes of the last workgroup read
// them after a workgroup barrier that follows the ticket.
__device__ __forceinline__ uint32_t take_ticket(uint32_t* counter) {
  return __hip_atomic_fetch_add(counter, 1u, __ATOMIC_ACQ_REL, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void reset_counter(uint32_t* counter) {
  __hip_atomic_store(counter, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

}  // namespace ss

namespace ss {

// ---- activation layout consumed by the W4A16 GEMMs ("prepared" layout) ----
// For a GEMM input x[M][K] with G = K / 128 quantisation groups, the matrix
// is stored as [M/16 tiles][G][4 fragments][64 lanes][8] fp16 so that a wave
// fetches each MFMA A-fragment with one coalesced 16-byte load per lane.
// Lane kq*16 + (m % 16) of fragment f holds 8 values of row m from k-range
// [128 g + 32 kq, +32), in the slot order the int4 dequantisation produces:
// fragments 0/1 take the even k of that range (first/second 16), fragments
// 2/3 the odd k.  Within a fragment the order is 0,4,2,6,8,12,10,14 (+1 for
// odd k).  Values are stored unchanged, so every fp16 input is accepted.
__host__ __device__ inline size_t prep_offset(int m, int k, int G) {
  const int mt = m >> 4, r16 = m & 15, g = k >> 7, j = k & 127, kq = j >> 5, t = j & 31;
  const int f = ((t & 1) << 1) | (t >> 4);
  const int u = (t & 15) >> 1;
  const int e = (u & 4) | ((u & 1) << 1) | ((u >> 1) & 1);
  return ((((size_t)mt * G + g) * 4 + f) * 64 + (kq * 16 + r16)) * 8 + e;
}

// Store the fp16 value h of activation (m, k) into a prepared buffer.
__device__ __forceinline__ void store_prepared(uint16_t* prep, int m, int k, int G, uint16_t h) {
  prep[prep_offset(m, k, G)] = h;
}

// Prepared-layout fragments of 32 consecutive activations k = 128 g + 32 kq
// + t, t = 0..31, of one row, given as 16 u32 (element t in half t % 2 of
// word t / 2): fragment 0 holds even t < 16, 1 even t >= 16, 2 odd t < 16,
// 3 odd t >= 16, each in slot order u = 0, 2, 1, 3, 4, 6, 5, 7 of
// u = (t % 16) / 2 -- the order prep_offset describes.  They belong at
// ((((m / 16) * G + g) * 4 + f) * 64 + kq * 16 + m % 16) * 8 halves.
__device__ __forceinline__ void pack_prepared(const uint32_t (&a)[16], u32x4 (&f)[4]) {
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const uint32_t* b = a + 8 * h;
    f[h] = u32x4{(b[0] & 0xFFFFu) | (b[2] << 16), (b[1] & 0xFFFFu) | (b[3] << 16),
                 (b[4] & 0xFFFFu) | (b[6] << 16), (b[5] & 0xFFFFu) | (b[7] << 16)};
    f[2 + h] = u32x4{(b[0] >> 16) | (b[2] & 0xFFFF0000u), (b[1] >> 16) | (b[3] & 0xFFFF0000u),
                     (b[4] >> 16) | (b[6] & 0xFFFF0000u), (b[5] >> 16) | (b[7] & 0xFFFF0000u)};
  }
}

}  // namespace ss
