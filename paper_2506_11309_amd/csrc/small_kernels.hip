// RMSNorm, KV commit, tree-mask query and workspace-initialisation kernels.
#include "ss_device.h"
#include "ss_internal.h"

namespace ss {

// ------------------------------------------------------------------ RMSNorm
// out = fp16(x / sqrt(mean(x^2) + eps) * gamma); one workgroup per row,
// fp32 sum of squares, fixed reduction order (deterministic).  Thread t owns
// the 32-element chunks c = t + 256 i (k = 32 c .. 32 c + 31), i.e. one
// prepared fragment set each.  With kRegs > 0 (rows of at most 8192 kRegs
// elements) the row and gamma are loaded once, up front, and kept in
// registers across the reduction; kRegs = 0 re-reads them (any width).
template <int kRegs>
__global__ __launch_bounds__(256) void rmsnorm_kernel(const uint16_t* __restrict__ x, int H, int ldx,
                                                      const uint16_t* __restrict__ gamma, float eps,
                                                      uint16_t* __restrict__ out, int ldo,
                                                      uint16_t* __restrict__ out_prep) {
  __shared__ float partial[4];
  const int m = blockIdx.x;
  const uint16_t* xr = x + (size_t)m * ldx;
  const int nch = H >> 5;
  constexpr int kR = kRegs > 0 ? kRegs : 1;
  u32x4 xv[kR][4], gv[kR][4];
  auto sumsq = [](const u32x4& v, float& acc) {
    const half8 h = bitcast<half8>(v);
#pragma unroll
    for (int e = 0; e < 8; ++e) acc = __builtin_fmaf((float)h[e], (float)h[e], acc);
  };
  float ss = 0.f;
  if constexpr (kRegs > 0) {
#pragma unroll
    for (int i = 0; i < kRegs; ++i) {
      const int c = threadIdx.x + 256 * i;
      if (c < nch) {
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          xv[i][q] = *reinterpret_cast<const u32x4*>(xr + 32 * c + 8 * q);
          gv[i][q] = *reinterpret_cast<const u32x4*>(gamma + 32 * c + 8 * q);
        }
      }
    }
#pragma unroll
    for (int i = 0; i < kRegs; ++i)
      if (threadIdx.x + 256 * i < nch)
#pragma unroll
        for (int q = 0; q < 4; ++q) sumsq(xv[i][q], ss);
  } else {
    for (int c = threadIdx.x; c < nch; c += 256)
#pragma unroll
      for (int q = 0; q < 4; ++q) sumsq(*reinterpret_cast<const u32x4*>(xr + 32 * c + 8 * q), ss);
  }
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) ss += __shfl_xor(ss, off, kWave);
  if (lane_id() == 0) partial[threadIdx.x >> 6] = ss;
  __syncthreads();
  const float total = (partial[0] + partial[1]) + (partial[2] + partial[3]);
  const float inv = 1.0f / sqrtf(total / (float)H + eps);
  uint16_t* orow = out + (size_t)m * ldo;
  const int G = H >> 7;
  auto emit = [&](int c, const u32x4 (&xs)[4], const u32x4 (&gs)[4]) {
    uint32_t w[16];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const half8 h = bitcast<half8>(xs[q]);
      const half8 gm = bitcast<half8>(gs[q]);
      half8 o;
#pragma unroll
      for (int e = 0; e < 8; ++e) o[e] = (_Float16)(((float)h[e] * inv) * (float)gm[e]);
      const u32x4 ob = bitcast<u32x4>(o);
      if (out) *reinterpret_cast<u32x4*>(orow + 32 * c + 8 * q) = ob;
#pragma unroll
      for (int e = 0; e < 4; ++e) w[4 * q + e] = ob[e];
    }
    if (out_prep) {
      u32x4 f[4];
      pack_prepared(w, f);
      const int g = c >> 2, kq = c & 3;
      uint16_t* base = out_prep + ((((size_t)(m >> 4) * G + g) * 4) * kWave + kq * 16 + (m & 15)) * 8;
#pragma unroll
      for (int fi = 0; fi < 4; ++fi) *reinterpret_cast<u32x4*>(base + (size_t)fi * kWave * 8) = f[fi];
    }
  };
  if constexpr (kRegs > 0) {
#pragma unroll
    for (int i = 0; i < kRegs; ++i) {
      const int c = threadIdx.x + 256 * i;
      if (c < nch) emit(c, xv[i], gv[i]);
    }
  } else {
    for (int c = threadIdx.x; c < nch; c += 256) {
      u32x4 xs[4], gs[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        xs[q] = *reinterpret_cast<const u32x4*>(xr + 32 * c + 8 * q);
        gs[q] = *reinterpret_cast<const u32x4*>(gamma + 32 * c + 8 * q);
      }
      emit(c, xs, gs);
    }
  }
}

void launch_rmsnorm(const uint16_t* x, int M, int H, int ldx, const uint16_t* gamma, float eps,
                    uint16_t* out, int ldo, uint16_t* out_prep, hipStream_t st) {
  const int nch = H / 32;
  if (nch <= 256)
    hipLaunchKernelGGL(rmsnorm_kernel<1>, dim3(M), dim3(256), 0, st, x, H, ldx, gamma, eps, out, ldo, out_prep);
  else if (nch <= 512)
    hipLaunchKernelGGL(rmsnorm_kernel<2>, dim3(M), dim3(256), 0, st, x, H, ldx, gamma, eps, out, ldo, out_prep);
  else
    hipLaunchKernelGGL(rmsnorm_kernel<0>, dim3(M), dim3(256), 0, st, x, H, ldx, gamma, eps, out, ldo, out_prep);
}

// ---------------------------------------------------------------- KV commit
// One workgroup per (layer, K|V, kv head).  Wave 0 derives the accepted
// path from the device parent array: the ancestor-or-self mask of the
// accepted node, whose set bits in increasing order are the root-to-node
// path (indices grow along any root path since parent[i] < i).  Every
// thread then loads its 16-byte column slice of all L source rows into
// registers; after a barrier it stores them to rows P .. P+L-1, so no write
// can clobber a source another thread has yet to read.
constexpr int kCommitMaxRowsPerThread = 8;  // 64 rows, D = 128: 16 B x 8 rows per thread

__device__ __forceinline__ bool commit_setup(const int32_t* parent, int T, const int32_t* accepted,
                                             const int32_t* prefix_len, int S_max, int* s_path,
                                             int* s_L, int* s_P, int* s_err) {
  // wave 0 only
  uint64_t anc;
  int depth;
  const bool ok = tree_masks_wave(parent, T, anc, depth);
  const int lane = lane_id();
  const int acc = *accepted;
  const int P = *prefix_len;
  int err = 0;
  if (!ok) err |= SWIFTSPEC_DEVERR_BAD_TREE;
  if (acc < 0 || acc >= T) err |= SWIFTSPEC_DEVERR_BAD_ACCEPTED;
  if (P < 0 || P > S_max - T) err |= SWIFTSPEC_DEVERR_BAD_PREFIX;
  const uint64_t path = shfl_u64(anc, (acc >= 0 && acc < T) ? acc : 0);
  if (lane < T && ((path >> lane) & 1ull)) {
    const int rank = __popcll(path & ((1ull << lane) - 1ull));
    s_path[rank] = lane;
  }
  if (lane == 0) {
    *s_L = __popcll(path);
    *s_P = P;
    *s_err = err;
  }
  return err == 0;
}

__global__ __launch_bounds__(256) void kv_commit_kernel(uint16_t* k_cache, uint16_t* v_cache,
                                                        int64_t layer_stride, int Hkv, int S_max,
                                                        int D, const int32_t* prefix_len,
                                                        const int32_t* parent, int T,
                                                        const int32_t* accepted, void* ws) {
  __shared__ int s_path[64];
  __shared__ int s_L, s_P, s_err;
  const int idx = blockIdx.x;
  const int head = idx % Hkv;
  const int which = (idx / Hkv) & 1;
  const int layer = idx / (2 * Hkv);
  if (threadIdx.x < 64) commit_setup(parent, T, accepted, prefix_len, S_max, s_path, &s_L, &s_P, &s_err);
  __syncthreads();
  if (s_err) {
    if (idx == 0 && threadIdx.x == 0) report_error(ws, (uint32_t)s_err);
    return;
  }
  const int L = s_L, P = s_P;
  uint16_t* base = (which ? v_cache : k_cache) + (size_t)layer * layer_stride + ((size_t)head * S_max + P) * D;
  const int vec_per_row = D / 8;
  const int rows_per_pass = 256 / vec_per_row;
  const int c8 = (threadIdx.x % vec_per_row) * 8;
  const int r0 = threadIdx.x / vec_per_row;
  u32x4 buf[kCommitMaxRowsPerThread];
#pragma unroll
  for (int j = 0; j < kCommitMaxRowsPerThread; ++j) {
    const int i = r0 + j * rows_per_pass;
    if (i < L) buf[j] = *reinterpret_cast<const u32x4*>(base + (size_t)s_path[i] * D + c8);
  }
  __syncthreads();  // every source row read before any row is written
#pragma unroll
  for (int j = 0; j < kCommitMaxRowsPerThread; ++j) {
    const int i = r0 + j * rows_per_pass;
    if (i < L) *reinterpret_cast<u32x4*>(base + (size_t)i * D + c8) = buf[j];
  }
}

// Advances the device prefix length by the accepted path length (runs after
// the copy kernel in stream order).
__global__ void prefix_advance_kernel(int32_t* prefix_len, const int32_t* parent, int T,
                                      const int32_t* accepted, int S_max) {
  __shared__ int s_path[64];
  __shared__ int s_L, s_P, s_err;
  commit_setup(parent, T, accepted, prefix_len, S_max, s_path, &s_L, &s_P, &s_err);
  __syncthreads();
  if (threadIdx.x == 0 && s_err == 0) *prefix_len = s_P + s_L;
}

void launch_kv_commit(uint16_t* k_cache, uint16_t* v_cache, int n_layers, int64_t layer_stride,
                      int Hkv, int S_max, int D, int32_t* prefix_len, const int32_t* parent, int T,
                      const int32_t* accepted, int advance, void* ws, hipStream_t st) {
  hipLaunchKernelGGL(kv_commit_kernel, dim3(n_layers * 2 * Hkv), dim3(256), 0, st, k_cache, v_cache,
                     layer_stride, Hkv, S_max, D, prefix_len, parent, T, accepted, ws);
  if (advance)
    hipLaunchKernelGGL(prefix_advance_kernel, dim3(1), dim3(64), 0, st, prefix_len, parent, T, accepted,
                       S_max);
}

// ------------------------------------------- draft-side KV reorganisation
// The draft model's cache after re-rooting (Sec. 3.2, Fig. 5): rows
// [P, P+N) hold a forest of draft nodes (parent -1: below the last prefix
// token).  Wave 0 of every workgroup derives, from the forest's
// ancestor-or-self masks, the verified path (the set bits of last's mask,
// in increasing order: indices grow along any root path) and, if kept, the
// nodes having `last` as a proper ancestor (in increasing order); row P + i
// then takes the old row of the i-th node of path ++ kept, with the same
// read-all-then-write pattern as the commit.  Workgroup 0 also writes the
// kept nodes' parents renumbered into the new tree cache (-1 below last).
__device__ __forceinline__ bool reorg_setup(const int32_t* parent, int N, const int32_t* d_last,
                                            const int32_t* d_keep, const int32_t* prefix_len, int S_max,
                                            int* s_rows, int* s_L, int* s_S, int* s_P, int* s_err,
                                            int32_t* new_parent) {
  // wave 0 only
  uint64_t anc;
  int depth;
  const bool ok = tree_masks_wave<true>(parent, N, anc, depth);
  const int lane = lane_id();
  const int last = *d_last;
  const bool keep = *d_keep != 0;
  const int P = *prefix_len;
  int err = 0;
  if (!ok) err |= SWIFTSPEC_DEVERR_BAD_TREE;
  if (last < -1 || last >= N) err |= SWIFTSPEC_DEVERR_BAD_ACCEPTED;
  if (P < 0 || P > S_max - N) err |= SWIFTSPEC_DEVERR_BAD_PREFIX;
  const bool have = err == 0 && last >= 0;
  const uint64_t path = have ? shfl_u64(anc, last) : 0ull;
  const bool mine_kept = have && keep && lane < N && lane != last && ((anc >> last) & 1ull);
  const uint64_t kept = __ballot(mine_kept);
  const int L = __popcll(path), S = __popcll(kept);
  const uint64_t below = (1ull << lane) - 1ull;
  if (lane < N && ((path >> lane) & 1ull)) s_rows[__popcll(path & below)] = lane;
  if (mine_kept) {
    const int j = __popcll(kept & below);
    s_rows[L + j] = lane;
    if (new_parent) {
      const int p = parent[lane];
      new_parent[j] = p == last ? -1 : __popcll(kept & ((1ull << p) - 1ull));
    }
  }
  if (lane == 0) {
    *s_L = L;
    *s_S = S;
    *s_P = P;
    *s_err = err;
  }
  return err == 0;
}

__global__ __launch_bounds__(256) void kv_reorganize_kernel(uint16_t* k_cache, uint16_t* v_cache,
                                                            int64_t layer_stride, int Hkv, int S_max, int D,
                                                            const int32_t* prefix_len, const int32_t* parent,
                                                            int N, const int32_t* d_last, const int32_t* d_keep,
                                                            int32_t* new_parent, int32_t* n_kept, void* ws) {
  __shared__ int s_rows[64];
  __shared__ int s_L, s_S, s_P, s_err;
  const int idx = blockIdx.x;
  const int head = idx % Hkv;
  const int which = (idx / Hkv) & 1;
  const int layer = idx / (2 * Hkv);
  if (threadIdx.x < 64)
    reorg_setup(parent, N, d_last, d_keep, prefix_len, S_max, s_rows, &s_L, &s_S, &s_P, &s_err,
                idx == 0 ? new_parent : nullptr);
  __syncthreads();
  if (s_err) {
    if (idx == 0 && threadIdx.x == 0) report_error(ws, (uint32_t)s_err);
    return;
  }
  const int R = s_L + s_S, P = s_P;
  if (idx == 0 && threadIdx.x == 0 && n_kept) *n_kept = s_S;
  uint16_t* base = (which ? v_cache : k_cache) + (size_t)layer * layer_stride + ((size_t)head * S_max + P) * D;
  const int vec_per_row = D / 8;
  const int rows_per_pass = 256 / vec_per_row;
  const int c8 = (threadIdx.x % vec_per_row) * 8;
  const int r0 = threadIdx.x / vec_per_row;
  u32x4 buf[kCommitMaxRowsPerThread];
#pragma unroll
  for (int j = 0; j < kCommitMaxRowsPerThread; ++j) {
    const int i = r0 + j * rows_per_pass;
    if (i < R) buf[j] = *reinterpret_cast<const u32x4*>(base + (size_t)s_rows[i] * D + c8);
  }
  __syncthreads();  // every source row read before any row is written
#pragma unroll
  for (int j = 0; j < kCommitMaxRowsPerThread; ++j) {
    const int i = r0 + j * rows_per_pass;
    if (i < R) *reinterpret_cast<u32x4*>(base + (size_t)i * D + c8) = buf[j];
  }
}

// The prefix grows by the path length (after the copy kernel, in stream order).
__global__ void reorg_prefix_advance_kernel(int32_t* prefix_len, const int32_t* parent, int N, const int32_t* d_last,
                                            const int32_t* d_keep, int S_max) {
  __shared__ int s_rows[64];
  __shared__ int s_L, s_S, s_P, s_err;
  reorg_setup(parent, N, d_last, d_keep, prefix_len, S_max, s_rows, &s_L, &s_S, &s_P, &s_err, nullptr);
  __syncthreads();
  if (threadIdx.x == 0 && s_err == 0) *prefix_len = s_P + s_L;
}

void launch_kv_reorganize(uint16_t* k_cache, uint16_t* v_cache, int n_layers, int64_t layer_stride, int Hkv,
                          int S_max, int D, int32_t* prefix_len, const int32_t* parent, int N, const int32_t* d_last,
                          const int32_t* d_keep, int32_t* new_parent, int32_t* n_kept, int advance, void* ws,
                          hipStream_t st) {
  hipLaunchKernelGGL(kv_reorganize_kernel, dim3(n_layers * 2 * Hkv), dim3(256), 0, st, k_cache, v_cache,
                     layer_stride, Hkv, S_max, D, prefix_len, parent, N, d_last, d_keep, new_parent, n_kept, ws);
  if (advance)
    hipLaunchKernelGGL(reorg_prefix_advance_kernel, dim3(1), dim3(64), 0, st, prefix_len, parent, N, d_last, d_keep,
                       S_max);
}

// ---------------------------------------------------------- tree masks
__global__ __launch_bounds__(64) void tree_masks_kernel(const int32_t* parents, int T, uint64_t* anc,
                                                        int32_t* depth, int32_t* status) {
  const int t = blockIdx.x;
  uint64_t a;
  int d;
  const bool ok = tree_masks_wave(parents + (size_t)t * T, T, a, d);
  const int lane = lane_id();
  if (lane < T) {
    anc[(size_t)t * T + lane] = a;
    depth[(size_t)t * T + lane] = d;
  }
  if (lane == 0) status[t] = ok ? 0 : (int32_t)SWIFTSPEC_DEVERR_BAD_TREE;
}

void launch_tree_masks(const int32_t* parents, int n_trees, int T, uint64_t* anc, int32_t* depth,
                       int32_t* status, hipStream_t st) {
  hipLaunchKernelGGL(tree_masks_kernel, dim3(n_trees), dim3(64), 0, st, parents, T, anc, depth, status);
}

// -------------------------------------------------------- clock sample
// One wave: shader-clock and 100 MHz real-time counters before and after a
// bounded wait of `ticks` real-time ticks.
__global__ __launch_bounds__(64) void clock_sample_kernel(uint64_t* __restrict__ out, uint32_t ticks) {
  const uint64_t c0 = __builtin_amdgcn_s_memtime();
  const uint64_t r0 = __builtin_amdgcn_s_memrealtime();
  uint64_t r = r0;
  for (int i = 0; i < (1 << 22) && r - r0 < ticks; ++i) {
    __builtin_amdgcn_s_sleep(1);
    r = __builtin_amdgcn_s_memrealtime();
  }
  const uint64_t c1 = __builtin_amdgcn_s_memtime();
  r = __builtin_amdgcn_s_memrealtime();
  if (threadIdx.x == 0) {
    out[0] = c0;
    out[1] = r0;
    out[2] = c1;
    out[3] = r;
  }
}

void launch_clock_sample(uint64_t* out, uint32_t ticks, hipStream_t st) {
  hipLaunchKernelGGL(clock_sample_kernel, dim3(1), dim3(64), 0, st, out, ticks);
}

// ------------------------------------------------------ workspace init
__global__ void fill_zero_kernel(uint32_t* p, size_t n) {
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x)
    p[i] = 0u;
}

void launch_ws_init(void* ws, size_t bytes, hipStream_t st) {
  const size_t n = bytes / 4;
  hipLaunchKernelGGL(fill_zero_kernel, dim3(64), dim3(256), 0, st, reinterpret_cast<uint32_t*>(ws), n);
}

}  // namespace ss
