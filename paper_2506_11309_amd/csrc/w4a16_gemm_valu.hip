// W4A16 GEMM on the vector ALUs only (no matrix cores), for comparing the
// two ways of computing the int4 projections of a decoder layer at M = tree
// size (Sec. 3.3; Sec. 5.1 for the int4 group-128 setting):
//     y[m][n] = sum_k x[m][k] * (q[n][k] - z[n][g]) * s[n][g] (+ residual).
//
// Same operands as the matrix-core kernel: the kernel-native weight copy
// (1 KB per 16-column x 128-k block) and the activations in the prepared
// operand layout.  One wave owns one 16-column tile and one 16-row M-tile
// over a slice of the groups (a workgroup: 4 / MT tiles x MT M-tiles, so the
// waves of one tile share its weight block through the caches); lane
// (n = lane % 16, kq = lane / 16) dequantises its 32 nibbles of column n
// (k in [128 g + 32 kq, +32)) to 16 fp16 pairs of exact integers (magic
// numbers 1024 and 64, as in the matrix-core kernel), and for each of its 16 token
// rows forms the 32-term dot product with v_dot2_f32_f16 (16 instructions per
// row and group) against the row's four activation fragments, which the
// workgroup stages through a 3-slot LDS ring (lanes of one kq read the same
// 16 bytes: LDS broadcast).  At the end of the slice the four kq lanes of a
// column are summed with two shuffles; slices are summed in order by a
// second kernel, which also adds the residual (deterministic).
#include "ss_device.h"
#include "ss_internal.h"

namespace ss {

constexpr int kValuRing = 4;   // register ring of weight blocks
constexpr int kValuLds = 3;    // LDS ring of activation fragments
constexpr int kValuWaves = 2048;

struct ValuArgs {
  const u32x4* q;
  const uint32_t* sz;
  const uint16_t* a;  // prepared activations [MT][G][4][64][8]
  int K, N, G, M, gslice, ntb;
  float* part;        // [ksplit][M][N]
};

// ROWS = token rows per wave: 16 (one M-tile) or, for M < 16, the next
// power of two >= M, so that the dot products scale with M.
template <int MT, int ROWS>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(4))) void w4a16_gemm_valu_kernel(ValuArgs a) {
  constexpr int TPW = 4 / MT;         // column tiles per workgroup (MT in {1, 2, 4})
  __shared__ u32x4 abuf[kValuLds][MT][4][kWave];
  const int tid = threadIdx.x;
  const int lane = lane_id();
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int ncol = lane & 15, kq = lane >> 4;
  const int tb = blockIdx.x % a.ntb, sl = blockIdx.x / a.ntb;
  const int tile = tb * TPW + wave / MT;
  const int mrow = wave % MT;         // this wave's M-tile
  const int G = a.G;
  const int g0 = sl * a.gslice;
  const int ng = min(G, g0 + a.gslice) - g0;  // >= 1 by construction of the plan

  u32x4 wr[kValuRing];
  uint32_t szr[kValuRing];
  u32x4 ar[kValuRing][MT];
  auto load = [&](int i, u32x4& w, uint32_t& sz, u32x4 (&r)[MT]) {
    int ii = i < ng ? i : ng - 1;
    asm volatile("" : "+s"(ii));
    const int g = g0 + ii;
    const size_t tg = (size_t)tile * G + g;
    w = a.q[tg * kWave + lane];
    sz = a.sz[tg * 16 + ncol];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
      r[mt] = reinterpret_cast<const u32x4*>(a.a)[(((size_t)mt * G + g) * 4 + wave) * kWave + lane];
  };
  auto store_a = [&](int slot, const u32x4 (&r)[MT]) {
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) abuf[slot][mt][wave][lane] = r[mt];
  };
  // exact dequantisation as in the matrix-core GEMM: low nibbles in 0x6400
  // (1024 + q), high nibbles (bits 4-7) in 0x5400 (64 + q), minus 1024 + z
  // resp. 64 + z
  uint32_t magic_lo = 0x64006400u, magic_hi = 0x54005400u;
  asm volatile("" : "+v"(magic_lo), "+v"(magic_hi));
  auto deq = [&](uint32_t x, uint32_t m, uint32_t magic, half2v zz) {
    return bitcast<half2v>(bitcast<half2v>((x & m) | (magic & ~m)) - zz);
  };

  float acc[ROWS];
#pragma unroll
  for (int r = 0; r < ROWS; ++r) acc[r] = 0.f;

  auto compute = [&](int slot, const u32x4& w, uint32_t sz) {
    const uint32_t s0 = w[0] >> 8, s1 = w[1] >> 8, s2 = w[2] >> 8, s3 = w[3] >> 8;
    constexpr uint32_t kLo = 0x000F000Fu, kHi = 0x00F000F0u;
    const uint32_t z = (sz >> 16) & 0xFFu;
    const half2v zlo = bitcast<half2v>((0x6400u + z) * 0x00010001u);
    const half2v zhi = bitcast<half2v>((0x5400u + 16u * z) * 0x00010001u);
    auto dl = [&](uint32_t x) { return deq(x, kLo, magic_lo, zlo); };
    auto dh = [&](uint32_t x) { return deq(x, kHi, magic_hi, zhi); };
    // B pairs in the element order of the four activation fragments
    const half2v b[16] = {dl(w[0]), dl(s0), dl(w[1]), dl(s1), dl(w[2]), dl(s2), dl(w[3]), dl(s3),
                          dh(w[0]), dh(s0), dh(w[1]), dh(s1), dh(w[2]), dh(s2), dh(w[3]), dh(s3)};
    const float sc = h2f((uint16_t)(sz & 0xFFFFu));
    // fragment f of row r at xb[f * 64 + r].  The base is passed through an
    // empty asm that depends on the row two before, so that the compiler
    // keeps at most two rows' fragment reads (16 registers each) in flight
    // instead of hoisting all of them ahead of the dot products.
    uint32_t xoff = (uint32_t)(((slot * MT + mrow) * 4 * kWave + kq * 16) * sizeof(u32x4));
#pragma unroll
    for (int r = 0; r < ROWS; ++r) {
      if (r >= 2) asm volatile("" : "+v"(xoff) : "v"(acc[r - 2]));
      const u32x4* xb = reinterpret_cast<const u32x4*>(reinterpret_cast<const char*>(&abuf[0][0][0][0]) + xoff);
      float c = 0.f;
#pragma unroll
      for (int f = 0; f < 4; ++f) {
        const u32x4 xv = xb[f * kWave + r];
#pragma unroll
        for (int e = 0; e < 4; ++e) c = __builtin_amdgcn_fdot2(bitcast<half2v>(xv[e]), b[4 * f + e], c, false);
      }
      acc[r] = __builtin_fmaf(c, sc, acc[r]);
    }
  };

  // step i: load group i + R - 1, write group i + 1's fragments to LDS slot
  // (i + 1) % 3 (last read at step i - 2), barrier, compute group i; whole
  // rounds, loads past the slice repeat its last group
#pragma unroll
  for (int j = 0; j < kValuRing - 1; ++j) load(j, wr[j], szr[j], ar[j]);
  store_a(0, ar[0]);
  for (int i0 = 0; i0 < ng; i0 += kValuRing) {
#pragma unroll
    for (int J = 0; J < kValuRing; ++J) {
      const int i = i0 + J;
      const int nx = (J + kValuRing - 1) % kValuRing;
      load(i + kValuRing - 1, wr[nx], szr[nx], ar[nx]);
      if (i < ng) {
        if (i + 1 < ng) store_a((i + 1) % kValuLds, ar[(J + 1) % kValuRing]);
        lds_barrier();
        compute(i % kValuLds, wr[J], szr[J]);
      } else {
        asm volatile("" : : "v"(wr[J]), "v"(szr[J]));
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) asm volatile("" : : "v"(ar[(J + 1) % kValuRing][mt]));
      }
    }
  }

  // sum the four k-quarters of each column; lanes 0..15 publish the slice's sums
  const int col = tile * 16 + ncol;
#pragma unroll
  for (int r = 0; r < ROWS; ++r) {
    float v = acc[r];
    v += __shfl_xor(v, 16, kWave);
    v += __shfl_xor(v, 32, kWave);
    const int m = mrow * 16 + r;
    if (kq == 0 && m < a.M) a.part[((size_t)sl * a.M + m) * a.N + col] = v;
  }
}

// y[m][n] = fp16( sum over slices in order + residual ); one thread each.
__global__ __launch_bounds__(256) void w4a16_valu_reduce_kernel(const float* __restrict__ part, int ksplit, int M,
                                                                 int N, uint16_t* __restrict__ y, int ldy,
                                                                 const uint16_t* __restrict__ res, int ldr) {
  const long idx = (long)blockIdx.x * 256 + threadIdx.x;
  if (idx >= (long)M * N) return;
  const int m = (int)(idx / N), n = (int)(idx % N);
  float v = 0.f;
  for (int s = 0; s < ksplit; ++s) v += part[((size_t)s * M + m) * N + n];
  if (res) v += h2f(res[(size_t)m * ldr + n]);
  y[(size_t)m * ldy + n] = f2h(v);
}

static int valu_mt(int M) {
  const int mt = (M + 15) / 16;
  return mt <= 1 ? 1 : mt == 2 ? 2 : 4;
}

ValuGemmPlan plan_w4a16_gemm_valu(int M, int K, int N) {
  ValuGemmPlan p;
  const int tiles = N / 16, G = K / 128;
  const int waves = tiles * valu_mt(M);
  int ks = (kValuWaves + waves - 1) / waves;
  if (ks > G) ks = G;
  if (ks < 1) ks = 1;
  p.gslice = (G + ks - 1) / ks;
  p.ksplit = (G + p.gslice - 1) / p.gslice;
  p.part_bytes = (size_t)p.ksplit * M * N * 4;
  return p;
}

void launch_w4a16_gemm_valu(const void* packed, int K, int N, const uint16_t* aprep, int M, uint16_t* y,
                            int ldy, const uint16_t* res, int ldr, float* part, const ValuGemmPlan& p,
                            hipStream_t st) {
  ValuArgs a;
  a.q = reinterpret_cast<const u32x4*>(packed);
  a.sz = reinterpret_cast<const uint32_t*>(reinterpret_cast<const char*>(packed) + (size_t)K * N / 2);
  a.a = aprep;
  a.K = K;
  a.N = N;
  a.G = K / 128;
  a.M = M;
  a.gslice = p.gslice;
  const int MT = valu_mt(M);
  a.ntb = (N / 16) / (4 / MT);
  a.part = part;
  const dim3 grid(a.ntb * p.ksplit);
  if (MT == 1) {
    if (M <= 1) hipLaunchKernelGGL((w4a16_gemm_valu_kernel<1, 1>), grid, dim3(256), 0, st, a);
    else if (M <= 2) hipLaunchKernelGGL((w4a16_gemm_valu_kernel<1, 2>), grid, dim3(256), 0, st, a);
    else if (M <= 4) hipLaunchKernelGGL((w4a16_gemm_valu_kernel<1, 4>), grid, dim3(256), 0, st, a);
    else if (M <= 8) hipLaunchKernelGGL((w4a16_gemm_valu_kernel<1, 8>), grid, dim3(256), 0, st, a);
    else hipLaunchKernelGGL((w4a16_gemm_valu_kernel<1, 16>), grid, dim3(256), 0, st, a);
  } else if (MT == 2) {
    hipLaunchKernelGGL((w4a16_gemm_valu_kernel<2, 16>), grid, dim3(256), 0, st, a);
  } else {
    hipLaunchKernelGGL((w4a16_gemm_valu_kernel<4, 16>), grid, dim3(256), 0, st, a);
  }
  const long total = (long)M * N;
  hipLaunchKernelGGL(w4a16_valu_reduce_kernel, dim3((unsigned)((total + 255) / 256)), dim3(256), 0, st, part,
                     p.ksplit, M, N, y, ldy, res, ldr);
}

}  // namespace ss
