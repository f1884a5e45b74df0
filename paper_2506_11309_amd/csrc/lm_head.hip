// Dense fp16 LM head at small M for gfx950: logits[m][v] = fp16( xn[m] . W[v] ),
// xn = the final RMSNorm of the last hidden states (written by rmsnorm_kernel),
// W [V][H] fp16 row-major (the vocabulary projection of the 80-layer step).
//
// HBM-bound: the weight matrix (2.1 GB at V = 128256, H = 8192) is read once.
// Mapping (v_mfma_f32_16x16x32_f16, wave64): B operand = 16 vocabulary rows
// of W, lane (n = lane % 16, kq = lane / 16) loads the 16 bytes
// W[16 t + n][32 s + 8 kq .. +7] of k-step s -- the four lanes of a row read
// 64 contiguous bytes; A operand = 16 rows of xn from LDS in the same k
// order.  A workgroup (4 waves x 2 tiles) owns 128 vocabulary rows for the
// whole K: no split, no partials.  K advances in blocks of 128: each thread
// stages its share of the block's activations through a register ring into a
// 3-slot LDS ring (one fence-free barrier per block), and each wave's weight
// loads run two blocks ahead in the same ring.
#include "ss_device.h"
#include "ss_internal.h"

namespace ss {

constexpr int kLmRing = 3;
constexpr int kLmCols = 2;              // 16-row tiles of W per wave

struct LmArgs {
  const uint16_t* xn;  // [M][H] fp16
  const uint16_t* W;   // [V][H] fp16
  uint16_t* logits;    // [M][ldl]
  int M, H, V, ldl;
};

template <int MT>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(2))) void lm_head_kernel(LmArgs a) {
  constexpr int KST = 128 + 8;  // halves per LDS row (16-byte pad)
  __shared__ uint16_t xs[kLmRing][MT * 16 * KST];
  const int tid = threadIdx.x;
  const int lane = lane_id();
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int n16 = lane & 15, kq = lane >> 4;
  const int tile0 = blockIdx.x * (4 * kLmCols) + wave * kLmCols;  // first 16-row tile of this wave
  const int ntiles = a.V >> 4;
  const int nkb = a.H >> 7;

  // activations of block kb: thread t stages vectors t + 256 j (row v / 16,
  // 16-byte column v % 16); rows >= M are zero
  auto load_x = [&](int kb, u32x4 (&r)[MT]) {
    int b = kb < nkb ? kb : nkb - 1;
    asm volatile("" : "+s"(b));
#pragma unroll
    for (int j = 0; j < MT; ++j) {
      const int v = tid + 256 * j, row = v >> 4, c = v & 15;
      r[j] = row < a.M ? *reinterpret_cast<const u32x4*>(a.xn + (size_t)row * a.H + b * 128 + c * 8)
                       : u32x4{0u, 0u, 0u, 0u};
    }
  };
  auto store_x = [&](int slot, const u32x4 (&r)[MT]) {
#pragma unroll
    for (int j = 0; j < MT; ++j) {
      const int v = tid + 256 * j, row = v >> 4, c = v & 15;
      *reinterpret_cast<u32x4*>(&xs[slot][row * KST + c * 8]) = r[j];
    }
  };
  // weights of block kb for this wave's tiles (tiles past V repeat the last
  // valid one and are not stored)
  auto load_w = [&](int kb, u32x4 (&r)[kLmCols][4]) {
    int b = kb < nkb ? kb : nkb - 1;
    asm volatile("" : "+s"(b));
#pragma unroll
    for (int ct = 0; ct < kLmCols; ++ct) {
      const int t = tile0 + ct < ntiles ? tile0 + ct : ntiles - 1;
      const uint16_t* row = a.W + (size_t)(t * 16 + n16) * a.H + b * 128 + 8 * kq;
#pragma unroll
      for (int s = 0; s < 4; ++s) r[ct][s] = *reinterpret_cast<const u32x4*>(row + 32 * s);
    }
  };

  f32x4 acc[MT][kLmCols];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int ct = 0; ct < kLmCols; ++ct) acc[mt][ct] = f32x4{0.f, 0.f, 0.f, 0.f};

  auto compute = [&](int slot, const u32x4 (&w)[kLmCols][4]) {
#pragma unroll
    for (int s = 0; s < 4; ++s) {
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) {
        const half8 af = *reinterpret_cast<const half8*>(&xs[slot][(mt * 16 + n16) * KST + 32 * s + 8 * kq]);
#pragma unroll
        for (int ct = 0; ct < kLmCols; ++ct)
          acc[mt][ct] = __builtin_amdgcn_mfma_f32_16x16x32_f16(af, bitcast<half8>(w[ct][s]), acc[mt][ct], 0, 0, 0);
      }
    }
  };

  // step kb: load activations and weights of block kb + 2, write block
  // kb + 1's activations to LDS slot (kb + 1) % 3 (last read at step kb - 2),
  // barrier, compute block kb
  u32x4 xr[kLmRing][MT];
  u32x4 wr[kLmRing][kLmCols][4];
#pragma unroll
  for (int j = 0; j < kLmRing - 1; ++j) {
    load_x(j, xr[j]);
    load_w(j, wr[j]);
  }
  store_x(0, xr[0]);
  for (int k0 = 0; k0 < nkb; k0 += kLmRing) {
#pragma unroll
    for (int J = 0; J < kLmRing; ++J) {
      const int kb = k0 + J;
      load_x(kb + kLmRing - 1, xr[(J + kLmRing - 1) % kLmRing]);
      load_w(kb + kLmRing - 1, wr[(J + kLmRing - 1) % kLmRing]);
      if (kb < nkb) {
        if (kb + 1 < nkb) store_x((kb + 1) % kLmRing, xr[(J + 1) % kLmRing]);
        lds_barrier();
        compute(kb % kLmRing, wr[J]);
      } else {
        // retire the slot's loads so that no load into a ring register is
        // pending where the compiler reuses it
#pragma unroll
        for (int j = 0; j < MT; ++j) asm volatile("" : : "v"(xr[(J + 1) % kLmRing][j]));
#pragma unroll
        for (int ct = 0; ct < kLmCols; ++ct)
#pragma unroll
          for (int s = 0; s < 4; ++s) asm volatile("" : : "v"(wr[J][ct][s]));
      }
    }
  }

  // lane holds rows 4 kq + r of column n16 of each tile
#pragma unroll
  for (int ct = 0; ct < kLmCols; ++ct) {
    const int t = tile0 + ct;
    if (t >= ntiles) continue;
    const int col = t * 16 + n16;
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int m = mt * 16 + kq * 4 + r;
        if (m < a.M) a.logits[(size_t)m * a.ldl + col] = f2h(acc[mt][ct][r]);
      }
  }
}

void launch_lm_head(const uint16_t* xn, int M, int H, const uint16_t* W, int V, uint16_t* logits, int ldl,
                    hipStream_t st) {
  LmArgs a{xn, W, logits, M, H, V, ldl};
  const dim3 grid((V / 16 + 4 * kLmCols - 1) / (4 * kLmCols));
  switch ((M + 15) / 16) {
    case 1: hipLaunchKernelGGL(lm_head_kernel<1>, grid, dim3(256), 0, st, a); break;
    case 2: hipLaunchKernelGGL(lm_head_kernel<2>, grid, dim3(256), 0, st, a); break;
    case 3: hipLaunchKernelGGL(lm_head_kernel<3>, grid, dim3(256), 0, st, a); break;
    default: hipLaunchKernelGGL(lm_head_kernel<4>, grid, dim3(256), 0, st, a); break;
  }
}

}  // namespace ss
