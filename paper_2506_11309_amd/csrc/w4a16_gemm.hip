// W4A16 GEMMs at small M (the tree size) for gfx950.
//
// y[m][n] = sum_k x[m][k] * W'[n][k],  W'[n][k] = (q[n][k] - z[n][g]) * s[n][g],
// g = k / 128: the int4 AWQ-style projections of a decoder layer (SwiftSpec
// Sec. 3.3 and Sec. 5.1), plain (+ residual) or as the fused SwiGLU whose
// gate and up tiles share the activation fragments (Sec. 3.3).
//
// Matrix-core mapping (v_mfma_f32_16x16x32_f16, wave64):
//   * A operand = activations in the "prepared" layout (ss_device.h), 16
//     token rows per M-tile; B operand = weights, 16 output columns per
//     N-tile.  Rows >= M are zero.
//   * Lane (n = lane % 16, kq = lane / 16) loads 16 bytes = k in
//     [128 g + 32 kq, +32) of weight row n: one wave-wide load covers one
//     16-column x 128-k block, i.e. exactly one (scale, zero) group.
//   * Dequantisation to exact integers with fp16 "magic numbers": OR-ing the
//     low nibble field into 0x6400 (1024, unit 1) gives 1024 + q, OR-ing the
//     high nibble field (bits 4-7) into 0x5400 (64, unit 1/16) gives 64 + q,
//     and one packed fp16 subtraction of 1024 + z (64 + z) leaves q - z
//     exactly.  Activations are used as given (any fp16 value), each MFMA
//     sum of a group is C_g = sum_k x (q - z), and the accumulator takes
//     s C_g (one mixed-precision FMA per output element, fp16 s read in
//     place).
//   * Stream-K scheduling: a fixed grid of workgroups (4 waves each) splits
//     the (N-block, group) iteration space into equal contiguous ranges; the
//     4 waves split an N-block's columns.  Per group, every wave loads 1 KB
//     contiguous blocks of its own weight tiles and a quarter of the group's
//     activation fragments into a register ring (6 groups deep up to 32
//     rows, 4 above), issued together so that the in-order vmcnt queue never
//     holds a weight prefetch behind an older activation load; the
//     activations pass through a 3-slot LDS ring shared by the 4 waves, with
//     one fence-free barrier per group.  An N-block split between
//     workgroups is published as fp32 partials; a fix-up kernel on the same
//     stream sums them in workgroup order (results are deterministic) and
//     runs the epilogue.  Consecutive ranges are placed on the same XCD
//     (blockIdx % 8 selects the XCD under round-robin dispatch).
#include "ss_device.h"
#include "ss_internal.h"

namespace ss {

// EPI_SWIGLU_SPLIT: the fused SwiGLU with the gate and the up tile of an
// output column in two different waves (waves 0, 1: gate tiles of the
// block's two columns; waves 2, 3: their up tiles), combined through LDS at
// the end: twice the waves of EPI_SWIGLU for the same columns, half the
// dequantisation and MFMA work per wave and step.
enum { EPI_PLAIN = 0, EPI_SWIGLU = 1, EPI_SWIGLU_SPLIT = 2 };

// Kernel-native copy of an int4 matrix (written by prepack_w4_kernel):
//   q : [N/16 tiles][G groups][64 lanes] x 16 bytes -- lane kq*16 + c holds
//       the packed nibbles of k in [128 g + 32 kq, +32) of row 16 t + c, in
//       the original byte order; one wave-wide load is 1 KB contiguous and a
//       tile's groups follow each other;
//   sz: [N/16][G][16] x u32 -- scale (fp16 bits) | zero << 16 of row 16 t + c.
struct W4Ptr {
  const u32x4* q;
  const uint32_t* sz;
};

struct GemmArgs {
  W4Ptr w0, w1;
  int K, N, G;
  const uint16_t* a;  // prepared activations [MT][G][4][64][8]
  int M;
  const uint16_t* x;      // normalised in the kernel: plain rows [M][ldx], RMSNorm weight gamma [K]
  int ldx;
  const uint16_t* gamma;
  float eps;
  uint16_t* y;        // plain output [M][ldy] (nullable)
  int ldy;
  uint16_t* yp;       // prepared output for a following GEMM with K = N (nullable)
  const uint16_t* res;
  int ldr;
  int nblocks, nwg;
  uint32_t units;  // N-blocks x groups; units x nwg < 2^30 (K N / 2 < 2^32)
  float* part;
};

// first unit of workgroup v's range (32-bit: units x nwg stays below 2^30
// because a packed matrix fits a 32-bit buffer range)
__device__ __forceinline__ int range_begin(uint32_t units, int v, int nwg) {
  return (int)((units * (uint32_t)v) / (uint32_t)nwg);
}

template <int MT, int NWV>
struct BStage {
  u32x4 b[NWV];
  uint32_t sz[NWV];
};

// Kernel shapes.  R = register-ring depth (groups whose loads are in flight
// or waiting to be used), OCC = waves per SIMD the register budget is cut
// for, NWG = workgroup cap.  Measured on the Llama-3-70B layer: three
// groups deep at two waves per SIMD everywhere (fewer, deeper-ringed
// workgroups were slower); the SwiGLU stream takes one
// workgroup per N-block when there are enough N-blocks to fill the chip (no
// split, so no partials and no fix-up kernel).
struct GemmShape {
  int ring, occ, nwg;
};
constexpr GemmShape gemm_shape(int MT, bool swiglu) {
  return MT > 2 ? GemmShape{3, 2, 512} : swiglu ? GemmShape{3, 2, 768} : GemmShape{3, 2, 512};
}
constexpr GemmShape gemm_shape_epi(int MT, int EPI) {
  return EPI == EPI_SWIGLU_SPLIT ? GemmShape{MT == 1 ? 4 : 3, 4, 1 << 30} : gemm_shape(MT, EPI == EPI_SWIGLU);
}
constexpr int kRingL = 3;  // LDS ring of activation fragments

// The four MFMA B operands of one 16-column x 128-k weight block as a lane
// holds it (16 bytes w: k in [128 g + 32 kq, +32) of column lane % 16; the
// block's scale|zero word sz), dequantised to exact q - z (see the magic
// numbers above the loop of w4a16_gemm_kernel): low nibbles of the first
// and second 16 k, then high nibbles.  magic_lo / magic_hi hold 0x64006400
// and 0x54005400 in registers.
struct BFrag {
  half8 lo_a, lo_b, hi_a, hi_b;
};
__device__ __forceinline__ BFrag dequant_block(u32x4 w, uint32_t sz, uint32_t magic_lo, uint32_t magic_hi) {
  auto deq = [&](uint32_t x, uint32_t m, uint32_t magic, half2v zz) {
    return bitcast<uint32_t>(bitcast<half2v>((x & m) | (magic & ~m)) - zz);
  };
  const uint32_t s0 = w[0] >> 8, s1 = w[1] >> 8, s2 = w[2] >> 8, s3 = w[3] >> 8;
  constexpr uint32_t kLo = 0x000F000Fu, kHi = 0x00F000F0u;
  const uint32_t z = (sz >> 16) & 0xFFu;
  const half2v zlo = bitcast<half2v>((0x6400u + z) * 0x00010001u);
  const half2v zhi = bitcast<half2v>((0x5400u + 16u * z) * 0x00010001u);
  auto dl = [&](uint32_t x) { return deq(x, kLo, magic_lo, zlo); };
  auto dh = [&](uint32_t x) { return deq(x, kHi, magic_hi, zhi); };
  BFrag f;
  f.lo_a = bitcast<half8>(u32x4{dl(w[0]), dl(s0), dl(w[1]), dl(s1)});
  f.lo_b = bitcast<half8>(u32x4{dl(w[2]), dl(s2), dl(w[3]), dl(s3)});
  f.hi_a = bitcast<half8>(u32x4{dh(w[0]), dh(s0), dh(w[1]), dh(s1)});
  f.hi_b = bitcast<half8>(u32x4{dh(w[2]), dh(s2), dh(w[3]), dh(s3)});
  return f;
}

// Output epilogue of one N-block from the accumulators of wave `wave`
// (kColW column tiles, for SwiGLU followed by the matching up tiles): lane
// holds rows 4 * (lane / 16) + r of column lane % 16 of each tile.  The
// residual is read first (load_residual) so that its loads can overlap
// other loads of the caller.
template <int MT, int NWV, int EPI>
struct Epilogue {
  static constexpr int kColW = (EPI == EPI_SWIGLU) ? NWV / 2 : NWV;
  static constexpr int kColB = 4 * kColW;
  float rv[MT][kColW][4];

  // rows m0 + 16 mt + ... (m0: first row of the caller's M-tiles)
  __device__ __forceinline__ void load_residual(const GemmArgs& a, int nb, int wave, int lane, int m0 = 0) {
    const int ncol = lane & 15, kq = lane >> 4;
    const int col0 = (nb * kColB + wave * kColW) * 16;
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
      for (int ct = 0; ct < kColW; ++ct)
#pragma unroll
        for (int r = 0; r < 4; ++r) rv[mt][ct][r] = 0.f;
    if (EPI == EPI_PLAIN && a.res) {
      // rows >= M read row 0 and are discarded
#pragma unroll
      for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int ct = 0; ct < kColW; ++ct)
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const int m = m0 + mt * 16 + kq * 4 + r;
            rv[mt][ct][r] = h2f(a.res[(size_t)(m < a.M ? m : 0) * a.ldr + col0 + ct * 16 + ncol]);
          }
    }
  }

  __device__ __forceinline__ void write(const GemmArgs& a, int nb, int wave, int lane,
                                        const f32x4 (&acc)[MT][NWV], int m0 = 0) const {
    const int ncol = lane & 15, kq = lane >> 4;
    const int col0 = (nb * kColB + wave * kColW) * 16;
    const int G2 = a.N >> 7;
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
      for (int ct = 0; ct < kColW; ++ct) {
        const int ncl = col0 + ct * 16 + ncol;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int m = m0 + mt * 16 + kq * 4 + r;
          if (m < a.M) {
            float val;
            if (EPI == EPI_SWIGLU) {
              const float gte = acc[mt][ct][r], up = acc[mt][ct + kColW][r];
              val = gte / (1.0f + __expf(-gte)) * up;
            } else {
              val = acc[mt][ct][r] + rv[mt][ct][r];
            }
            const uint16_t h = f2h(val);
            if (a.y) a.y[(size_t)m * a.ldy + ncl] = h;
            if (a.yp) store_prepared(a.yp, m, ncl, G2, h);
          }
        }
      }
  }
};

// Partial-sum slots: workgroup v publishes the accumulators of its range's
// first (slot 0) and last (slot 1) N-block when another range shares them;
// per slot, wave w's MT x kColW x kSrc fragments of 64 lanes x f32x4.  Plain
// stores and loads: the fix-up runs in the next kernel on the stream.
template <int MT, int NWV, int EPI>
__device__ __forceinline__ float* part_slot(const GemmArgs& a, int v, int slot, int wave) {
  constexpr int kColW = (EPI == EPI_SWIGLU) ? NWV / 2 : NWV;
  constexpr int kSrc = (EPI == EPI_SWIGLU) ? 2 : 1;
  constexpr int kWaveSlotFloats = MT * kColW * kSrc * kWave * 4;
  return a.part + (((size_t)v * 2 + slot) * 4 + wave) * kWaveSlotFloats;
}

template <int MT, int NWV, int EPI>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(gemm_shape_epi(MT, EPI).occ)))
void w4a16_gemm_kernel(GemmArgs a) {
  constexpr bool kSplit = EPI == EPI_SWIGLU_SPLIT;
  constexpr int kColW = (EPI == EPI_SWIGLU) ? NWV / 2 : NWV;  // output column tiles per wave
  constexpr int kColB = kSplit ? 2 : 4 * kColW;                // output column tiles per block
  constexpr int kSrc = (EPI == EPI_SWIGLU) ? 2 : 1;
  constexpr int kRing = gemm_shape_epi(MT, EPI).ring;
  static_assert(!kSplit || NWV == 1, "split SwiGLU: one tile per wave");
  __shared__ u32x4 abuf[kRingL][MT][4][kWave];  // activation fragments of 3 groups
  __shared__ f32x4 xch[kSplit ? 2 : 1][MT][kWave];  // split SwiGLU: the up sums for the gate waves

  const int tid = threadIdx.x;
  const int lane = lane_id();
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // uniform: scalar addressing
  const int ncol = lane & 15;
  const int kq = lane >> 4;
  const int G = a.G;
  const int b = blockIdx.x;
  const int v = (a.nwg % 8 == 0) ? (b % 8) * (a.nwg / 8) + b / 8 : b;
  const int u_lo = range_begin(a.units, v, a.nwg), u_hi = range_begin(a.units, v + 1, a.nwg);
  const int total = u_hi - u_lo;
  if (total <= 0) return;

  // Load cursor: unit u = (N-block u / G, group u % G), advanced once per
  // load step and held at the range's last unit (loads past the end repeat
  // it, so every step issues the same operations).
  int ld_i = 0, ld_nb = u_lo / G, ld_g = u_lo - (u_lo / G) * G;
  auto advance = [&]() {
    if (ld_i < total - 1) {
      ++ld_i;
      if (++ld_g == G) {
        ld_g = 0;
        ++ld_nb;
      }
    }
  };
  // Operand loads go through buffer resources: the wave-uniform part of an
  // address is a scalar offset and the lane's part a constant vector offset,
  // so a load costs no vector ALU work.
  const uint32_t q_bytes = (uint32_t)((size_t)a.K * a.N / 2), sz_bytes = (uint32_t)((size_t)a.N * G * 4);
  const auto rq0 = buffer_rsrc(a.w0.q, q_bytes), rs0 = buffer_rsrc(a.w0.sz, sz_bytes);
  const auto rq1 = buffer_rsrc(EPI != EPI_PLAIN ? a.w1.q : a.w0.q, q_bytes);
  const auto rs1 = buffer_rsrc(EPI != EPI_PLAIN ? a.w1.sz : a.w0.sz, sz_bytes);
  const auto ra = buffer_rsrc(a.a, (uint32_t)(MT * G * 4 * kWave * 16));
  const uint32_t lane16 = (uint32_t)lane * 16u, col4 = (uint32_t)ncol * 4u;
  auto load_b = [&](BStage<MT, NWV>& st) {
    const int tw = ld_nb * kColB + (kSplit ? (wave & 1) : wave * kColW);  // first column tile of this wave
#pragma unroll
    for (int nt = 0; nt < NWV; ++nt) {
      const bool up = (EPI == EPI_SWIGLU && nt >= kColW) || (kSplit && wave >= 2);
      const uint32_t tg = (uint32_t)((tw + nt % kColW) * G + ld_g);
      st.b[nt] = buffer_load_x4(up ? rq1 : rq0, lane16, tg * 1024u);
      st.sz[nt] = buffer_load_x1(up ? rs1 : rs0, col4, tg * 64u);
    }
  };
  // wave w stages fragment w of every M-tile of the cursor's group; with
  // one M-tile, lanes of rows at or past M load nothing (those rows are
  // zeros in the prepared layout; whatever the register holds reaches only
  // output rows that are not written)
  auto load_a = [&](u32x4 (&r)[MT]) {
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
      if (MT > 1 || ncol < a.M) r[mt] = buffer_load_x4(ra, lane16, (uint32_t)(((mt * G + ld_g) * 4 + wave) * 1024));
  };
  auto store_a = [&](int slot, const u32x4 (&r)[MT]) {
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) abuf[slot][mt][wave][lane] = r[mt];
  };

  f32x4 acc[MT][NWV];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int nt = 0; nt < NWV; ++nt) acc[mt][nt] = f32x4{0.f, 0.f, 0.f, 0.f};

  // Dequantisation to exact small integers: (w & 0x000F000F) | 0x64006400
  // is the fp16 pair (1024 + q, 1024 + q'), (w & 0x00F000F0) | 0x54005400 is
  // (64 + q, 64 + q') (the nibble sits at the 1/16 ... 1/2 mantissa bits of
  // 64, i.e. at units 1 ... 8); subtracting 1024 + z (resp. 64 + z) leaves
  // q - z exactly.  The MFMA sum of a group is C_g = sum_k x (q - z) and the
  // accumulator takes s C_g.  The magic constants are kept in registers
  // (opaque to the optimiser) so that mask-and-insert is one v_bfi_b32 with
  // the mask in a scalar register.
  uint32_t magic_lo = 0x64006400u, magic_hi = 0x54005400u;
  asm volatile("" : "+v"(magic_lo), "+v"(magic_hi));
  auto read_a = [&](int slot, half8 (&af)[MT][4]) {
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
      for (int f = 0; f < 4; ++f) af[mt][f] = bitcast<half8>(abuf[slot][mt][f][lane]);
  };
  // group sums C_g of one unit (and the tiles' scale words); applied to the
  // accumulators one step later, so that no instruction waits on the MFMAs
  // just issued
  auto mfma_unit = [&](const half8 (&af)[MT][4], const BStage<MT, NWV>& st, f32x4 (&c)[MT][NWV],
                       uint32_t (&sw)[NWV]) {
#pragma unroll
    for (int nt = 0; nt < NWV; ++nt) {
      const BFrag bf = dequant_block(st.b[nt], st.sz[nt], magic_lo, magic_hi);
      sw[nt] = st.sz[nt];
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) {
        f32x4 cc = {0.f, 0.f, 0.f, 0.f};
        cc = __builtin_amdgcn_mfma_f32_16x16x32_f16(af[mt][0], bf.lo_a, cc, 0, 0, 0);
        cc = __builtin_amdgcn_mfma_f32_16x16x32_f16(af[mt][1], bf.lo_b, cc, 0, 0, 0);
        cc = __builtin_amdgcn_mfma_f32_16x16x32_f16(af[mt][2], bf.hi_a, cc, 0, 0, 0);
        cc = __builtin_amdgcn_mfma_f32_16x16x32_f16(af[mt][3], bf.hi_b, cc, 0, 0, 0);
        c[mt][nt] = cc;
      }
    }
  };
  auto apply = [&](const f32x4 (&c)[MT][NWV], const uint32_t (&sw)[NWV]) {
#pragma unroll
    for (int nt = 0; nt < NWV; ++nt)
#pragma unroll
      for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int r = 0; r < 4; ++r)
          acc[mt][nt][r] = __builtin_fmaf(c[mt][nt][r], (float)bitcast<half2v>(sw[nt])[0], acc[mt][nt][r]);
  };

  auto emit = [&](int nb) {
    Epilogue<MT, NWV, EPI> ep;
    ep.load_residual(a, nb, wave, lane);
    ep.write(a, nb, wave, lane, acc);
  };
  auto zero_acc = [&]() {
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
      for (int nt = 0; nt < NWV; ++nt) acc[mt][nt] = f32x4{0.f, 0.f, 0.f, 0.f};
  };
  // End of an N-block's share inside the range: write the outputs if the
  // range holds the whole N-block, else publish the partial (slot 0: the
  // range's first N-block, slot 1: its last) for the fix-up kernel.
  auto flush = [&](int nb) {
    const bool full = (long)nb * G >= u_lo && (long)(nb + 1) * G <= u_hi;
    if constexpr (kSplit) {
      // every range holds whole blocks: the up waves hand their sums to the
      // gate waves of the same columns, which write silu(gate) * up
      if (wave >= 2) {
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) xch[wave - 2][mt][lane] = acc[mt][0];
      }
      __syncthreads();
      if (wave < 2) {
        const int col = (nb * kColB + wave) * 16 + ncol;
        const int G2 = a.N >> 7;
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) {
          const f32x4 u = xch[wave][mt][lane];
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const int m = mt * 16 + kq * 4 + r;
            if (m < a.M) {
              const float gte = acc[mt][0][r];
              const uint16_t h = f2h(gte / (1.0f + __expf(-gte)) * u[r]);
              if (a.y) a.y[(size_t)m * a.ldy + col] = h;
              if (a.yp) store_prepared(a.yp, m, col, G2, h);
            }
          }
        }
      }
      __syncthreads();  // the exchange buffer is free for the range's next block
      (void)full;
    } else if (full) {
      emit(nb);
    } else {
      float* mine = part_slot<MT, NWV, EPI>(a, v, nb == u_lo / G ? 0 : 1, wave);
#pragma unroll
      for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int ct = 0; ct < kColW; ++ct) {
          const int t = mt * kColW + ct;
          *reinterpret_cast<f32x4*>(mine + ((size_t)(t * kSrc) * kWave + lane) * 4) = acc[mt][ct];
          if (EPI == EPI_SWIGLU)
            *reinterpret_cast<f32x4*>(mine + ((size_t)(t * kSrc + 1) * kWave + lane) * 4) = acc[mt][ct + kColW];
        }
    }
    zero_acc();
  };


  // ---- one continuous pipeline over the range's units ----
  // Step i (R = ring depth): issue the activation and weight loads of unit
  // i + R - 1 into register slot (i + R - 1) % R, write unit i + 1's
  // activation fragments (loaded R - 2 steps earlier; the compiler waits
  // for exactly that load) to LDS slot (i + 1) % 3 (last read at step
  // i - 2), barrier, compute unit i (whose fragments were written at step
  // i - 1) and flush when unit i ends its N-block's share.  Loads past the range's
  // end repeat its last unit (L2 hits), so every step issues the same
  // operations and the compiler's waits stay exact; the loop runs whole
  // rounds of R steps.
  BStage<MT, NWV> bs[kRing];
  u32x4 ar[kRing][MT];
#pragma unroll
  for (int j = 0; j < kRing - 1; ++j) {
    load_a(ar[j]);
    load_b(bs[j]);
    advance();
  }
  store_a(0, ar[0]);

  // a step past the range's end still retires its register slot, so that no
  // load into a ring register is pending where the compiler reuses it
  auto consume = [&](const BStage<MT, NWV>& st, const u32x4 (&r)[MT]) {
#pragma unroll
    for (int nt = 0; nt < NWV; ++nt) asm volatile("" : : "v"(st.b[nt]), "v"(st.sz[nt]));
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) asm volatile("" : : "v"(r[mt]));
  };
  // Up to 32 rows the fragments and group sums are double-buffered: at step i
  // the wave reads unit i + 1's fragments (its LDS slot is complete once the
  // barrier of step i has passed) and applies unit i - 1's sums.  Above 32
  // rows the second buffers would cost the second wave per SIMD, so step i
  // reads, multiplies and applies its own unit.
  constexpr bool kPipe = MT <= 2 && !kSplit;
  constexpr int kBuf = kPipe ? 2 : 1;
  half8 af[kBuf][MT][4];
  f32x4 cs[kBuf][MT][NWV];
  uint32_t sc[kBuf][NWV];
#pragma unroll
  for (int q = 0; q < kBuf; ++q)
#pragma unroll
    for (int nt = 0; nt < NWV; ++nt) {
      sc[q][nt] = 0u;
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) cs[q][mt][nt] = f32x4{0.f, 0.f, 0.f, 0.f};
    }
  lds_barrier();
  if constexpr (kPipe) read_a(0, af[0]);
  // compute cursor: N-block and group of unit i
  int c_nb = u_lo / G, c_g = u_lo - (u_lo / G) * G;
  for (int i0 = 0; i0 < total; i0 += 2 * kRing) {
#pragma unroll
    for (int J = 0; J < 2 * kRing; ++J) {
      const int i = i0 + J;
      const int R = J % kRing, bq = kPipe ? (J & 1) : 0;
      load_a(ar[(R + kRing - 1) % kRing]);
      load_b(bs[(R + kRing - 1) % kRing]);
      advance();
      if (i < total) {
        if (i + 1 < total) store_a((i + 1) % kRingL, ar[(R + 1) % kRing]);
        lds_barrier();
        if constexpr (kPipe) {
          if (i + 1 < total) read_a((i + 1) % kRingL, af[bq ^ 1]);
          mfma_unit(af[bq], bs[R], cs[bq], sc[bq]);
          apply(cs[bq ^ 1], sc[bq ^ 1]);
        } else {
          read_a(i % kRingL, af[0]);
          mfma_unit(af[0], bs[R], cs[0], sc[0]);
        }
        if (i == total - 1 || c_g == G - 1) {
          apply(cs[bq], sc[bq]);
#pragma unroll
          for (int nt = 0; nt < NWV; ++nt) sc[bq][nt] = 0u;
          flush(c_nb);
        } else if constexpr (!kPipe) {
          apply(cs[0], sc[0]);
        }
        if (++c_g == G) {
          c_g = 0;
          ++c_nb;
        }
      } else {
        consume(bs[R], ar[(R + 1) % kRing]);
      }
    }
  }
}

// Split N-blocks: one workgroup per M-tile of an N-block (grid MT times the
// N-blocks) sums that tile's partials of the block's contributing ranges in
// workgroup order (deterministic) and writes its 16 rows; N-blocks inside
// one range were written by the GEMM kernel.  (One workgroup for all M-tiles
// of a block was slower: at 32 rows 20.4 -> 19.1 us for the 70B QKV, 35.3
// -> 34.1 us for the down projection; at 64 rows 51.4 -> 48.6 us for the
// down projection, whose one-workgroup form needs 256 VGPRs.)
template <int MT, int NWV, int EPI>
__global__ __launch_bounds__(256) void w4a16_fixup_kernel(GemmArgs a) {
  constexpr int MS = 1;  // M-tiles per workgroup
  constexpr int kBatch = 8;
  constexpr int kColW = (EPI == EPI_SWIGLU) ? NWV / 2 : NWV;
  constexpr int kSrc = (EPI == EPI_SWIGLU) ? 2 : 1;
  // the GEMM orders its ranges XCD-major (workgroup b on XCD b % 8 takes
  // range (b % 8) nwg/8 + b / 8), so the blocks of XCD x are the x-th eighth
  // of all blocks: fix-up workgroup (b, M-tile group) takes one of those of
  // its own XCD (b % 8, the grid holding MT copies of the blocks),
  // whose partials that XCD's L2 wrote
  const int b = blockIdx.x % a.nblocks;
  const int mt0 = blockIdx.x / a.nblocks;  // this workgroup's M-tile
  const int nb = (a.nwg % 8 == 0 && a.nblocks % 8 == 0) ? (b % 8) * (a.nblocks / 8) + b / 8 : b;
  const uint32_t U = a.units, lo = (uint32_t)(nb * a.G), nwg = (uint32_t)a.nwg;
  const int c_first = (int)(((lo + 1) * nwg - 1) / U);
  const int c_last = (int)(((lo + (uint32_t)a.G) * nwg - 1) / U);
  if (c_first == c_last) return;
  // every contributor after the first begins its range inside this block
  // (slot 0, its first block); the first one holds it in slot 1 (its last
  // block) unless its range begins exactly at the block
  const int slot_first = range_begin(U, c_first, a.nwg) < (int)lo ? 1 : 0;
  const int lane = lane_id();
  const int wave = __builtin_amdgcn_readfirstlane((int)threadIdx.x >> 6);
  Epilogue<MS, NWV, EPI> ep;
  ep.load_residual(a, nb, wave, lane, mt0 * 16);  // in flight with the first partial loads
  f32x4 acc[MS][NWV];
#pragma unroll
  for (int mt = 0; mt < MS; ++mt)
#pragma unroll
    for (int nt = 0; nt < NWV; ++nt) acc[mt][nt] = f32x4{0.f, 0.f, 0.f, 0.f};
  for (int c0 = c_first; c0 <= c_last; c0 += kBatch) {
    // kBatch contributors' loads in flight at once, summed in order
    f32x4 pa[kBatch][MS][kColW], pb[kBatch][MS][kColW];
#pragma unroll
    for (int j = 0; j < kBatch; ++j) {
      const int c = c0 + j <= c_last ? c0 + j : c_last;
      const float* src = part_slot<MT, NWV, EPI>(a, c, c == c_first ? slot_first : 0, wave);
#pragma unroll
      for (int mt = 0; mt < MS; ++mt)
#pragma unroll
        for (int ct = 0; ct < kColW; ++ct) {
          const int t = (mt0 + mt) * kColW + ct;
          pa[j][mt][ct] = *reinterpret_cast<const f32x4*>(src + ((size_t)(t * kSrc) * kWave + lane) * 4);
          if (EPI == EPI_SWIGLU) pb[j][mt][ct] = *reinterpret_cast<const f32x4*>(src + ((size_t)(t * kSrc + 1) * kWave + lane) * 4);
        }
    }
#pragma unroll
    for (int j = 0; j < kBatch; ++j) {
      if (c0 + j > c_last) break;
#pragma unroll
      for (int mt = 0; mt < MS; ++mt)
#pragma unroll
        for (int ct = 0; ct < kColW; ++ct) {
          acc[mt][ct] += pa[j][mt][ct];
          if (EPI == EPI_SWIGLU) acc[mt][ct + kColW] += pb[j][mt][ct];
        }
    }
  }
  ep.write(a, nb, wave, lane, acc, mt0 * 16);
}

// ------------------------------------------------- small M, small weights
// Up to 16 rows and a few megabytes of weights (the 1B-shaped layer's and
// the 8B-shaped layer's QKV and O projections, tensor-parallel shards) the
// stream-K kernel's time is its fixed costs: first loads, the split
// partials and the fix-up kernel.  Here one workgroup owns one 16-column
// output tile over the whole K range: its W waves take contiguous group
// ranges, each streaming its own weight blocks and activation fragments
// (the prepared layout's four fragments of the group, straight into the
// MFMA A operand) through a 3-deep register ring, and the W partial sums
// are added in wave order through LDS (results deterministic), then wave 0
// adds the residual and writes the tile.  No partials leave the workgroup
// and no second kernel runs.  Every workgroup reads the whole activation
// matrix (from L2): four times the weight bytes, which is why the plan
// keeps it to small weights.

template <int W, int NT>
__global__ __launch_bounds__(64 * W) void w4a16_kslice_kernel(GemmArgs a) {
  constexpr int kR = 3;
  static_assert(NT == 1 || NT == 2, "plain, or fused SwiGLU (gate and up tile of one column tile)");
  __shared__ f32x4 red[W][NT][kWave];
  const int lane = lane_id();
  const int wave = __builtin_amdgcn_readfirstlane((int)threadIdx.x >> 6);
  const int ncol = lane & 15, kq = lane >> 4;
  const int t = blockIdx.x;
  const int G = a.G;
  const int g0 = wave * G / W, n = (wave + 1) * G / W - g0;  // >= 1: the plan keeps G >= W
  const uint32_t q_bytes = (uint32_t)((size_t)a.K * a.N / 2), sz_bytes = (uint32_t)((size_t)a.N * G * 4);
  const auto rq0 = buffer_rsrc(a.w0.q, q_bytes), rs0 = buffer_rsrc(a.w0.sz, sz_bytes);
  const auto rq1 = buffer_rsrc(NT == 2 ? a.w1.q : a.w0.q, q_bytes);
  const auto rs1 = buffer_rsrc(NT == 2 ? a.w1.sz : a.w0.sz, sz_bytes);
  const auto ra = buffer_rsrc(a.a, (uint32_t)(G * 4 * kWave * 16));
  const uint32_t lane16 = (uint32_t)lane * 16u, col4 = (uint32_t)ncol * 4u;
  struct Stage {
    u32x4 b[NT];
    uint32_t sz[NT];
    u32x4 x[4];
  };
  // group i of this wave's range (loads past its end repeat its last group)
  auto load = [&](Stage& st, int i) {
    const int g = g0 + (i < n ? i : n - 1);
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      const uint32_t tg = (uint32_t)(t * G + g);
      st.b[nt] = buffer_load_x4(nt ? rq1 : rq0, lane16, tg * 1024u);
      st.sz[nt] = buffer_load_x1(nt ? rs1 : rs0, col4, tg * 64u);
    }
    // lanes of rows at or past M load nothing (zeros in the prepared
    // layout; the MFMA rows they feed are not written)
    if (ncol < a.M) {
#pragma unroll
      for (int f = 0; f < 4; ++f) st.x[f] = buffer_load_x4(ra, lane16, (uint32_t)((g * 4 + f) * 1024));
    }
  };
  uint32_t magic_lo = 0x64006400u, magic_hi = 0x54005400u;
  asm volatile("" : "+v"(magic_lo), "+v"(magic_hi));
  f32x4 acc[NT];
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) acc[nt] = f32x4{0.f, 0.f, 0.f, 0.f};
  Stage ring[kR];
#pragma unroll
  for (int j = 0; j < kR - 1; ++j) load(ring[j], j);
  for (int i0 = 0; i0 < n; i0 += kR) {
#pragma unroll
    for (int J = 0; J < kR; ++J) {
      const int i = i0 + J;
      load(ring[(J + kR - 1) % kR], i + kR - 1);
      const Stage& st = ring[J];
      if (i < n) {
        const u32x4* xa = st.x;
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) {
          const BFrag bf = dequant_block(st.b[nt], st.sz[nt], magic_lo, magic_hi);
          f32x4 cc = {0.f, 0.f, 0.f, 0.f};
          cc = __builtin_amdgcn_mfma_f32_16x16x32_f16(bitcast<half8>(xa[0]), bf.lo_a, cc, 0, 0, 0);
          cc = __builtin_amdgcn_mfma_f32_16x16x32_f16(bitcast<half8>(xa[1]), bf.lo_b, cc, 0, 0, 0);
          cc = __builtin_amdgcn_mfma_f32_16x16x32_f16(bitcast<half8>(xa[2]), bf.hi_a, cc, 0, 0, 0);
          cc = __builtin_amdgcn_mfma_f32_16x16x32_f16(bitcast<half8>(xa[3]), bf.hi_b, cc, 0, 0, 0);
#pragma unroll
          for (int r = 0; r < 4; ++r)
            acc[nt][r] = __builtin_fmaf(cc[r], (float)bitcast<half2v>(st.sz[nt])[0], acc[nt][r]);
        }
      } else {
        // retire the slot's pending loads before the registers are reused
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) asm volatile("" : : "v"(st.b[nt]), "v"(st.sz[nt]));
#pragma unroll
        for (int f = 0; f < 4; ++f) asm volatile("" : : "v"(st.x[f]));
      }
    }
  }
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) red[wave][nt][lane] = acc[nt];
  __syncthreads();
  if (wave != 0) return;
  f32x4 sum[NT];
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) {
    sum[nt] = red[0][nt][lane];
#pragma unroll
    for (int w = 1; w < W; ++w) sum[nt] += red[w][nt][lane];
  }
  const int col = t * 16 + ncol;
  const int G2 = a.N >> 7;
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int m = 4 * kq + r;
    if (m < a.M) {
      float val;
      if constexpr (NT == 2) {
        const float gte = sum[0][r];
        val = gte / (1.0f + __expf(-gte)) * sum[1][r];
      } else {
        val = sum[0][r] + (a.res ? h2f(a.res[(size_t)m * a.ldr + col]) : 0.f);
      }
      const uint16_t h = f2h(val);
      if (a.y) a.y[(size_t)m * a.ldy + col] = h;
      if (a.yp) store_prepared(a.yp, m, col, G2, h);
    }
  }
}


// ------------------------------------------- small M, RMSNorm in the GEMM
// The QKV projection and the fused SwiGLU read the RMSNorm of the residual
// stream (the decoder layer of Sec. 2).  Where the K-split plan gives each
// wave at most NG (2 or 4) groups, the workgroup (which reads all of K
// anyway) normalises the plain rows x itself: every wave issues all its
// loads up front (the row chunks of its groups, gamma, then the weight
// blocks, so that the row sums wait for the row chunks only), sums x^2
// over its groups, the waves' sums meet in LDS,
// and each lane forms its operand values exactly as the norm kernel does,
// fp16((x * inv) * gamma) in fp32, inv = 1 / sqrt(sum_k x^2 / K + eps), so
// the operand is rounded where the unfused chain rounds it.  Rows at or
// past M lie outside the buffer range of x and load as zeros, without a
// branch.  The rows of one load sit at one stride (often a multiple of
// 4 KB), and lanes reading the same 16-byte position of their rows collide
// in the vector cache (a row stride of 4 KB + 16 B was 0.8 us faster on the
// 1B-shaped QKV, one of 4 KB + 128 B no faster): load f of row r takes the
// 16-byte chunk f ^ (r & 3) and two rounds of bitwise lane selects put the
// chunks back in order.
template <int W, int NT, int NG>
__global__ __launch_bounds__(64 * W) void w4a16_kslice_norm_kernel(GemmArgs a) {
  static_assert(NT == 1 || NT == 2, "plain, or fused SwiGLU (gate and up tile of one column tile)");
  static_assert(NG == 2 || NG == 4, "groups per wave");
  __shared__ f32x4 red[W][NT][kWave];
  __shared__ float red_ss[W][16];
  __shared__ u32x4 gam[W][kWave];
  const int lane = lane_id();
  const int wave = __builtin_amdgcn_readfirstlane((int)threadIdx.x >> 6);
  const int ncol = lane & 15, kq = lane >> 4;
  const int t = blockIdx.x;
  const int G = a.G;
  const int g0 = wave * G / W, n = (wave + 1) * G / W - g0;  // 1 .. NG: the plan keeps W <= G <= NG W
  const uint32_t q_bytes = (uint32_t)((size_t)a.K * a.N / 2), sz_bytes = (uint32_t)((size_t)a.N * G * 4);
  const auto rq0 = buffer_rsrc(a.w0.q, q_bytes), rs0 = buffer_rsrc(a.w0.sz, sz_bytes);
  const auto rq1 = buffer_rsrc(NT == 2 ? a.w1.q : a.w0.q, q_bytes);
  const auto rs1 = buffer_rsrc(NT == 2 ? a.w1.sz : a.w0.sz, sz_bytes);
  const auto rx = buffer_rsrc(a.x, (uint32_t)((size_t)a.M * a.ldx * 2));
  // gamma over this wave's groups only (chunk c = 16 j + 4 kq + f of group
  // g0 + j); chunks past them load as zeros
  const auto rgm = buffer_rsrc(a.gamma + g0 * 128, (uint32_t)(n * 256));
  const uint32_t lane16 = (uint32_t)lane * 16u, col4 = (uint32_t)ncol * 4u;
  // this lane's 32 values k = 128 g + 32 kq + t of row ncol, at g = 0
  const uint32_t xrow = (uint32_t)((ncol * a.ldx + 32 * kq) * 2);
  const int xsw = ncol & 3;  // load f takes chunk f ^ xsw
  const uint32_t xm1 = 0u - (uint32_t)(xsw & 1), xm2 = 0u - (uint32_t)(xsw >> 1);

  // the row chunks first, then gamma, then the weights: the row sums wait
  // for the first loads only, while the weight blocks are still in flight
  u32x4 b[NG][NT], x[NG][4];
  uint32_t sz[NG][NT];
#pragma unroll
  for (int j = 0; j < NG; ++j) {
    const int g = g0 + (j < n ? j : n - 1);  // past the range: repeat the last group, unused
#pragma unroll
    for (int f = 0; f < 4; ++f) x[j][f] = buffer_load_x4(rx, xrow + (uint32_t)((f ^ xsw) * 16), (uint32_t)(g * 256));
  }
  const u32x4 gv = buffer_load_x4(rgm, lane16, 0);
#pragma unroll
  for (int j = 0; j < NG; ++j) {
    const int g = g0 + (j < n ? j : n - 1);
    const uint32_t tg = (uint32_t)(t * G + g);
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      b[j][nt] = buffer_load_x4(nt ? rq1 : rq0, lane16, tg * 1024u);
      sz[j][nt] = buffer_load_x1(nt ? rs1 : rs0, col4, tg * 64u);
    }
  }
  gam[wave][lane] = gv;

  // chunk c is in load c ^ xsw: bitwise selects under the masks xm1, xm2 (a
  // conditional operator here becomes an indexed copy through scratch
  // memory); then this wave's part of each row's sum of squares
  float ssq = 0.f;
#pragma unroll
  for (int j = 0; j < NG; ++j) {
    u32x4 t1[4];
#pragma unroll
    for (int c = 0; c < 4; ++c)
#pragma unroll
      for (int e = 0; e < 4; ++e) t1[c][e] = (x[j][c ^ 1][e] & xm1) | (x[j][c][e] & ~xm1);
#pragma unroll
    for (int c = 0; c < 4; ++c)
#pragma unroll
      for (int e = 0; e < 4; ++e) x[j][c][e] = (t1[c ^ 2][e] & xm2) | (t1[c][e] & ~xm2);
    if (j < n) {
#pragma unroll
      for (int c = 0; c < 4; ++c)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const half2v v = bitcast<half2v>(x[j][c][e]);
          ssq = __builtin_amdgcn_fdot2(v, v, ssq, false);
        }
    }
  }
  ssq += __shfl_xor(ssq, 16, kWave);
  ssq += __shfl_xor(ssq, 32, kWave);
  if (kq == 0) red_ss[wave][ncol] = ssq;
  __syncthreads();
  float tot = red_ss[0][ncol];
#pragma unroll
  for (int w = 1; w < W; ++w) tot += red_ss[w][ncol];
  const float inv = 1.0f / sqrtf(tot / (float)a.K + a.eps);

  uint32_t magic_lo = 0x64006400u, magic_hi = 0x54005400u;
  asm volatile("" : "+v"(magic_lo), "+v"(magic_hi));
  f32x4 acc[NT];
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) acc[nt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int j = 0; j < NG; ++j) {
    if (j < n) {
      uint32_t w[16];
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        const u32x4 gm = gam[wave][16 * j + 4 * kq + c];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          // (x * inv) * gamma, each product rounded to fp32, then to fp16:
          // fused multiply-adds of +0 are those products (up to the sign
          // of an exact zero) and take the fp16 operands directly
          const half2v v = bitcast<half2v>(x[j][c][e]), gg = bitcast<half2v>(gm[e]);
          half2v o;
          o[0] = (_Float16)__builtin_fmaf(__builtin_fmaf((float)v[0], inv, 0.f), (float)gg[0], 0.f);
          o[1] = (_Float16)__builtin_fmaf(__builtin_fmaf((float)v[1], inv, 0.f), (float)gg[1], 0.f);
          w[4 * c + e] = bitcast<uint32_t>(o);
        }
      }
      u32x4 xa[4];
      pack_prepared(w, xa);
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) {
        const BFrag bf = dequant_block(b[j][nt], sz[j][nt], magic_lo, magic_hi);
        f32x4 cc = {0.f, 0.f, 0.f, 0.f};
        cc = __builtin_amdgcn_mfma_f32_16x16x32_f16(bitcast<half8>(xa[0]), bf.lo_a, cc, 0, 0, 0);
        cc = __builtin_amdgcn_mfma_f32_16x16x32_f16(bitcast<half8>(xa[1]), bf.lo_b, cc, 0, 0, 0);
        cc = __builtin_amdgcn_mfma_f32_16x16x32_f16(bitcast<half8>(xa[2]), bf.hi_a, cc, 0, 0, 0);
        cc = __builtin_amdgcn_mfma_f32_16x16x32_f16(bitcast<half8>(xa[3]), bf.hi_b, cc, 0, 0, 0);
#pragma unroll
        for (int r = 0; r < 4; ++r)
          acc[nt][r] = __builtin_fmaf(cc[r], (float)bitcast<half2v>(sz[j][nt])[0], acc[nt][r]);
      }
    }
  }
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) red[wave][nt][lane] = acc[nt];
  __syncthreads();
  if (wave != 0) return;
  f32x4 sum[NT];
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) {
    sum[nt] = red[0][nt][lane];
#pragma unroll
    for (int w = 1; w < W; ++w) sum[nt] += red[w][nt][lane];
  }
  const int col = t * 16 + ncol;
  const int G2 = a.N >> 7;
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int m = 4 * kq + r;
    if (m < a.M) {
      float val;
      if constexpr (NT == 2) {
        const float gte = sum[0][r];
        val = gte / (1.0f + __expf(-gte)) * sum[1][r];
      } else {
        val = sum[0][r] + (a.res ? h2f(a.res[(size_t)m * a.ldr + col]) : 0.f);
      }
      const uint16_t h = f2h(val);
      if (a.y) a.y[(size_t)m * a.ldy + col] = h;
      if (a.yp) store_prepared(a.yp, m, col, G2, h);
    }
  }
}

// ------------------------------------------------------- activation prep
// x [M][ldx] fp16 -> prepared layout; one thread per (M-tile, group, lane).
__global__ __launch_bounds__(256) void prepare_activations_kernel(const uint16_t* __restrict__ x, int M,
                                                                  int ldx, int G, int MT,
                                                                  uint16_t* __restrict__ out) {
  const int idx = blockIdx.x * 256 + threadIdx.x;
  if (idx >= MT * G * kWave) return;
  const int lane = idx % kWave;
  const int g = (idx / kWave) % G;
  const int mt = idx / (kWave * G);
  const int m = mt * 16 + (lane & 15);
  const int kq = lane >> 4;
  uint32_t a[16];
  if (m < M) {
    const u32x4* src = reinterpret_cast<const u32x4*>(x + (size_t)m * ldx + g * 128 + kq * 32);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const u32x4 v = src[i];
      a[4 * i] = v[0];
      a[4 * i + 1] = v[1];
      a[4 * i + 2] = v[2];
      a[4 * i + 3] = v[3];
    }
  } else {
#pragma unroll
    for (int i = 0; i < 16; ++i) a[i] = 0u;
  }
  u32x4 f[4];
  pack_prepared(a, f);
  uint16_t* base = out + (((size_t)mt * G + g) * 4) * kWave * 8;
#pragma unroll
  for (int fi = 0; fi < 4; ++fi) *reinterpret_cast<u32x4*>(base + ((size_t)fi * kWave + lane) * 8) = f[fi];
}

void launch_prepare_activations(const uint16_t* x, int M, int ldx, int K, uint16_t* out, hipStream_t st) {
  const int G = K / 128, MT = (M + 15) / 16;
  const int threads = MT * G * kWave;
  hipLaunchKernelGGL(prepare_activations_kernel, dim3((threads + 255) / 256), dim3(256), 0, st, x, M, ldx, G,
                     MT, out);
}

// ------------------------------------------------------------- prepack
// Canonical int4 matrix -> kernel-native copy (see W4Ptr).  A pure
// rearrangement of the same bits; one wave per (tile, group).
__global__ __launch_bounds__(256) void prepack_w4_kernel(const uint8_t* __restrict__ q,
                                                         const uint16_t* __restrict__ s,
                                                         const uint8_t* __restrict__ z, int K, int N,
                                                         u32x4* __restrict__ qp, uint32_t* __restrict__ szp) {
  const int G = K >> 7;
  const long item = (long)blockIdx.x * 4 + (threadIdx.x >> 6);  // (tile, group)
  if (item >= (long)(N >> 4) * G) return;
  const int t = (int)(item / G), g = (int)(item % G);
  const int lane = lane_id();
  const int n = t * 16 + (lane & 15), kq = lane >> 4;
  qp[item * kWave + lane] = *reinterpret_cast<const u32x4*>(q + (size_t)n * (K >> 1) + (size_t)g * 64 + kq * 16);
  if (lane < 16) {
    const size_t si = (size_t)n * G + g;
    szp[item * 16 + lane] = (uint32_t)s[si] | ((uint32_t)z[si] << 16);
  }
}

void launch_prepack_w4(const uint8_t* q, const uint16_t* s, const uint8_t* z, int K, int N, void* packed,
                       hipStream_t st) {
  const long items = (long)(N / 16) * (K / 128);
  u32x4* qp = reinterpret_cast<u32x4*>(packed);
  uint32_t* szp = reinterpret_cast<uint32_t*>(reinterpret_cast<char*>(packed) + (size_t)K * N / 2);
  hipLaunchKernelGGL(prepack_w4_kernel, dim3((unsigned)((items + 3) / 4)), dim3(256), 0, st, q, s, z, K, N, qp,
                     szp);
}

// ----------------------------------------------------------------- launch

template <int MT, int NW, int EPI>
static void launch_t(const GemmLaunch& L, hipStream_t st) {
  GemmArgs a;
  auto unpack = [&](const void* p) {
    return W4Ptr{reinterpret_cast<const u32x4*>(p),
                 reinterpret_cast<const uint32_t*>(reinterpret_cast<const char*>(p) + (size_t)L.K * L.N / 2)};
  };
  a.w0 = unpack(L.w0);
  a.w1 = unpack(L.w1);
  a.K = L.K;
  a.N = L.N;
  a.G = L.K / 128;
  a.a = L.aprep;
  a.M = L.M;
  a.y = L.y;
  a.ldy = L.ldy;
  a.yp = L.yprep;
  a.res = L.res;
  a.ldr = L.ldr;
  a.nblocks = L.nblocks;
  a.nwg = L.nwg;
  a.units = (uint32_t)(L.nblocks * a.G);
  a.part = L.part;
  hipLaunchKernelGGL((w4a16_gemm_kernel<MT, NW, EPI>), dim3(L.nwg), dim3(256), 0, st, a);
  // ranges split no N-block when every workgroup gets whole N-blocks (the
  // split SwiGLU is only planned that way)
  if constexpr (EPI != EPI_SWIGLU_SPLIT) {
    if (L.nblocks % L.nwg != 0) {
      hipLaunchKernelGGL((w4a16_fixup_kernel<MT, NW, EPI>), dim3(L.nblocks * MT), dim3(256), 0, st, a);
    }
  }
}

// instantiated shapes: SwiGLU one gate + one up tile per wave, or (up to 32
// rows) one tile per wave with gate and up in different waves; plain one or
// two tiles per wave
template <int MT, int EPI>
static void launch_nw(const GemmLaunch& L, hipStream_t st) {
  if constexpr (EPI == EPI_SWIGLU) {
    if constexpr (MT <= 2) {
      if (L.nw == 1) {
        launch_t<MT, 1, EPI_SWIGLU_SPLIT>(L, st);
        return;
      }
    }
    launch_t<MT, 2, EPI>(L, st);
  } else if constexpr (MT <= 2) {
    if (L.nw == 2) launch_t<MT, 2, EPI>(L, st);
    else launch_t<MT, 1, EPI>(L, st);
  } else {
    if (L.nw == 2) launch_t<MT, 2, EPI>(L, st);
    else launch_t<MT, 1, EPI>(L, st);
  }
}

template <int EPI>
static void launch_mt(const GemmLaunch& L, hipStream_t st) {
  switch ((L.M + 15) / 16) {
    case 1: launch_nw<1, EPI>(L, st); break;
    case 2: launch_nw<2, EPI>(L, st); break;
    case 3: launch_nw<3, EPI>(L, st); break;
    default: launch_nw<4, EPI>(L, st); break;
  }
}

static GemmArgs kslice_args(const GemmLaunch& L) {
  GemmArgs a = {};
  auto unpack = [&](const void* p) {
    return W4Ptr{reinterpret_cast<const u32x4*>(p),
                 reinterpret_cast<const uint32_t*>(reinterpret_cast<const char*>(p) + (size_t)L.K * L.N / 2)};
  };
  a.w0 = unpack(L.w0);
  a.w1 = unpack(L.w1);
  a.K = L.K;
  a.N = L.N;
  a.G = L.K / 128;
  a.a = L.aprep;
  a.M = L.M;
  a.y = L.y;
  a.ldy = L.ldy;
  a.yp = L.yprep;
  a.res = L.res;
  a.ldr = L.ldr;
  a.x = L.xnorm;
  a.ldx = L.ldx;
  a.gamma = L.gamma;
  a.eps = L.eps;
  return a;
}

template <int W, int NT>
static void launch_kslice(const GemmLaunch& L, hipStream_t st) {
  hipLaunchKernelGGL((w4a16_kslice_kernel<W, NT>), dim3(L.N / 16), dim3(64 * W), 0, st, kslice_args(L));
}

template <int W, int NT, int NG>
static void launch_kslice_norm(const GemmLaunch& L, hipStream_t st) {
  hipLaunchKernelGGL((w4a16_kslice_norm_kernel<W, NT, NG>), dim3(L.N / 16), dim3(64 * W), 0, st, kslice_args(L));
}

bool norm_in_kslice(const GemmPlan& p, int K) {
  return p.ksw > 0 && (K / 128 + p.ksw - 1) / p.ksw <= kNormMaxGroupsPerWave;
}

void launch_w4a16_gemm(const GemmLaunch& L, hipStream_t st) {
  // K-split plans give the fused SwiGLU 4 waves, plain GEMMs 4 or 8
  if (L.ksw && L.xnorm) {
    const bool two = (L.K / 128 + L.ksw - 1) / L.ksw <= 2;  // groups per wave (norm_in_kslice: <= 4)
    if (L.swiglu) two ? launch_kslice_norm<4, 2, 2>(L, st) : launch_kslice_norm<4, 2, 4>(L, st);
    else if (L.ksw == 8) two ? launch_kslice_norm<8, 1, 2>(L, st) : launch_kslice_norm<8, 1, 4>(L, st);
    else two ? launch_kslice_norm<4, 1, 2>(L, st) : launch_kslice_norm<4, 1, 4>(L, st);
    return;
  }
  if (L.ksw) {
    if (L.swiglu) launch_kslice<4, 2>(L, st);
    else if (L.ksw == 8) launch_kslice<8, 1>(L, st);
    else launch_kslice<4, 1>(L, st);
    return;
  }
  if (L.swiglu) launch_mt<EPI_SWIGLU>(L, st);
  else launch_mt<EPI_PLAIN>(L, st);
}

GemmPlan plan_w4a16_gemm(int M, int K, int N, bool swiglu) {
  // nw = 16-column source tiles per wave (SwiGLU: half gate, half up); a
  // block (one workgroup's N-range) holds 4 waves' tiles
  GemmPlan p;
  const int tiles = N / 16;
  const int MT = (M + 15) / 16;
  const int G = K / 128;
  const size_t mbytes = (size_t)K * N / 2;
  if (MT == 1 && G >= 8 && tiles >= 128 && mbytes <= ((size_t)32 << 20) && (!swiglu || M <= 8)) {
    // up to 16 rows (a fused SwiGLU: up to 8) and at most 32 MB per matrix:
    // one workgroup per column tile, K split across its waves, no partials
    // or fix-up.  Every workgroup reads the activations of the rows it
    // computes (rows past M are not loaded), so the L2 reads are M / 4
    // (SwiGLU: M / 8) times the weight bytes.  Measured against the forms below:
    // 1B QKV 8.8 -> 4.2 us, O 8.4 -> 4.4 us, down 10.7 -> 7.0 us, SwiGLU
    // 9.5 -> 7.4 us; 8B O 10.1 -> 6.6 us, down 15.4 -> 14.5 us; TP4 shard
    // QKV 11.4 -> 8.9 us, O 10.0 -> 7.1 us, SwiGLU 20.5 -> 16.2 us, down
    // 15.4 -> 13.4 us.  The 8B SwiGLU at 16 rows (twice the activation
    // reads) is slower, 17.5 -> 21.4 us, and stays on the 2-column form.
    // A SwiGLU workgroup streams two tiles: 4 waves (8: 7.4 -> 8.5 us).
    p.ksw = (!swiglu && G >= 16) ? 8 : 4;
    p.nw = 1;
    p.nblocks = tiles;
    p.nwg = tiles;
    p.part_bytes = 0;
    p.prep_bytes = (size_t)MT * G * 4 * kWave * 16;
    return p;
  }
  if (swiglu && MT <= 2 && tiles % 2 == 0 && tiles / 4 < 256 && tiles / 2 >= 256) {
    // gate and up tiles in different waves, one workgroup per 2 columns:
    // where the 4-column blocks are too few to fill the chip on their own
    // (the 8B width: 224 blocks, 20.5 -> 18 us at 16 rows; the 1B width:
    // 128 blocks, 14.3 -> 9.2 us at 8 rows) this replaces stream-K and its
    // fix-up; at the 70B width (448 blocks) it is slower, 56 -> 72 us at 32
    // rows, as every workgroup reads the activations for half the columns
    p.nw = 1;
    p.nblocks = tiles / 2;
    p.nwg = p.nblocks;
    p.part_bytes = 0;
    p.prep_bytes = (size_t)MT * (K / 128) * 4 * kWave * 16;
    return p;
  }
  if (swiglu) {
    p.nw = 2;  // one gate and one up tile per wave
    p.nblocks = tiles / 4;
  } else {
    // two tiles per wave halve the LDS fragment reads per weight byte: up
    // to 32 rows where that still leaves at least 64 blocks and K is long
    // (the 70B projections; at the 8B widths, 48 and 32 blocks, one tile per
    // wave is 10-26 % faster, and at K = 2048 15 %), above 32 rows where K
    // is long enough to keep the split-K partials small
    p.nw = (((MT <= 2 && tiles / 8 >= 64 && K >= 8192) || K >= 16384) && tiles % 8 == 0) ? 2 : 1;
    p.nblocks = tiles / (4 * p.nw);
  }
  const long units = (long)p.nblocks * (K / 128);
  int cap = gemm_shape(MT, swiglu).nwg;
  // whole N-blocks per workgroup when they alone fill the chip (the SwiGLU
  // at the 70B width: 448 blocks; at 48 and 64 rows 11 % faster than
  // stream-K, whose gate and up partials cost a 16 us fix-up at 64 rows)
  if (swiglu && p.nblocks >= 256 && p.nblocks <= 2 * cap) cap = p.nblocks;
  // up to 32 rows, about 8 ranges per N-block: more split the blocks into
  // slivers whose partials the fix-up must sum (1B-shaped projections with
  // 32 blocks: 12.0 -> 10.6 us at 256 workgroups instead of 512)
  if (!swiglu && MT <= 2 && 8 * p.nblocks < cap) cap = 8 * p.nblocks;
  p.nwg = (int)(units < cap ? units : cap);
  const int col_w = swiglu ? p.nw / 2 : p.nw;
  const int src = swiglu ? 2 : 1;
  p.part_bytes = (size_t)p.nwg * 2 * 4 * MT * col_w * src * kWave * 16;
  p.prep_bytes = (size_t)MT * (K / 128) * 4 * kWave * 16;
  return p;
}

}  // namespace ss
