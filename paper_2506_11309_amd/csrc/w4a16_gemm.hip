// W4A16 GEMMs at small M (the tree size) for gfx950.
//
// y[m][n] = sum_k x[m][k] * W'[n][k], W'[n][k] = (q[n][k] - z[n][g]) * s[n][g],
// g = k / 128: the int4 AWQ-style projections of a decoder layer
// (SwiftSpec Sec. 3.3 and Sec. 5.1).  Variants: plain (+ residual), fused
// SwiGLU (gate and up tiles share the activation fragments, Sec. 3.3), and
// a dense fp16-weight variant for the LM head.
//
// Mapping onto the matrix cores (v_mfma_f32_16x16x32_f16, wave64):
//   * A operand = activations, 16 token rows per M-tile (rows >= M are zero);
//     B operand = weights, 16 output columns per N-tile.
//   * One 16-byte load per lane fetches 32 consecutive k of one weight row:
//     lane (n = lane % 16, kq = lane / 16) reads k in [32 kq, 32 kq + 32) of
//     a 128-wide quantisation group, so one wave-wide load covers exactly a
//     16 x 128 (column x group) block and one (scale, zero) pair per lane.
//   * Dequantisation in registers without shifts of the high nibbles:
//       (w & 0x000F000F) | 0x64006400  = fp16 pair (1024 + q_lo, ...)
//       (w & 0x00F000F0) | 0x64006400  = fp16 pair (1024 + 16 q_hi, ...)
//     followed by one packed fp16 subtraction of (1024 + z) resp.
//     (1024 + 16 z), both exact.  Low-nibble k slots are matched with
//     activations pre-multiplied by 16 (exact in fp16), so every product is
//     16 x (q - z); the group sum is scaled by s / 16 in fp32.  The k-slot
//     order inside an MFMA is a permutation of the group's k, applied
//     identically to both operands.
//   * Each workgroup (4 waves) owns NW N-tiles for one K-split; its waves
//     take interleaved quantisation groups (so together they stream 256
//     contiguous bytes of every weight row), and reduce through LDS.
//   * K-splits of one N-block are combined by the last-arriving workgroup
//     (atomic ticket) in split order, so the result is deterministic.
//     Partials use agent-scope coherent 8-byte stores/loads; blockIdx is
//     laid out so all splits of an N-block share blockIdx % 8 (one XCD when
//     workgroups are dispatched round-robin over the 8 XCDs).
#include "ss_device.h"
#include "ss_internal.h"

namespace ss {

struct W4Ptr {
  const uint8_t* q;
  const uint16_t* s;
  const uint8_t* z;
};

enum { EPI_PLAIN = 0, EPI_SWIGLU = 1 };

__device__ __forceinline__ uint32_t pk_lo(uint32_t u, uint32_t v) { return (u & 0xFFFFu) | (v << 16); }
__device__ __forceinline__ uint32_t pk_hi(uint32_t u, uint32_t v) { return (u >> 16) | (v & 0xFFFF0000u); }

// Activation fragments of one 16-row M-tile for one group, from 32
// consecutive fp16 of the lane's row (a[0..15] = pairs (x_2j, x_2j+1)).
// frag[0] / frag[1]: low-nibble slots of k 0..15 / 16..31, times 16;
// frag[2] / frag[3]: high-nibble slots.
__device__ __forceinline__ void act_fragments(const u32x4 raw[4], half8 frag[4]) {
  uint32_t a[16];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    a[4 * i + 0] = raw[i][0];
    a[4 * i + 1] = raw[i][1];
    a[4 * i + 2] = raw[i][2];
    a[4 * i + 3] = raw[i][3];
  }
  const _Float16 sixteen = (_Float16)16.0f;
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const uint32_t* b = a + 8 * h;
    u32x4 lo = {pk_lo(b[0], b[2]), pk_lo(b[1], b[3]), pk_lo(b[4], b[6]), pk_lo(b[5], b[7])};
    u32x4 hi = {pk_hi(b[0], b[2]), pk_hi(b[1], b[3]), pk_hi(b[4], b[6]), pk_hi(b[5], b[7])};
    frag[h] = bitcast<half8>(lo) * sixteen;
    frag[2 + h] = bitcast<half8>(hi);
  }
}

// Weight fragments (same slot order) from the lane's 16 packed bytes.
__device__ __forceinline__ void weight_fragments(const u32x4 w, uint32_t zero, half8 frag[4]) {
  const uint32_t magic = 0x64006400u;
  const _Float16 c_lo = (_Float16)(-(1024.0f + (float)zero));
  const _Float16 c_hi = (_Float16)(-(1024.0f + 16.0f * (float)zero));
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const uint32_t d0 = w[2 * h], d1 = w[2 * h + 1];
    const uint32_t s0 = d0 >> 8, s1 = d1 >> 8;
    u32x4 lo = {(d0 & 0x000F000Fu) | magic, (s0 & 0x000F000Fu) | magic, (d1 & 0x000F000Fu) | magic,
                (s1 & 0x000F000Fu) | magic};
    u32x4 hi = {(d0 & 0x00F000F0u) | magic, (s0 & 0x00F000F0u) | magic, (d1 & 0x00F000F0u) | magic,
                (s1 & 0x00F000F0u) | magic};
    frag[h] = bitcast<half8>(lo) + c_lo;
    frag[2 + h] = bitcast<half8>(hi) + c_hi;
  }
}

template <int MT, int NW, int EPI>
struct GemmTile {
  static constexpr int kTiles = MT * NW;
};

template <int MT, int NW, int EPI>
__global__ __launch_bounds__(256) void w4a16_gemm_kernel(
    W4Ptr w0, W4Ptr w1, int K, int N, const uint16_t* __restrict__ x, int M, int ldx,
    uint16_t* __restrict__ y, int ldy, const uint16_t* __restrict__ res, int ldr, int nblocks,
    int nsplit, float* __restrict__ part, uint32_t* __restrict__ counters) {
  constexpr int kTiles = MT * NW;
  constexpr int kColTiles = (EPI == EPI_SWIGLU) ? NW / 2 : NW;  // output column tiles per block
  constexpr int kSrc = (EPI == EPI_SWIGLU) ? 2 : 1;               // source tiles per output unit
  constexpr int kChunkOut = 8 / kSrc;                              // output units per LDS chunk
  static_assert(kTiles >= 1, "empty tile");
  __shared__ f32x4 red[4][8][kWave];
  __shared__ uint32_t s_ticket;

  const int lane = lane_id();
  const int wave = threadIdx.x >> 6;
  const int nb = blockIdx.x % nblocks;
  const int ks = blockIdx.x / nblocks;
  const int G = K >> 7;
  const int g_begin = (int)(((long)ks * G) / nsplit);
  const int g_end = (int)(((long)(ks + 1) * G) / nsplit);
  const int ncol = lane & 15;
  const int kq = lane >> 4;
  const int col0 = nb * kColTiles * 16;

  // per-tile weight row pointers (row = output column)
  const uint8_t* qrow[NW];
  const uint16_t* srow[NW];
  const uint8_t* zrow[NW];
#pragma unroll
  for (int nt = 0; nt < NW; ++nt) {
    const W4Ptr& w = (EPI == EPI_SWIGLU && nt >= kColTiles) ? w1 : w0;
    const int col = col0 + (nt % kColTiles) * 16 + ncol;
    qrow[nt] = w.q + (size_t)col * (K >> 1) + kq * 16;
    srow[nt] = w.s + (size_t)col * G;
    zrow[nt] = w.z + (size_t)col * G;
  }
  const uint16_t* xrow[MT];
  bool xvalid[MT];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) {
    const int m = mt * 16 + ncol;
    xvalid[mt] = m < M;
    xrow[mt] = x + (size_t)(xvalid[mt] ? m : 0) * ldx + kq * 32;
  }

  f32x4 acc[MT][NW];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int nt = 0; nt < NW; ++nt) acc[mt][nt] = f32x4{0.f, 0.f, 0.f, 0.f};

  u32x4 a_cur[MT][4], b_cur[NW];
  uint16_t s_cur[NW];
  uint8_t z_cur[NW];
  auto load_group = [&](int g, u32x4 (&a_raw)[MT][4], u32x4 (&b_raw)[NW], uint16_t (&s_raw)[NW],
                        uint8_t (&z_raw)[NW]) {
#pragma unroll
    for (int nt = 0; nt < NW; ++nt) {
      b_raw[nt] = *reinterpret_cast<const u32x4*>(qrow[nt] + (size_t)g * 64);
      s_raw[nt] = srow[nt][g];
      z_raw[nt] = zrow[nt][g];
    }
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
      const u32x4* src = reinterpret_cast<const u32x4*>(xrow[mt] + (size_t)g * 128);
#pragma unroll
      for (int i = 0; i < 4; ++i) a_raw[mt][i] = xvalid[mt] ? src[i] : u32x4{0u, 0u, 0u, 0u};
    }
  };

  int g = g_begin + wave;
  if (g < g_end) load_group(g, a_cur, b_cur, s_cur, z_cur);
  for (; g < g_end; g += 4) {
    u32x4 a_nxt[MT][4], b_nxt[NW];
    uint16_t s_nxt[NW];
    uint8_t z_nxt[NW];
    const bool more = g + 4 < g_end;
    if (more) load_group(g + 4, a_nxt, b_nxt, s_nxt, z_nxt);

    half8 afrag[MT][4];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) act_fragments(a_cur[mt], afrag[mt]);
#pragma unroll
    for (int nt = 0; nt < NW; ++nt) {
      half8 bfrag[4];
      weight_fragments(b_cur[nt], z_cur[nt], bfrag);
      const float sc = h2f(s_cur[nt]) * 0.0625f;
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) {
        f32x4 c = {0.f, 0.f, 0.f, 0.f};
        c = __builtin_amdgcn_mfma_f32_16x16x32_f16(afrag[mt][0], bfrag[0], c, 0, 0, 0);
        c = __builtin_amdgcn_mfma_f32_16x16x32_f16(afrag[mt][1], bfrag[1], c, 0, 0, 0);
        c = __builtin_amdgcn_mfma_f32_16x16x32_f16(afrag[mt][2], bfrag[2], c, 0, 0, 0);
        c = __builtin_amdgcn_mfma_f32_16x16x32_f16(afrag[mt][3], bfrag[3], c, 0, 0, 0);
#pragma unroll
        for (int r = 0; r < 4; ++r) acc[mt][nt][r] = __builtin_fmaf(c[r], sc, acc[mt][nt][r]);
      }
    }
    if (more) {
#pragma unroll
      for (int nt = 0; nt < NW; ++nt) {
        b_cur[nt] = b_nxt[nt];
        s_cur[nt] = s_nxt[nt];
        z_cur[nt] = z_nxt[nt];
      }
#pragma unroll
      for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int i = 0; i < 4; ++i) a_cur[mt][i] = a_nxt[mt][i];
    }
  }

  // ---- reduce the 4 waves' K-slices through LDS (fixed order) ----
  // Output unit u (a column tile, or a (gate, up) tile pair for SwiGLU):
  // mt = u / kColTiles, ct = u % kColTiles; wave w finishes units u = w + 4 j.
  // Units go through LDS in chunks of at most 8 source tiles (32 KB).
  constexpr int kOut = MT * kColTiles;
  constexpr int kJ = (kOut + 3) / 4;
  f32x4 sum_a[kJ], sum_b[kJ];
#pragma unroll
  for (int u0 = 0; u0 < kOut; u0 += kChunkOut) {
#pragma unroll
    for (int du = 0; du < kChunkOut; ++du) {
      const int u = u0 + du;
      if (u < kOut) {
        const int mt = u / kColTiles, ct = u % kColTiles;
        red[wave][du * kSrc][lane] = acc[mt][ct];
        if (EPI == EPI_SWIGLU) red[wave][du * kSrc + 1][lane] = acc[mt][ct + kColTiles];
      }
    }
    __syncthreads();
#pragma unroll
    for (int j = 0; j < kChunkOut / 4; ++j) {
      const int du = wave + 4 * j;
      const int J = u0 / 4 + j;
      if (J < kJ && u0 + du < kOut) {
        const int ta = du * kSrc;
        sum_a[J] = red[0][ta][lane] + red[1][ta][lane] + red[2][ta][lane] + red[3][ta][lane];
        if (EPI == EPI_SWIGLU)
          sum_b[J] = red[0][ta + 1][lane] + red[1][ta + 1][lane] + red[2][ta + 1][lane] + red[3][ta + 1][lane];
      }
    }
    __syncthreads();
  }

  if (nsplit > 1) {
    // publish this split's partial, then the last arriving split combines
    constexpr int kParts = kSrc;
    float* mine = part + ((size_t)(nb * nsplit + ks) * kOut * kParts) * kWave * 4;
#pragma unroll
    for (int j = 0; j < kJ; ++j) {
      const int t = wave + 4 * j;
      if (t < kOut) {
        store_agent_f32x4(mine + ((size_t)(t * kParts) * kWave + lane) * 4, sum_a[j]);
        if (EPI == EPI_SWIGLU) store_agent_f32x4(mine + ((size_t)(t * kParts + 1) * kWave + lane) * 4, sum_b[j]);
      }
    }
    wait_all_memory();
    __syncthreads();
    if (threadIdx.x == 0) s_ticket = take_ticket(&counters[nb]);
    __syncthreads();
    if (s_ticket != (uint32_t)(nsplit - 1)) return;
#pragma unroll
    for (int j = 0; j < kJ; ++j) {
      const int t = wave + 4 * j;
      if (t < kOut) {
        f32x4 sa = {0.f, 0.f, 0.f, 0.f}, sb = {0.f, 0.f, 0.f, 0.f};
        for (int s = 0; s < nsplit; ++s) {
          const float* src = part + ((size_t)(nb * nsplit + s) * kOut * kParts) * kWave * 4;
          sa += load_agent_f32x4(src + ((size_t)(t * kParts) * kWave + lane) * 4);
          if (EPI == EPI_SWIGLU) sb += load_agent_f32x4(src + ((size_t)(t * kParts + 1) * kWave + lane) * 4);
        }
        sum_a[j] = sa;
        sum_b[j] = sb;
      }
    }
    if (threadIdx.x == 0) reset_counter(&counters[nb]);
  }

  // ---- epilogue: lane holds rows 4 * (lane / 16) + r of column lane % 16 ----
#pragma unroll
  for (int j = 0; j < kJ; ++j) {
    const int t = wave + 4 * j;
    if (t < kOut) {
      const int mt = t / kColTiles, ct = t % kColTiles;
      const int n = col0 + ct * 16 + ncol;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int m = mt * 16 + kq * 4 + r;
        if (m < M) {
          float v;
          if (EPI == EPI_SWIGLU) {
            const float gte = sum_a[j][r], up = sum_b[j][r];
            v = gte / (1.0f + __expf(-gte)) * up;
          } else {
            v = sum_a[j][r];
            if (res) v += h2f(res[(size_t)m * ldr + n]);
          }
          y[(size_t)m * ldy + n] = f2h(v);
        }
      }
    }
  }
}

// ----------------------------------------------------------------- launch

template <int MT, int NW, int EPI>
static void launch_t(const GemmLaunch& L, hipStream_t st) {
  W4Ptr a{L.w0.q, L.w0.s, L.w0.z}, b{L.w1.q, L.w1.s, L.w1.z};
  hipLaunchKernelGGL((w4a16_gemm_kernel<MT, NW, EPI>), dim3(L.nblocks * L.nsplit), dim3(256), 0, st,
                     a, b, L.K, L.N, L.x, L.M, L.ldx, L.y, L.ldy, L.res, L.ldr, L.nblocks, L.nsplit,
                     L.part, L.counters);
}

template <int MT, int EPI>
static void launch_nw(const GemmLaunch& L, hipStream_t st) {
  switch (L.nw) {
    case 4: launch_t<MT, 4, EPI>(L, st); break;
    case 2: launch_t<MT, 2, EPI>(L, st); break;
    default:
      if (EPI == EPI_PLAIN) launch_t<MT, 1, EPI_PLAIN>(L, st);
      break;
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

void launch_w4a16_gemm(const GemmLaunch& L, hipStream_t st) {
  if (L.swiglu) launch_mt<EPI_SWIGLU>(L, st);
  else launch_mt<EPI_PLAIN>(L, st);
}

}  // namespace ss

namespace ss {

GemmPlan plan_w4a16_gemm(int M, int K, int N, bool swiglu) {
  GemmPlan p;
  const int tiles = N / 16;
  const int MT = (M + 15) / 16;
  if (swiglu) {
    p.nw = (tiles % 2 == 0) ? 4 : 2;
    p.nblocks = tiles / (p.nw / 2);
  } else {
    p.nw = (tiles % 4 == 0) ? 4 : (tiles % 2 == 0 ? 2 : 1);
    p.nblocks = tiles / p.nw;
  }
  // about two workgroups per CU; every wave keeps at least one group per split
  const int G = K / 128;
  const int target = 512;
  int ns = (target + p.nblocks - 1) / p.nblocks;
  int max_split = G / 4;
  if (max_split < 1) max_split = 1;
  if (ns > max_split) ns = max_split;
  if (ns > 32) ns = 32;
  if (ns < 1) ns = 1;
  p.nsplit = ns;
  const int col_tiles = swiglu ? p.nw / 2 : p.nw;
  const int src = swiglu ? 2 : 1;
  p.part_bytes = ns > 1 ? (size_t)p.nblocks * ns * MT * col_tiles * src * kWave * 16 : 0;
  return p;
}

}  // namespace ss
