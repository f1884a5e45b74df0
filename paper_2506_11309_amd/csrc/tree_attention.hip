// Tree-masked grouped-query attention of the draft-tree tokens over the KV
// cache, with the rotary embedding fused in (SwiftSpec Sec. 3.1 target-side
// square mask; Sec. 3.3 masked attention; Sec. 4 positions from tree depth).
//
// Query rows of one kv head g: r = i * G + hh (node i, query head g*G + hh),
// R = T * G rows.  Workgroup = 4 waves = 64 query rows (one 16-row tile per
// wave).  Grid = Hkv x RB x (S + 1):
//   * splits 0..S-1 each take a contiguous chunk of the prefix keys [0, P)
//     (P is read on the device, so one launch shape serves every step);
//   * split S takes the T tree keys: it rotates the tree's keys, applies the
//     ancestor mask, and (row block 0 only) writes rotated keys and values
//     to cache rows [P, P+T).  Tree keys are consumed from registers/LDS, so
//     no workgroup reads a cache row another one is writing.
// Scores use S^T = K . Q^T on v_mfma_f32_16x16x32_f16: the result leaves
// each lane with four consecutive keys of one query row, which is exactly
// the A-operand layout the P.V product needs (keys are the reduction index),
// so probabilities never leave registers.  V is staged transposed in LDS so
// its B fragments are two 8-byte LDS reads.  Online softmax in fp32.
// The S + 1 partial results (unnormalised O, running max, running sum) of a
// row block are merged by the last workgroup to arrive (atomic ticket), in
// split order, so results are deterministic.  blockIdx % Hkv = g keeps one
// head's workgroups on one XCD when Hkv divides 8.
#include "ss_device.h"
#include "ss_internal.h"

namespace ss {

constexpr int kKeyTile = 64;

struct AttnArgs {
  const uint16_t* q;
  const uint16_t* k;
  const uint16_t* v;
  uint16_t* k_cache;
  uint16_t* v_cache;
  const int32_t* prefix_len;
  const int32_t* parent;
  const float* rope;
  uint16_t* out;
  uint16_t* out_prep;
  void* ws;
  float* part;
  int ldq, ldkv, ldo, S_max, T, Hq, Hkv, G, R, RB, nsplit;
  float scale_log2;  // softmax scale * log2(e)
};

template <int D>
struct AttnSmem {
  static constexpr int kKStride = D + 8;         // halves per K row (pad: 16 B)
  static constexpr int kVStride = kKeyTile + 4;  // halves per V^T row (pad: 8 B)
  uint16_t k[kKeyTile * kKStride];
  uint16_t vt[D * kVStride];
  uint64_t anc[64];
  int32_t depth[64];
  int32_t status;
  uint32_t ticket;
};

__device__ __forceinline__ float exp2_approx(float x) { return exp2f(x); }

template <int D>
__global__ __launch_bounds__(256) void tree_attention_kernel(AttnArgs a) {
  constexpr int KS = D / 32;  // k-steps of the QK^T product
  constexpr int DT = D / 16;  // d tiles of the PV product
  constexpr int HALF = D / 2;
  __shared__ AttnSmem<D> sm;

  const int lane = lane_id();
  const int wave = threadIdx.x >> 6;
  const int n16 = lane & 15;
  const int kq = lane >> 4;
  const int g = blockIdx.x % a.Hkv;
  const int rest = blockIdx.x / a.Hkv;
  const int sp = rest % (a.nsplit + 1);
  const int rb = rest / (a.nsplit + 1);
  const bool tree_split = sp == a.nsplit;

  // ---- per-step device data: prefix length and tree masks ----
  if (wave == 0) {
    uint64_t anc;
    int depth;
    const bool ok = tree_masks_wave(a.parent, a.T, anc, depth);
    if (lane < 64) {
      sm.anc[lane] = anc;
      sm.depth[lane] = depth;
    }
    if (lane == 0) {
      const int P = *a.prefix_len;
      int st = 0;
      if (!ok) st |= SWIFTSPEC_DEVERR_BAD_TREE;
      if (P < 0 || P > a.S_max - a.T) st |= SWIFTSPEC_DEVERR_BAD_PREFIX;
      sm.status = st;
      if (st && blockIdx.x == 0) report_error(a.ws, (uint32_t)st);
    }
  }
  __syncthreads();
  if (sm.status) return;
  const int P = *a.prefix_len;

  // ---- this wave's 16 query rows: rotated Q as B fragments ----
  const int row = rb * 64 + wave * 16 + n16;
  const bool row_ok = row < a.R;
  const int node = row_ok ? row / a.G : 0;
  const int qhead = g * a.G + (row_ok ? row % a.G : 0);
  half8 qf[KS];
  {
    float qv[KS][8];
    const uint16_t* qsrc = a.q + (size_t)node * a.ldq + qhead * D;
#pragma unroll
    for (int j = 0; j < KS; ++j) {
      u32x4 raw = row_ok ? *reinterpret_cast<const u32x4*>(qsrc + 32 * j + 8 * kq) : u32x4{0, 0, 0, 0};
      half8 h = bitcast<half8>(raw);
#pragma unroll
      for (int e = 0; e < 8; ++e) qv[j][e] = (float)h[e];
    }
    const float* cs = a.rope + (size_t)(P + sm.depth[node]) * D;  // [D/2][2]
#pragma unroll
    for (int j = 0; j < KS / 2; ++j) {
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const int d = 32 * j + 8 * kq + e;  // < D/2; partner d + D/2 sits in k-step j + KS/2
        const float c = cs[2 * d], s = cs[2 * d + 1];
        const float x1 = qv[j][e], x2 = qv[j + KS / 2][e];
        qv[j][e] = x1 * c - x2 * s;
        qv[j + KS / 2][e] = x2 * c + x1 * s;
      }
    }
#pragma unroll
    for (int j = 0; j < KS; ++j) {
      half8 h;
#pragma unroll
      for (int e = 0; e < 8; ++e) h[e] = (_Float16)qv[j][e];
      qf[j] = h;
    }
  }

  // ---- key range ----
  int k_lo = 0, k_hi = 0;
  if (!tree_split) {
    const int per = (P + a.nsplit - 1) / a.nsplit;
    const int chunk = ((per + kKeyTile - 1) / kKeyTile) * kKeyTile;
    k_lo = min(P, sp * chunk);
    k_hi = min(P, k_lo + chunk);
  }

  float m_run = -INFINITY, l_run = 0.f;  // for row n16 of this wave (replicated over kq)
  f32x4 o[DT];
#pragma unroll
  for (int dt = 0; dt < DT; ++dt) o[dt] = f32x4{0.f, 0.f, 0.f, 0.f};

  const uint16_t* kc = a.k_cache + (size_t)g * a.S_max * D;
  const uint16_t* vc = a.v_cache + (size_t)g * a.S_max * D;
  constexpr int kVecPerRow = D / 8;                       // 16-byte vectors per key row
  constexpr int kVecPerThread = kKeyTile * kVecPerRow / 256;  // per tile, for K and for V

  const int ntiles = tree_split ? 1 : (k_hi - k_lo + kKeyTile - 1) / kKeyTile;
  for (int tile = 0; tile < ntiles; ++tile) {
    const int key0 = k_lo + tile * kKeyTile;
    // ---- stage K (row-major) and V (transposed) into LDS ----
    if (!tree_split) {
#pragma unroll
      for (int it = 0; it < kVecPerThread; ++it) {
        const int idx = threadIdx.x + it * 256;
        const int kr = idx / kVecPerRow, c8 = (idx % kVecPerRow) * 8;
        const int key = key0 + kr;
        u32x4 kv = {0, 0, 0, 0}, vv = {0, 0, 0, 0};
        if (key < k_hi) {
          kv = *reinterpret_cast<const u32x4*>(kc + (size_t)key * D + c8);
          vv = *reinterpret_cast<const u32x4*>(vc + (size_t)key * D + c8);
        }
        *reinterpret_cast<u32x4*>(&sm.k[kr * AttnSmem<D>::kKStride + c8]) = kv;
        const uint16_t* vh = reinterpret_cast<const uint16_t*>(&vv);
#pragma unroll
        for (int e = 0; e < 8; ++e) sm.vt[(c8 + e) * AttnSmem<D>::kVStride + kr] = vh[e];
      }
    } else {
      // tree keys: rotate k at position P + depth, round to fp16; copy v.
      // Thread handles (key kr, 8 rotation pairs starting at c8 < D/2).
      constexpr int kPairVecs = HALF / 8;
      for (int idx = threadIdx.x; idx < kKeyTile * kPairVecs; idx += 256) {
        const int kr = idx / kPairVecs, c8 = (idx % kPairVecs) * 8;
        u32x4 k1 = {0, 0, 0, 0}, k2 = {0, 0, 0, 0}, v1 = {0, 0, 0, 0}, v2 = {0, 0, 0, 0};
        if (kr < a.T) {
          const uint16_t* ks = a.k + (size_t)kr * a.ldkv + g * D;
          const uint16_t* vs = a.v + (size_t)kr * a.ldkv + g * D;
          u32x4 r1 = *reinterpret_cast<const u32x4*>(ks + c8);
          u32x4 r2 = *reinterpret_cast<const u32x4*>(ks + c8 + HALF);
          v1 = *reinterpret_cast<const u32x4*>(vs + c8);
          v2 = *reinterpret_cast<const u32x4*>(vs + c8 + HALF);
          const float* cs = a.rope + (size_t)(P + sm.depth[kr]) * D;
          half8 h1 = bitcast<half8>(r1), h2 = bitcast<half8>(r2), o1, o2;
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            const float c = cs[2 * (c8 + e)], s = cs[2 * (c8 + e) + 1];
            const float x1 = (float)h1[e], x2 = (float)h2[e];
            o1[e] = (_Float16)(x1 * c - x2 * s);
            o2[e] = (_Float16)(x2 * c + x1 * s);
          }
          k1 = bitcast<u32x4>(o1);
          k2 = bitcast<u32x4>(o2);
          if (rb == 0) {
            uint16_t* kd = a.k_cache + ((size_t)g * a.S_max + P + kr) * D;
            uint16_t* vd = a.v_cache + ((size_t)g * a.S_max + P + kr) * D;
            *reinterpret_cast<u32x4*>(kd + c8) = k1;
            *reinterpret_cast<u32x4*>(kd + c8 + HALF) = k2;
            *reinterpret_cast<u32x4*>(vd + c8) = v1;
            *reinterpret_cast<u32x4*>(vd + c8 + HALF) = v2;
          }
        }
        *reinterpret_cast<u32x4*>(&sm.k[kr * AttnSmem<D>::kKStride + c8]) = k1;
        *reinterpret_cast<u32x4*>(&sm.k[kr * AttnSmem<D>::kKStride + c8 + HALF]) = k2;
        const uint16_t* vh1 = reinterpret_cast<const uint16_t*>(&v1);
        const uint16_t* vh2 = reinterpret_cast<const uint16_t*>(&v2);
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          sm.vt[(c8 + e) * AttnSmem<D>::kVStride + kr] = vh1[e];
          sm.vt[(c8 + HALF + e) * AttnSmem<D>::kVStride + kr] = vh2[e];
        }
      }
    }
    __syncthreads();

    // ---- S^T = K . Q^T for the tile's 4 key subtiles ----
    f32x4 s[4];
#pragma unroll
    for (int st = 0; st < 4; ++st) {
      f32x4 c = {0.f, 0.f, 0.f, 0.f};
      const uint16_t* krow = &sm.k[(st * 16 + n16) * AttnSmem<D>::kKStride + 8 * kq];
#pragma unroll
      for (int j = 0; j < KS; ++j) {
        half8 kf = *reinterpret_cast<const half8*>(krow + 32 * j);
        c = __builtin_amdgcn_mfma_f32_16x16x32_f16(kf, qf[j], c, 0, 0, 0);
      }
      s[st] = c;  // lane: keys st*16 + 4*kq + r (r < 4), query row n16
    }
    // ---- mask, online softmax (base 2) ----
    const int key_end = tree_split ? a.T : (k_hi - key0);
    const uint64_t anc = sm.anc[node];
    float tmax = -INFINITY;
#pragma unroll
    for (int st = 0; st < 4; ++st)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int kr = st * 16 + 4 * kq + r;
        bool ok = kr < key_end;
        if (tree_split) ok = ok && ((anc >> kr) & 1ull);
        const float v = ok ? s[st][r] * a.scale_log2 : -INFINITY;
        s[st][r] = v;
        tmax = fmaxf(tmax, v);
      }
    tmax = fmaxf(tmax, __shfl_xor(tmax, 16, kWave));
    tmax = fmaxf(tmax, __shfl_xor(tmax, 32, kWave));
    const float m_new = fmaxf(m_run, tmax);
    const float alpha = (m_new == -INFINITY) ? 1.f : exp2_approx(m_run - m_new);
    float psum = 0.f;
    half8 pf[2];
#pragma unroll
    for (int st = 0; st < 4; ++st)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const float p = (s[st][r] == -INFINITY) ? 0.f : exp2_approx(s[st][r] - m_new);
        psum += p;
        pf[st >> 1][(st & 1) * 4 + r] = (_Float16)p;
      }
    psum += __shfl_xor(psum, 16, kWave);
    psum += __shfl_xor(psum, 32, kWave);
    l_run = l_run * alpha + psum;
    m_run = m_new;
    // rescale O: lane holds rows 4*kq + r; fetch those rows' alpha
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const float ar = __shfl(alpha, 4 * kq + r, kWave);
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) o[dt][r] *= ar;
    }
    // ---- O += P . V; keys of pair pp: subtiles 2pp and 2pp+1 ----
#pragma unroll
    for (int pp = 0; pp < 2; ++pp) {
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) {
        const uint16_t* vrow = &sm.vt[(dt * 16 + n16) * AttnSmem<D>::kVStride];
        u32x2 lo = *reinterpret_cast<const u32x2*>(vrow + (2 * pp) * 16 + 4 * kq);
        u32x2 hi = *reinterpret_cast<const u32x2*>(vrow + (2 * pp + 1) * 16 + 4 * kq);
        half8 vf = bitcast<half8>(u32x4{lo[0], lo[1], hi[0], hi[1]});
        o[dt] = __builtin_amdgcn_mfma_f32_16x16x32_f16(pf[pp], vf, o[dt], 0, 0, 0);
      }
    }
    __syncthreads();
  }

  // ---- publish this split's partial ----
  const int nparts = a.nsplit + 1;
  const size_t grp = (size_t)g * a.RB + rb;
  const size_t part_stride = (size_t)4 * DT * kWave * 4 + 4 * 16 * 2;  // floats per workgroup partial
  float* mine = a.part + (grp * nparts + sp) * part_stride;
#pragma unroll
  for (int dt = 0; dt < DT; ++dt) store_agent_f32x4(mine + ((size_t)(wave * DT + dt) * kWave + lane) * 4, o[dt]);
  float* ml = mine + (size_t)4 * DT * kWave * 4;
  if (kq == 0) {
    store_agent_u64(ml + (wave * 16 + n16) * 2, bitcast<uint64_t>(f32x2{m_run, l_run}));
  }
  wait_all_memory();
  __syncthreads();
  uint32_t* counter = ws_counters(a.ws) + grp;
  if (threadIdx.x == 0) sm.ticket = take_ticket(counter);
  __syncthreads();
  if (sm.ticket != (uint32_t)(nparts - 1)) return;

  // ---- last arrival: merge the partials in split order ----
  float mrow[4];
#pragma unroll
  for (int r = 0; r < 4; ++r) mrow[r] = -INFINITY;
  const float* base = a.part + grp * nparts * part_stride;
  for (int s2 = 0; s2 < nparts; ++s2) {
    const float* mlp = base + s2 * part_stride + (size_t)4 * DT * kWave * 4;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      f32x2 v2 = bitcast<f32x2>(load_agent_u64(mlp + (wave * 16 + 4 * kq + r) * 2));
      mrow[r] = fmaxf(mrow[r], v2[0]);
    }
  }
  float lsum[4] = {0.f, 0.f, 0.f, 0.f};
  f32x4 acc[DT];
#pragma unroll
  for (int dt = 0; dt < DT; ++dt) acc[dt] = f32x4{0.f, 0.f, 0.f, 0.f};
  for (int s2 = 0; s2 < nparts; ++s2) {
    const float* src = base + s2 * part_stride;
    const float* mlp = src + (size_t)4 * DT * kWave * 4;
    float w[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      f32x2 v2 = bitcast<f32x2>(load_agent_u64(mlp + (wave * 16 + 4 * kq + r) * 2));
      w[r] = (v2[0] == -INFINITY) ? 0.f : exp2_approx(v2[0] - mrow[r]);
      lsum[r] += w[r] * v2[1];
    }
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) {
      f32x4 ov = load_agent_f32x4(src + ((size_t)(wave * DT + dt) * kWave + lane) * 4);
#pragma unroll
      for (int r = 0; r < 4; ++r) acc[dt][r] += w[r] * ov[r];
    }
  }
  if (threadIdx.x == 0) reset_counter(counter);
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int orow = rb * 64 + wave * 16 + 4 * kq + r;
    if (orow < a.R) {
      const int i = orow / a.G, qh = g * a.G + orow % a.G;
      const float inv = 1.0f / lsum[r];
      uint16_t* dst = a.out + (size_t)i * a.ldo + qh * D;
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) {
        const uint16_t h = f2h(acc[dt][r] * inv);
        dst[dt * 16 + n16] = h;
        if (a.out_prep) store_prepared(a.out_prep, i, qh * D + dt * 16 + n16, (a.Hq * D) >> 7, h);
      }
    }
  }
}

AttnPlan plan_tree_attention(int T, int Hq, int Hkv, int D, int S_max) {
  AttnPlan p;
  const int G = Hq / Hkv;
  const int R = T * G;
  const int RB = (R + 63) / 64;
  const int groups = Hkv * RB;
  // about 256 workgroups in flight, at least one key tile per prefix split
  int ns = 256 / groups - 1;
  const int max_tiles = (S_max - T + kKeyTile - 1) / kKeyTile;
  if (ns > max_tiles) ns = max_tiles;
  if (ns < 1) ns = 1;
  p.nsplit = ns;
  p.chunk = 0;
  const size_t part_stride = (size_t)4 * (D / 16) * kWave * 4 + 4 * 16 * 2;
  p.part_bytes = (size_t)groups * (ns + 1) * part_stride * sizeof(float);
  return p;
}

void launch_tree_attention(const AttnLaunch& L, hipStream_t st) {
  AttnArgs a;
  a.q = L.q;
  a.k = L.k;
  a.v = L.v;
  a.k_cache = L.k_cache;
  a.v_cache = L.v_cache;
  a.prefix_len = L.prefix_len;
  a.parent = L.parent;
  a.rope = L.rope;
  a.out = L.out;
  a.out_prep = L.out_prep;
  a.ws = L.ws;
  a.part = L.part;
  a.ldq = L.ldq;
  a.ldkv = L.ldkv;
  a.ldo = L.ldo;
  a.S_max = L.S_max;
  a.T = L.T;
  a.Hq = L.Hq;
  a.Hkv = L.Hkv;
  a.G = L.Hq / L.Hkv;
  a.R = L.T * a.G;
  a.RB = (a.R + 63) / 64;
  a.nsplit = L.nsplit;
  a.scale_log2 = L.scale * 1.4426950408889634f;
  const dim3 grid(L.Hkv * a.RB * (L.nsplit + 1));
  if (L.D == 64) hipLaunchKernelGGL(tree_attention_kernel<64>, grid, dim3(256), 0, st, a);
  else hipLaunchKernelGGL(tree_attention_kernel<128>, grid, dim3(256), 0, st, a);
}

}  // namespace ss
