// Tree-masked grouped-query attention of the draft-tree tokens over the KV
// cache, with the rotary embedding fused in (SwiftSpec Sec. 3.1 target-side
// square mask; Sec. 3.3 masked attention; Sec. 4 positions from tree depth).
//
// Query rows of one kv head g: r = i * G + hh (node i, query head g*G + hh),
// R = T * G rows.  Workgroup = W waves = 16 W query rows (one 16-row tile
// per wave), W = 8 for R >= 128, else 4.  Grid = Hkv x RB x (S + 1):
//   * splits 0..S-1 each take a contiguous chunk of the prefix keys [0, P)
//     (P is read on the device, so one launch shape serves every step);
//   * split S takes the T tree keys: it rotates the tree's keys, applies the
//     ancestor mask, and (row block 0 only) writes rotated keys and values
//     to cache rows [P, P+T).  Tree keys are consumed from registers/LDS, so
//     no workgroup reads a cache row another one is writing.
// Prefix keys stream in 64-key tiles: each thread loads its share of a
// tile's K and V rows into a 5-deep register ring (tiles t+1..t+4 in
// flight while tile t is computed), writes them row-major to a 3-slot LDS
// ring, and a fence-free barrier per tile hands the tile to all waves.
// Scores use S^T = K . Q^T on v_mfma_f32_16x16x32_f16: the result leaves
// each lane with four consecutive keys of one query row, which is exactly
// the A-operand layout the P.V product needs (keys are the reduction index),
// so probabilities never leave registers.  The V B-operand (key-major per d
// column) comes from the row-major tile through ds_read_b64_tr_b16: in each
// 16-lane group, lane j receives element j % 4 of the 8-byte rows addressed
// by lanes j / 4 + 4e, e = 0..3.  Online softmax in fp32, base 2.
// Each split publishes its rows' output normalised by their own softmax
// sum (fp16) and their log-sum-exp (fp32); a second kernel on the same
// stream merges the S + 1 partials of a row block in split order, so
// results are deterministic.  blockIdx % Hkv = g keeps one head's
// workgroups on one XCD when Hkv divides 8.
#include <type_traits>

#include "ss_device.h"
#include "ss_internal.h"

namespace ss {

constexpr int kKeyTile = 64;
constexpr int kAttnRing = 5;  // register ring of K/V tiles
constexpr int kAttnLds = 3;   // LDS ring of K/V tiles

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
  // draft model (non-square mask): N tree-cache rows [P, P+N) below the
  // prefix (a forest, cache_parent), the T new tokens are leaves below
  // leaf_parent[i] and see only themselves among the new rows; target
  // model: N = 0, leaf_parent = NULL, the T new tokens form the tree
  int N;
  const int32_t* cache_parent;
  const int32_t* leaf_parent;
};

typedef short v4i16 __attribute__((ext_vector_type(4)));

// Reduction over the four lanes l, l ^ 16, l ^ 32, l ^ 48 (the four key
// quarters of one query row in the score layout), in registers: with both
// operands holding x, v_permlane16_swap_b32 leaves 16-lane rows (0, 0, 2, 2)
// of x in the first register and rows (1, 1, 3, 3) in the second, and
// v_permlane32_swap_b32 leaves the lower half twice and the upper half
// twice, so op over the two registers after each swap reduces first across
// lane ^ 16, then across lane ^ 32.  (The s_nop covers the wait states a
// permlane needs after a vector ALU write of its operands.)
template <class Op>
__device__ __forceinline__ float quarter_reduce(float x, Op op) {
  uint32_t a = bitcast<uint32_t>(x), b = a;
  asm volatile("s_nop 1\n\tv_permlane16_swap_b32 %0, %1" : "+v"(a), "+v"(b));
  x = op(bitcast<float>(a), bitcast<float>(b));
  a = bitcast<uint32_t>(x);
  b = a;
  asm volatile("s_nop 1\n\tv_permlane32_swap_b32 %0, %1" : "+v"(a), "+v"(b));
  return op(bitcast<float>(a), bitcast<float>(b));
}

// Bytes of one workgroup's partial: O normalised by its row sum, fp16
// [W waves][D/16 d-tiles][64 lanes][4 rows], then the fp32 base-2
// log-sum-exp m + log2(l) of its 16 W rows (-inf for a row that saw no
// key).  Normalised values are bounded by max |v|, so fp16 holds them with
// the output's own precision.
template <int D>
__host__ __device__ constexpr size_t attn_part_bytes(int waves) {
  return (size_t)waves * (D / 16) * kWave * 8 + (size_t)waves * 16 * 4;
}
constexpr int kMaxParts = 32;  // prefix splits + tree split, merged in one pass

template <int D, int W>
__global__ __launch_bounds__(64 * W) void tree_attention_kernel(AttnArgs a) {
  constexpr int NT = 64 * W;         // threads
  constexpr int KS = D / 32;         // k-steps of the QK^T product
  constexpr int DT = D / 16;         // d tiles of the PV product
  constexpr int HALF = D / 2;
  constexpr int KST = D + 16;        // halves per LDS row (32-byte pad)
  constexpr int VPR = D / 8;         // 16-byte vectors per key row
  constexpr int NV = kKeyTile * VPR / NT;  // vectors per thread per matrix per tile
  static_assert(NV >= 1 && kKeyTile * VPR % NT == 0, "tile split");
  __shared__ uint16_t ks[kAttnLds][kKeyTile * KST];
  __shared__ uint16_t vs[kAttnLds][kKeyTile * KST];
  __shared__ uint64_t s_anc[64];
  __shared__ uint64_t s_cmask[64];  // draft model: visible tree-cache rows of each new token
  __shared__ int32_t s_depth[64];
  __shared__ int32_t s_status;

  const int tid = threadIdx.x;
  const int lane = lane_id();
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int n16 = lane & 15;
  const int kq = lane >> 4;
  const int g = blockIdx.x % a.Hkv;
  const int rest = blockIdx.x / a.Hkv;
  const int sp = rest % (a.nsplit + 1);
  const int rb = rest / (a.nsplit + 1);
  const bool tree_split = sp == a.nsplit;

  // ---- prefix length; this split's first key tiles go out before anything
  // else (an out-of-range P addresses from 0 and is rejected below) ----
  const int P_dev = __builtin_amdgcn_readfirstlane(*a.prefix_len);
  const bool p_ok = P_dev >= 0 && P_dev <= a.S_max - a.T - a.N;
  const int P = p_ok ? P_dev : 0;
  const int PK = P + a.N;  // the splits stream keys [0, PK); the new rows go to PK + i
  int k_lo = 0, k_hi = 0, ntiles = 0;
  if (!tree_split) {
    const int per = (PK + a.nsplit - 1) / a.nsplit;
    const int chunk = ((per + kKeyTile - 1) / kKeyTile) * kKeyTile;
    k_lo = min(PK, sp * chunk);
    k_hi = min(PK, k_lo + chunk);
    ntiles = (k_hi - k_lo + kKeyTile - 1) / kKeyTile;
  }
  k_lo = __builtin_amdgcn_readfirstlane(k_lo);
  k_hi = __builtin_amdgcn_readfirstlane(k_hi);
  ntiles = __builtin_amdgcn_readfirstlane(ntiles);
  const uint16_t* kc = a.k_cache + (size_t)g * a.S_max * D;
  const uint16_t* vc = a.v_cache + (size_t)g * a.S_max * D;
  u32x4 kbuf[kAttnRing][NV], vbuf[kAttnRing][NV];
  // tile t (clamped to the chunk's last; rows past k_hi repeat row k_hi - 1
  // and are masked).  Only called when ntiles > 0.
  auto load_tile = [&](int t, u32x4 (&kd)[NV], u32x4 (&vd)[NV]) {
    int tt = __builtin_amdgcn_readfirstlane(t < ntiles ? t : ntiles - 1);
    asm volatile("" : "+s"(tt));
    const int key0 = k_lo + tt * kKeyTile;
#pragma unroll
    for (int j = 0; j < NV; ++j) {
      const int idx = tid + j * NT;
      const int key = min(key0 + idx / VPR, k_hi - 1);
      const int c8 = (idx % VPR) * 8;
      kd[j] = *reinterpret_cast<const u32x4*>(kc + (size_t)key * D + c8);
      vd[j] = *reinterpret_cast<const u32x4*>(vc + (size_t)key * D + c8);
    }
  };
  auto retire = [&](const u32x4 (&kd)[NV], const u32x4 (&vd)[NV]) {
#pragma unroll
    for (int j = 0; j < NV; ++j) asm volatile("" : : "v"(kd[j]), "v"(vd[j]));
  };
  if (ntiles > 0) {
#pragma unroll
    for (int j = 0; j < kAttnRing - 1; ++j) load_tile(j, kbuf[j], vbuf[j]);
  }

  // ---- tree masks and validity ----
  if (wave == 0) {
    uint64_t anc, cmask = 0ull;
    int depth;
    bool ok;
    if (a.leaf_parent) {
      // draft model: the tree cache's forest masks; new token i sees the
      // cached root path of its parent (the parent included) and itself,
      // at depth one more than its parent's (0 below the last prefix token)
      uint64_t canc;
      int cdepth;
      const bool fok = tree_masks_wave<true>(a.cache_parent, a.N, canc, cdepth);
      const int lp = lane < a.T ? a.leaf_parent[lane] : -1;
      const bool lok = __all(lane >= a.T || (lp >= -1 && lp < a.N));
      const int src = (lp >= 0 && lp < a.N) ? lp : 0;
      const uint64_t pm = shfl_u64(canc, src);
      const int pd = __shfl(cdepth, src, kWave);
      const bool has = lane < a.T && lp >= 0 && lp < a.N;
      cmask = has ? pm : 0ull;
      depth = has ? pd + 1 : 0;
      anc = lane < a.T ? (1ull << lane) : 0ull;
      ok = fok && lok;
    } else {
      ok = tree_masks_wave(a.parent, a.T, anc, depth);
    }
    s_anc[lane] = anc;
    s_cmask[lane] = cmask;
    s_depth[lane] = depth;
    if (lane == 0) {
      int st = 0;
      if (!ok) st |= SWIFTSPEC_DEVERR_BAD_TREE;
      if (!p_ok) st |= SWIFTSPEC_DEVERR_BAD_PREFIX;
      s_status = st;
      if (st && blockIdx.x == 0) report_error(a.ws, (uint32_t)st);
    }
  }
  __syncthreads();
  const int nparts = a.nsplit + 1;
  const size_t grp = (size_t)g * a.RB + rb;
  char* mine = reinterpret_cast<char*>(a.part) + (grp * nparts + sp) * attn_part_bytes<D>(W);
  float* lse = reinterpret_cast<float*>(mine + (size_t)W * (D / 16) * kWave * 8);
  if (s_status) {
    // invalid tree or prefix: empty partials, so the merge leaves the output alone
    if (ntiles > 0) {
#pragma unroll
      for (int j = 0; j < kAttnRing - 1; ++j) retire(kbuf[j], vbuf[j]);
    }
    if (tid < 16 * W) lse[tid] = -INFINITY;
    return;
  }

  // ---- this wave's 16 query rows: rotated Q as B fragments ----
  const int row = rb * (16 * W) + wave * 16 + n16;
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
    const float* cs = a.rope + (size_t)(P + s_depth[node]) * D;  // [D/2][2]
#pragma unroll
    for (int j = 0; j < KS / 2; ++j) {
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const int d = 32 * j + 8 * kq + e;  // < D/2; partner d + D/2 sits in k-step j + KS/2
        const float c = cs[2 * d], sn = cs[2 * d + 1];
        const float x1 = qv[j][e], x2 = qv[j + KS / 2][e];
        qv[j][e] = x1 * c - x2 * sn;
        qv[j + KS / 2][e] = x2 * c + x1 * sn;
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

  // running maximum of row n16 (the same in its four lanes) and this lane's
  // share of the row's running sum (its 16 keys of every tile); the shares
  // are added once, at the end
  float m_run = -INFINITY, l_run = 0.f;
  f32x4 o[DT];
#pragma unroll
  for (int dt = 0; dt < DT; ++dt) o[dt] = f32x4{0.f, 0.f, 0.f, 0.f};
  const uint64_t anc = s_anc[node];
  const uint64_t cmask = s_cmask[node];

  // ---- one 64-key tile from LDS slot `slot`: scores, mask, softmax, P.V ----
  // mode 0: no mask beyond key_end; 1: tree keys, ancestor-or-self bits;
  // 2: streamed keys reaching the draft tree cache, key kr of the tile is
  // row kbase + kr of the tree cache (negative: a prefix row)
  auto compute = [&](int slot, int key_end, int mode, int kbase) {
    f32x4 s[4];
#pragma unroll
    for (int st = 0; st < 4; ++st) {
      f32x4 c = {0.f, 0.f, 0.f, 0.f};
      const uint16_t* krow = &ks[slot][(st * 16 + n16) * KST + 8 * kq];
#pragma unroll
      for (int j = 0; j < KS; ++j) {
        half8 kf = *reinterpret_cast<const half8*>(krow + 32 * j);
        c = __builtin_amdgcn_mfma_f32_16x16x32_f16(kf, qf[j], c, 0, 0, 0);
      }
      s[st] = c;  // lane: keys st*16 + 4*kq + r (r < 4), query row n16
    }
    // raw scores q.k; the softmax scale and log2 e (c > 0) enter in fp32 at
    // the exponent, 2^(c s - m); full prefix tiles need no mask
    const float c2 = a.scale_log2;
    float tmax = -INFINITY;
    if (mode == 0 && key_end >= kKeyTile) {
#pragma unroll
      for (int st = 0; st < 4; ++st)
#pragma unroll
        for (int r = 0; r < 4; ++r) tmax = fmaxf(tmax, s[st][r]);
    } else {
#pragma unroll
      for (int st = 0; st < 4; ++st)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int kr = st * 16 + 4 * kq + r;
          bool ok = kr < key_end;
          if (mode == 1) ok = ok && ((anc >> kr) & 1ull);
          if (mode == 2) {
            const int cr = kbase + kr;
            ok = ok && (cr < 0 || (cr < 64 && ((cmask >> (cr & 63)) & 1ull)));
          }
          const float v = ok ? s[st][r] : -INFINITY;
          s[st][r] = v;
          tmax = fmaxf(tmax, v);
        }
    }
    tmax = quarter_reduce(tmax, [](float x, float y) { return fmaxf(x, y); });
    const float m_new = fmaxf(m_run, tmax * c2);  // base-2 units
    // reference point of the exponentials: m_new, or 0 while the row has seen
    // no key (then every exponent is -inf and its 2^x is 0, never NaN)
    const float m_use = (m_new == -INFINITY) ? 0.f : m_new;
    const float alpha = __builtin_amdgcn_exp2f(m_run - m_use);
    float pr[16];
    half8 pf[2];
#pragma unroll
    for (int st = 0; st < 4; ++st)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        pr[st * 4 + r] = __builtin_amdgcn_exp2f(__builtin_fmaf(s[st][r], c2, -m_use));
        pf[st >> 1][(st & 1) * 4 + r] = (_Float16)pr[st * 4 + r];
      }
#pragma unroll
    for (int w = 1; w < 16; w *= 2)  // pairwise sum of the lane's 16 keys
#pragma unroll
      for (int e = 0; e < 16; e += 2 * w) pr[e] += pr[e + w];
    l_run = l_run * alpha + pr[0];
    m_run = m_new;
    // rescale O (lane holds rows 4*kq + r; fetch those rows' alpha), unless
    // no row's maximum moved
    if (__any(alpha != 1.f)) {
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const float ar = __shfl(alpha, 4 * kq + r, kWave);
#pragma unroll
        for (int dt = 0; dt < DT; ++dt) o[dt][r] *= ar;
      }
    }
    // O += P . V.  A-slot 8 kq + 4 h + r of pf[pp] holds key 32 pp + 16 h +
    // 4 kq + r; the B fragment of d-tile dt needs V[that key][16 dt + n16],
    // i.e. two transpose reads of 4 consecutive keys (h = 0, 1), for which
    // this lane addresses key kb + n16 / 4, columns 16 dt + 4 (n16 % 4) + 0..3.
#pragma unroll
    for (int pp = 0; pp < 2; ++pp) {
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) {
        v4i16 hv[2];
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          const int kb = 32 * pp + 16 * h + 4 * kq + (n16 >> 2);
          const uint16_t* pv = &vs[slot][kb * KST + 16 * dt + 4 * (n16 & 3)];
          hv[h] = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
              (__attribute__((address_space(3))) v4i16*)(pv));
        }
        const half8 vf = bitcast<half8>(u32x4{bitcast<u32x2>(hv[0])[0], bitcast<u32x2>(hv[0])[1],
                                              bitcast<u32x2>(hv[1])[0], bitcast<u32x2>(hv[1])[1]});
        o[dt] = __builtin_amdgcn_mfma_f32_16x16x32_f16(pf[pp], vf, o[dt], 0, 0, 0);
      }
    }
  };

  if (tree_split) {
    // tree keys: rotate k at position P + depth, round to fp16; copy v.
    // Thread handles (key kr, 8 rotation pairs starting at c8 < D/2).
    constexpr int kPairVecs = HALF / 8;
    for (int idx = tid; idx < kKeyTile * kPairVecs; idx += NT) {
      const int kr = idx / kPairVecs, c8 = (idx % kPairVecs) * 8;
      u32x4 k1 = {0, 0, 0, 0}, k2 = {0, 0, 0, 0}, v1 = {0, 0, 0, 0}, v2 = {0, 0, 0, 0};
      if (kr < a.T) {
        const uint16_t* ksrc = a.k + (size_t)kr * a.ldkv + g * D;
        const uint16_t* vsrc = a.v + (size_t)kr * a.ldkv + g * D;
        u32x4 r1 = *reinterpret_cast<const u32x4*>(ksrc + c8);
        u32x4 r2 = *reinterpret_cast<const u32x4*>(ksrc + c8 + HALF);
        v1 = *reinterpret_cast<const u32x4*>(vsrc + c8);
        v2 = *reinterpret_cast<const u32x4*>(vsrc + c8 + HALF);
        const float* cs = a.rope + (size_t)(P + s_depth[kr]) * D;
        half8 h1 = bitcast<half8>(r1), h2 = bitcast<half8>(r2), o1, o2;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const float c = cs[2 * (c8 + e)], sn = cs[2 * (c8 + e) + 1];
          const float x1 = (float)h1[e], x2 = (float)h2[e];
          o1[e] = (_Float16)(x1 * c - x2 * sn);
          o2[e] = (_Float16)(x2 * c + x1 * sn);
        }
        k1 = bitcast<u32x4>(o1);
        k2 = bitcast<u32x4>(o2);
        if (rb == 0) {
          uint16_t* kd = a.k_cache + ((size_t)g * a.S_max + PK + kr) * D;
          uint16_t* vd = a.v_cache + ((size_t)g * a.S_max + PK + kr) * D;
          *reinterpret_cast<u32x4*>(kd + c8) = k1;
          *reinterpret_cast<u32x4*>(kd + c8 + HALF) = k2;
          *reinterpret_cast<u32x4*>(vd + c8) = v1;
          *reinterpret_cast<u32x4*>(vd + c8 + HALF) = v2;
        }
      }
      *reinterpret_cast<u32x4*>(&ks[0][kr * KST + c8]) = k1;
      *reinterpret_cast<u32x4*>(&ks[0][kr * KST + c8 + HALF]) = k2;
      *reinterpret_cast<u32x4*>(&vs[0][kr * KST + c8]) = v1;
      *reinterpret_cast<u32x4*>(&vs[0][kr * KST + c8 + HALF]) = v2;
    }
    __syncthreads();
    compute(0, a.T, 1, 0);
  } else {
    // ---- prefix chunk of this split (first tiles already in flight) ----
    if (ntiles > 0) {
      auto store_tile = [&](int slot, const u32x4 (&kd)[NV], const u32x4 (&vd)[NV]) {
#pragma unroll
        for (int j = 0; j < NV; ++j) {
          const int idx = tid + j * NT;
          const int off = (idx / VPR) * KST + (idx % VPR) * 8;
          *reinterpret_cast<u32x4*>(&ks[slot][off]) = kd[j];
          *reinterpret_cast<u32x4*>(&vs[slot][off]) = vd[j];
        }
      };
      store_tile(0, kbuf[0], vbuf[0]);
      // step t: load tile t + 4, write tile t + 1 to LDS slot (t + 1) % 3
      // (last read at step t - 2), barrier, compute tile t; whole rounds of
      // five steps, steps past the end only load (the first one leaves)
      for (int t0 = 0; t0 < ntiles; t0 += kAttnRing) {
#pragma unroll
        for (int J = 0; J < kAttnRing; ++J) {
          const int t = t0 + J;
          load_tile(t + kAttnRing - 1, kbuf[(J + kAttnRing - 1) % kAttnRing], vbuf[(J + kAttnRing - 1) % kAttnRing]);
          if (t < ntiles) {
            if (t + 1 < ntiles) store_tile((t + 1) % kAttnLds, kbuf[(J + 1) % kAttnRing], vbuf[(J + 1) % kAttnRing]);
            lds_barrier();
            const int key0 = k_lo + t * kKeyTile;
            compute(t % kAttnLds, k_hi - key0, (a.N > 0 && key0 + kKeyTile > P) ? 2 : 0, key0 - P);
          } else {
            retire(kbuf[J], vbuf[J]);
          }
        }
      }
    }
  }

  // ---- publish this split's partial (merged by the next kernel) ----
  l_run = quarter_reduce(l_run, [](float x, float y) { return x + y; });
  float inv[4];
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const float lr = __shfl(l_run, 4 * kq + r, kWave);
    inv[r] = lr > 0.f ? 1.0f / lr : 0.f;
  }
#pragma unroll
  for (int dt = 0; dt < DT; ++dt) {
    const uint32_t lo = (uint32_t)f2h(o[dt][0] * inv[0]) | ((uint32_t)f2h(o[dt][1] * inv[1]) << 16);
    const uint32_t hi = (uint32_t)f2h(o[dt][2] * inv[2]) | ((uint32_t)f2h(o[dt][3] * inv[3]) << 16);
    *reinterpret_cast<u32x2*>(mine + ((size_t)(wave * DT + dt) * kWave + lane) * 8) = u32x2{lo, hi};
  }
  if (kq == 0) lse[wave * 16 + n16] = l_run > 0.f ? m_run + __log2f(l_run) : -INFINITY;
}

// Merge of the S + 1 <= NP partials of one 16-row x 16-column output tile,
// in split order: with L_s the log-sum-exp of a row in split s and O_s its
// normalised output, O = sum_s 2^(L_s - L) O_s, L = log2 sum_s 2^L_s (taken
// relative to max_s L_s).  One wave per tile (lane: rows 4 (lane / 16) + r,
// column lane % 16); every split's loads are issued at once, so the kernel
// is one memory round trip long.  Grid = Hkv x RB x W x D/16 with the KV
// head in blockIdx % Hkv, so that with 8 KV heads a head's merge runs on the
// XCD whose L2 holds the head's partials (round-robin dispatch puts
// blockIdx % 8 on XCD blockIdx % 8, as for the attention kernel).  A row that
// no split saw (only when the attention kernel rejected the tree or the
// prefix and published empty partials) is not written.
template <int D, int W, int NP>
__global__ __launch_bounds__(64) void tree_attention_merge_kernel(AttnArgs a) {
  constexpr int DT = D / 16;
  const int lane = lane_id();
  const int n16 = lane & 15, kq = lane >> 4;
  const int g = blockIdx.x % a.Hkv;
  const int rest = blockIdx.x / a.Hkv;
  const int dt = rest % DT;
  const int wave = (rest / DT) % W;
  const int rb = rest / (DT * W);
  const int grp = g * a.RB + rb;
  const int nparts = a.nsplit + 1;
  const size_t part_stride = attn_part_bytes<D>(W);
  const char* base = reinterpret_cast<const char*>(a.part) + (size_t)grp * nparts * part_stride;
  // the group's partials as one buffer: part j at scalar offset j * stride
  const auto rp = buffer_rsrc(base, (uint32_t)(nparts * part_stride));
  const uint32_t off_l = (uint32_t)(W * DT * kWave * 8 + (wave * 16 + 4 * kq) * 4);
  const uint32_t off_o = (uint32_t)(((wave * DT + dt) * kWave + lane) * 8);
  f32x4 ls[NP];
  u32x2 ov[NP];
#pragma unroll
  for (int j = 0; j < NP; ++j) {
    const uint32_t soff = (uint32_t)((j < nparts ? j : nparts - 1) * part_stride);
    ls[j] = bitcast<f32x4>(buffer_load_x4(rp, off_l, soff));
    ov[j] = bitcast<u32x2>(__builtin_amdgcn_raw_buffer_load_b64(rp, off_o, soff, 0));
  }
  // branch-free: parts past nparts weigh 2^-inf = 0
#pragma unroll
  for (int j = 0; j < NP; ++j)
    if (j >= nparts) ls[j] = f32x4{-INFINITY, -INFINITY, -INFINITY, -INFINITY};
  float lmax[4] = {-INFINITY, -INFINITY, -INFINITY, -INFINITY};
#pragma unroll
  for (int j = 0; j < NP; ++j)
#pragma unroll
    for (int r = 0; r < 4; ++r) lmax[r] = fmaxf(lmax[r], ls[j][r]);
  // a row that no split saw keeps lmax = -inf: its weights are computed
  // against 0 (all zero) and the row is not written
  float ref[4];
#pragma unroll
  for (int r = 0; r < 4; ++r) ref[r] = lmax[r] == -INFINITY ? 0.f : lmax[r];
  float wsum[4] = {0.f, 0.f, 0.f, 0.f}, acc[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int j = 0; j < NP; ++j)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const float w = __builtin_amdgcn_exp2f(ls[j][r] - ref[r]);
      wsum[r] += w;
      acc[r] = __builtin_fmaf(w, h2f((uint16_t)(ov[j][r >> 1] >> (16 * (r & 1)))), acc[r]);
    }
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int orow = rb * (16 * W) + wave * 16 + 4 * kq + r;
    if (orow < a.R && lmax[r] != -INFINITY) {
      const int i = orow / a.G, qh = g * a.G + orow % a.G;
      const uint16_t h = f2h(acc[r] / wsum[r]);
      a.out[(size_t)i * a.ldo + qh * D + dt * 16 + n16] = h;
      if (a.out_prep) store_prepared(a.out_prep, i, qh * D + dt * 16 + n16, (a.Hq * D) >> 7, h);
    }
  }
}

// merge launch: the partial count decides how many loads a lane issues
template <int D, int W>
static void launch_merge(const AttnArgs& a, hipStream_t st) {
  const dim3 mgrid(a.Hkv * a.RB * W * (D / 16));
  if (a.nsplit + 1 <= 16) hipLaunchKernelGGL((tree_attention_merge_kernel<D, W, 16>), mgrid, dim3(64), 0, st, a);
  else hipLaunchKernelGGL((tree_attention_merge_kernel<D, W, kMaxParts>), mgrid, dim3(64), 0, st, a);
}


// ============================================================================
// Target model (square tree mask, no tree cache).  The prefix keys stream
// in 32-key stages fetched straight into LDS by 16-byte buffer loads to LDS
// (lane i of a wave's load lands at 16-byte chunk i of a 1 KB block whose
// base the wave chooses), up to 8 stages deep, so no register ring is needed
// and up to seven stages (112 KB) are in flight per workgroup.  Every wave
// keeps 32 query rows (two 16-row tiles sharing each K and V fragment read
// from LDS); workgroups of 1, 2 or 4 waves (two workgroups per compute unit)
// or of 8 waves (one), two waves per SIMD either way.  The prologue makes
// two memory round trips (parent array and queries; then the rotary rows at
// P + depth, loaded ahead of the first stages).
// LDS layout of one stage (see KvLds): 1 KB blocks of key rows at a stride
// of 1088 (K) or 1152 (V) bytes, and within a block row i the 16-byte chunk
// c of the row stored at chunk c ^ x(i); each lane of a load fetches the
// global chunk that belongs at its position.  With these the K-fragment
// reads (16 rows, one chunk each) and the transposed V reads (8 rows, 32
// bytes each) hit every bank once, and all K reads of a lane are one base
// register plus immediate offsets.  Softmax: per-row reference maximum
// raised lazily (only when a stage's maximum exceeds it by more than 2^8;
// the unnormalised probabilities stay below 256, with fp16's relative
// precision), row sums formed by the matrix cores (P times a ones column);
// a stage whose scores all stay within 2^8 of the reference takes no
// cross-lane step (only a per-lane maximum and one wave-wide vote).
// Partials use the merge kernel's layout with two 16-row "virtual waves" per
// wave.
constexpr int kFastKeys = 32;         // keys per LDS stage
constexpr float kLazyRescale = 8.0f;  // log2 of the largest unnormalised probability

template <int D>
struct KvLds {
  static constexpr int kCpr = D / 8;                // 16-byte chunks per key row
  static constexpr int kRpb = 1024 / (2 * D);       // key rows per 1 KB block
  static constexpr int kBlocks = kFastKeys / kRpb;  // blocks per matrix and stage
  static constexpr int kKStride = 1088, kVStride = 1152;
  static constexpr int kKBytes = kBlocks * kKStride;
  static constexpr int kStage = kKBytes + kBlocks * kVStride;
  // chunk XOR of row i of a block: K on chunk bits 0-1, V on bits 1-2
  static __device__ __forceinline__ int xk(int i) { return D == 128 ? i : i >> 1; }
  static __device__ __forceinline__ int xv(int i) { return D == 128 ? 2 * i : 2 * (i >> 1); }
  // byte offsets of chunk c of stage key row `key` in the K / V region
  static __device__ __forceinline__ int k_off(int key, int c) {
    const int b = key / kRpb, i = key % kRpb;
    return b * kKStride + i * 2 * D + ((c ^ xk(i)) << 4);
  }
  static __device__ __forceinline__ int v_off(int key, int c) {
    const int b = key / kRpb, i = key % kRpb;
    return kKBytes + b * kVStride + i * 2 * D + ((c ^ xv(i)) << 4);
  }
};

// 16-byte global load issued as inline assembly: the compiler inserts no
// wait for it (it does not see the load), so the caller waits with vm_wait
// and then passes the value through after_wait, which the uses depend on
__device__ __forceinline__ u32x4 load_x4_untracked(const void* p) {
  u32x4 v;
  asm volatile("global_load_dwordx4 %0, %1, off" : "=v"(v) : "v"(p));
  return v;
}
template <typename T>
__device__ __forceinline__ void after_wait(T& x) {
  asm volatile("" : "+v"(x));
}
// wait until at most `behind` stages (LPW loads each) of this wave remain in flight
template <int LPW, int K>
__device__ __forceinline__ void vm_wait_stages(int behind) {
  if constexpr (K == 0) {
    vm_wait<0>();
  } else {
    if (behind >= K) vm_wait<LPW * K>();
    else vm_wait_stages<LPW, K - 1>(behind);
  }
}

// Stages per workgroup: about 70 KB of LDS, so that two workgroups share a
// compute unit (two waves per SIMD, from workgroups whose barriers are
// independent, so one's matrix-core work overlaps the other's softmax).
template <int D, int W>
struct FastAttnCfg {
  static constexpr int kLoadsPerWave = 2 * KvLds<D>::kBlocks / W;  // 1 KB loads per stage (K and V)
  static constexpr int kStages = D == 128 ? 4 : 8;
  static_assert(kLoadsPerWave * (kStages - 1) <= 63, "vmcnt range");
  static_assert((2 * KvLds<D>::kBlocks) % W == 0, "stage split");
};

template <int D, int W, int TPW>
__global__ __launch_bounds__(64 * W) __attribute__((amdgpu_waves_per_eu(W * TPW >= 8 ? 2 : 1))) void tree_attention_fast_kernel(AttnArgs a) {
  using L = KvLds<D>;
  using Cfg = FastAttnCfg<D, W>;
  constexpr int NS = Cfg::kStages;
  constexpr int LPW = Cfg::kLoadsPerWave;
  constexpr int KS = D / 32;   // k-steps of the QK^T product
  constexpr int DT = D / 16;   // d tiles of the PV product
  constexpr int HALF = D / 2;
  constexpr int VW = TPW * W;  // 16-row virtual waves of the partial layout
  __shared__ __attribute__((aligned(16))) char kvs[NS * L::kStage];
  const int tid = threadIdx.x;
  const int lane = lane_id();
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int n16 = lane & 15;
  const int kq = lane >> 4;
  const int g = blockIdx.x % a.Hkv;
  const int rest = blockIdx.x / a.Hkv;
  const int sp = rest % (a.nsplit + 1);
  const int rb = rest / (a.nsplit + 1);
  const bool tree_split = sp == a.nsplit;

  // ---- prologue, two memory round trips: (1) the parent array and this
  // wave's raw query rows; (2) after the tree masks (every wave forms them
  // for all nodes), the rotary rows at P + depth, issued ahead of the first
  // key and value stages so that waiting for them leaves those in flight ----
  const int par = lane < a.T ? a.parent[lane] : -1;
  int node[TPW], qhead[TPW];
  bool row_ok[TPW];
  u32x4 qraw[TPW][KS];
#pragma unroll
  for (int t2 = 0; t2 < TPW; ++t2) {
    const int row = rb * (16 * VW) + wave * (16 * TPW) + t2 * 16 + n16;
    row_ok[t2] = row < a.R;
    node[t2] = row_ok[t2] ? row / a.G : 0;
    qhead[t2] = g * a.G + (row_ok[t2] ? row % a.G : 0);
    const uint16_t* qsrc = a.q + (size_t)node[t2] * a.ldq + qhead[t2] * D + 8 * kq;
#pragma unroll
    for (int j = 0; j < KS; ++j) qraw[t2][j] = load_x4_untracked(qsrc + 32 * j);
  }
  const int P_dev = __builtin_amdgcn_readfirstlane(*a.prefix_len);
  const bool p_ok = P_dev >= 0 && P_dev <= a.S_max - a.T;
  const int P = p_ok ? P_dev : 0;
  // this split's key range: stages [t0, t1) of the prefix's 32-key stages
  int k_lo = 0, k_hi = 0, ntiles = 0;
  if (!tree_split) {
    const int tiles = (P + kFastKeys - 1) / kFastKeys;
    const int t0 = sp * tiles / a.nsplit, t1 = (sp + 1) * tiles / a.nsplit;
    k_lo = t0 * kFastKeys;
    k_hi = min(P, t1 * kFastKeys);
    ntiles = t1 - t0;
  }
  k_lo = __builtin_amdgcn_readfirstlane(k_lo);
  k_hi = __builtin_amdgcn_readfirstlane(k_hi);
  ntiles = __builtin_amdgcn_readfirstlane(ntiles);

  // ---- tree masks and validity ----
  uint64_t anc_all;
  int depth_all;
  const bool tree_ok = tree_masks_from(par, a.T, anc_all, depth_all);
  const int nparts = a.nsplit + 1;
  const size_t grp = (size_t)g * a.RB + rb;
  char* mine = reinterpret_cast<char*>(a.part) + (grp * nparts + sp) * attn_part_bytes<D>(VW);
  float* lse = reinterpret_cast<float*>(mine + (size_t)VW * DT * kWave * 8);
  if (!tree_ok || !p_ok) {
    // invalid tree or prefix: empty partials, so the merge leaves the output
    // alone (no key or value stage has been issued)
    if (blockIdx.x == 0 && tid == 0)
      report_error(a.ws, (tree_ok ? 0u : (uint32_t)SWIFTSPEC_DEVERR_BAD_TREE) |
                             (p_ok ? 0u : (uint32_t)SWIFTSPEC_DEVERR_BAD_PREFIX));
    if (tid < 16 * VW) lse[tid] = -INFINITY;
    vm_wait<0>();
    return;
  }
  uint64_t anc[TPW];
  u32x4 csraw[TPW][KS / 2][4];  // cos/sin pairs of dimensions 32 j + 8 kq + 0..7
#pragma unroll
  for (int t2 = 0; t2 < TPW; ++t2) {
    anc[t2] = shfl_u64(anc_all, node[t2]);
    const int dep = __shfl(depth_all, node[t2], kWave);
    const float* cs = a.rope + (size_t)(P + dep) * D;  // [D/2][2]
#pragma unroll
    for (int j = 0; j < KS / 2; ++j)
#pragma unroll
      for (int c = 0; c < 4; ++c) csraw[t2][j][c] = load_x4_untracked(cs + 2 * (32 * j + 8 * kq) + 4 * c);
  }

  // ---- the first stages of keys and values ----
  // the head's cache rows as buffer resources (loads past the last row
  // return zeros; such keys are masked)
  const uint32_t head_bytes = (uint32_t)((size_t)a.S_max * D * 2);
  const i32x4 rk = raw_rsrc(a.k_cache + (size_t)g * a.S_max * D, head_bytes);
  const i32x4 rv = raw_rsrc(a.v_cache + (size_t)g * a.S_max * D, head_bytes);
  // this lane's part of every 1 KB block: row i of the block, the global
  // chunk that belongs at its position (pos ^ x(i))
  const int li = lane / L::kCpr, lpos = lane % L::kCpr;
  const uint32_t voff_k = (uint32_t)(li * 2 * D + ((lpos ^ L::xk(li)) << 4));
  const uint32_t voff_v = (uint32_t)(li * 2 * D + ((lpos ^ L::xv(li)) << 4));
  // stage t (< ntiles) into slot t % NS: wave w issues block loads w, w + W,
  // ... of the stage's K blocks followed by its V blocks (blocks wholly past
  // k_hi reload the block holding row k_hi - 1)
  const int last_blk_row = k_hi > 0 ? ((k_hi - 1) / L::kRpb) * L::kRpb : 0;
  auto issue_tile = [&](int t) __attribute__((always_inline)) {
    const int row0 = k_lo + t * kFastKeys;
    const char* st = kvs + (t % NS) * L::kStage;
#pragma unroll
    for (int i = 0; i < LPW; ++i) {
      const int inst = i * W + wave;
      const bool isv = inst >= L::kBlocks;
      const int blk = isv ? inst - L::kBlocks : inst;
      const uint32_t soff = (uint32_t)min(row0 + blk * L::kRpb, last_blk_row) * (uint32_t)(2 * D);
      const char* dst = st + (isv ? L::kKBytes + blk * L::kVStride : blk * L::kKStride);
      buffer_load_lds16(isv ? rv : rk, isv ? voff_v : voff_k, soff,
                        __builtin_amdgcn_readfirstlane(lds_address(dst)));
    }
  };
#pragma unroll
  for (int j = 0; j < NS - 1; ++j)
    if (j < ntiles) issue_tile(j);
  // the query and rotary loads, older than those stages, have landed
  vm_wait_stages<LPW, NS - 1>(min(ntiles, NS - 1));

  // ---- this wave's 32 query rows (tiles t2 = 0, 1): rotated Q as B fragments ----
  const float c2 = a.scale_log2;
  half8 qf[TPW][KS];
#pragma unroll
  for (int t2 = 0; t2 < TPW; ++t2) {
    float qv[KS][8];
#pragma unroll
    for (int j = 0; j < KS; ++j) {
      after_wait(qraw[t2][j]);
      const half8 h = bitcast<half8>(qraw[t2][j]);
#pragma unroll
      for (int e = 0; e < 8; ++e) qv[j][e] = row_ok[t2] ? (float)h[e] : 0.f;
    }
#pragma unroll
    for (int j = 0; j < KS / 2; ++j) {
      float cs[16];
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        after_wait(csraw[t2][j][c]);
#pragma unroll
        for (int e = 0; e < 4; ++e) cs[4 * c + e] = bitcast<float>(csraw[t2][j][c][e]);
      }
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        // dimension 32 j + 8 kq + e (< D/2); its partner + D/2 sits in k-step j + KS/2
        const float c = cs[2 * e], sn = cs[2 * e + 1];
        const float x1 = qv[j][e], x2 = qv[j + KS / 2][e];
        qv[j][e] = x1 * c - x2 * sn;
        qv[j + KS / 2][e] = x2 * c + x1 * sn;
      }
    }
#pragma unroll
    for (int j = 0; j < KS; ++j) {
      half8 h;
#pragma unroll
      for (int e = 0; e < 8; ++e) h[e] = (_Float16)qv[j][e];
      qf[t2][j] = h;
    }
  }

  // per-row softmax state in the score layout (row n16 of tile t2), base 2:
  // the reference exponent m_ref and the rescale threshold thr (m_ref +
  // kLazyRescale once the row has seen a key, -inf before); output and row-sum
  // accumulators (O layout: rows 4 kq + r, column n16)
  float m_ref[TPW], thr[TPW];
  f32x4 o[TPW][DT], ol[TPW];
#pragma unroll
  for (int t2 = 0; t2 < TPW; ++t2) {
    m_ref[t2] = 0.f;
    thr[t2] = -INFINITY;
    ol[t2] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) o[t2][dt] = f32x4{0.f, 0.f, 0.f, 0.f};
  }
  const half8 ones = {(_Float16)1.f, (_Float16)1.f, (_Float16)1.f, (_Float16)1.f,
                      (_Float16)1.f, (_Float16)1.f, (_Float16)1.f, (_Float16)1.f};
  // LDS read offsets of this lane: K chunk 4 j + kq of key n16 (+ 16 h rows
  // = 16 h / kRpb blocks, + 64 j bytes); V 8-byte piece (n16 % 4) of columns
  // 16 dt + 4 (n16 % 4) of key 4 kq + n16 / 4 (+ 16 h rows), for dt % 4
  // (D = 128: + 128 bytes for dt >= 4)
  const int k_base = L::k_off(n16, kq);
  int v_base[DT < 4 ? DT : 4];
#pragma unroll
  for (int d2 = 0; d2 < (DT < 4 ? DT : 4); ++d2)
    v_base[d2] = L::v_off(4 * kq + (n16 >> 2), 2 * d2 + ((n16 & 3) >> 1)) + 8 * (n16 & 1);

  // ---- one 32-key stage at sb: keys [0, key_end) valid (kMask), tree
  // stages (kTree) also apply the ancestor-or-self mask of keys tree0 + k ----
  auto compute = [&](const char* sb, int key_end, int tree0, auto mask_tag, auto tree_tag)
      __attribute__((always_inline)) {
    constexpr bool kMask = decltype(mask_tag)::value;
    constexpr bool kTree = decltype(tree_tag)::value;
    // S^T: lane holds keys 16 h + 4 kq + r (h < 2, r < 4) of query row n16
    f32x4 s[TPW][2];
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      half8 kf[KS];
#pragma unroll
      for (int j = 0; j < KS; ++j)
        kf[j] = *reinterpret_cast<const half8*>(sb + k_base + (16 * h / L::kRpb) * L::kKStride + 64 * j);
#pragma unroll
      for (int t2 = 0; t2 < TPW; ++t2) {
        f32x4 c = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int j = 0; j < KS; ++j) c = __builtin_amdgcn_mfma_f32_16x16x32_f16(kf[j], qf[t2][j], c, 0, 0, 0);
        s[t2][h] = c;
      }
    }
    // this lane's largest score of each tile (masked keys -inf)
    float lm[TPW];
#pragma unroll
    for (int t2 = 0; t2 < TPW; ++t2) {
      if constexpr (kMask) {
#pragma unroll
        for (int h = 0; h < 2; ++h)
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const int kr = 16 * h + 4 * kq + r;
            bool ok = kr < key_end;
            if (kTree) ok = ok && ((anc[t2] >> (tree0 + kr)) & 1ull);
            if (!ok) s[t2][h][r] = -INFINITY;
          }
      }
      // (IEEE maximum: three-input v_maximum3_f32, where fmaxf would add
      // one quieting v_max per matrix-core result; a NaN score makes its
      // probability NaN either way)
      auto mx = [](float x, float y) { return __builtin_elementwise_maximum(x, y); };
      lm[t2] = mx(mx(mx(s[t2][0][0], s[t2][0][1]), mx(s[t2][0][2], s[t2][0][3])),
                  mx(mx(s[t2][1][0], s[t2][1][1]), mx(s[t2][1][2], s[t2][1][3])));
    }
    // move a row's reference up only when one of its scores exceeds it by
    // more than 2^8 (the probabilities then stay below 256), and set it at
    // the row's first key (scores scale by c2 > 0, so maxima commute with it)
    bool raise = lm[0] * c2 > thr[0];
    if constexpr (TPW == 2) raise = raise || lm[1] * c2 > thr[1];
    if (__any(raise)) {
#pragma unroll
      for (int t2 = 0; t2 < TPW; ++t2) {
        const float rmax = quarter_reduce(lm[t2], [](float x, float y) { return fmaxf(x, y); }) * c2;
        const bool seen = thr[t2] != -INFINITY;
        const float mn = seen ? fmaxf(m_ref[t2], rmax) : (rmax == -INFINITY ? m_ref[t2] : rmax);
        // rows that saw no key yet hold zero sums: their factor is 1
        const float alpha = seen ? __builtin_amdgcn_exp2f(m_ref[t2] - mn) : 1.f;
        m_ref[t2] = mn;
        if (seen || rmax != -INFINITY) thr[t2] = mn + kLazyRescale;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const float ar = __shfl(alpha, 4 * kq + r, kWave);
          ol[t2][r] *= ar;
#pragma unroll
          for (int dt = 0; dt < DT; ++dt) o[t2][dt][r] *= ar;
        }
      }
    }
    // probabilities 2^(c2 s - m_ref) <= 2^8 as the fp16 A fragment: slot
    // 8 kq + 4 h + r holds key 16 h + 4 kq + r
    half8 pf[TPW];
#pragma unroll
    for (int t2 = 0; t2 < TPW; ++t2) {
#pragma unroll
      for (int h = 0; h < 2; ++h)
#pragma unroll
        for (int r = 0; r < 4; ++r)
          pf[t2][h * 4 + r] = (_Float16)__builtin_amdgcn_exp2f(__builtin_fmaf(s[t2][h][r], c2, -m_ref[t2]));
      ol[t2] = __builtin_amdgcn_mfma_f32_16x16x32_f16(pf[t2], ones, ol[t2], 0, 0, 0);  // row sums
    }
    // O += P . V: V fragments by transposed reads, this lane addressing
    // key 16 h + 4 kq + n16 / 4, columns 16 dt + 4 (n16 % 4) + 0..3
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) {
      v4i16 hv[2];
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const char* pv = sb + v_base[dt & 3] + (16 * h / L::kRpb) * L::kVStride + (dt >> 2) * 128;
        hv[h] = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) v4i16*)(pv));
      }
      const half8 vf = bitcast<half8>(u32x4{bitcast<u32x2>(hv[0])[0], bitcast<u32x2>(hv[0])[1],
                                            bitcast<u32x2>(hv[1])[0], bitcast<u32x2>(hv[1])[1]});
#pragma unroll
      for (int t2 = 0; t2 < TPW; ++t2) o[t2][dt] = __builtin_amdgcn_mfma_f32_16x16x32_f16(pf[t2], vf, o[t2][dt], 0, 0, 0);
    }
  };

  if (tree_split) {
    // tree keys: rotate k at position P + depth, round to fp16; copy v; write
    // both to the cache (row block 0) and to stages 0 and 1 (keys 0-31 and
    // 32-63) in the stage layout
    constexpr int kPairVecs = HALF / 8;
    for (int idx = tid; idx < 64 * kPairVecs; idx += 64 * W) {
      const int kr = idx / kPairVecs, c8 = (idx % kPairVecs) * 8;
      const int kdep = __shfl(depth_all, kr, kWave);  // kr < 64; every lane takes part
      u32x4 k1 = {0, 0, 0, 0}, k2 = {0, 0, 0, 0}, v1 = {0, 0, 0, 0}, v2 = {0, 0, 0, 0};
      if (kr < a.T) {
        const uint16_t* ksrc = a.k + (size_t)kr * a.ldkv + g * D;
        const uint16_t* vsrc = a.v + (size_t)kr * a.ldkv + g * D;
        const u32x4 r1 = *reinterpret_cast<const u32x4*>(ksrc + c8);
        const u32x4 r2 = *reinterpret_cast<const u32x4*>(ksrc + c8 + HALF);
        v1 = *reinterpret_cast<const u32x4*>(vsrc + c8);
        v2 = *reinterpret_cast<const u32x4*>(vsrc + c8 + HALF);
        const float* cs = a.rope + (size_t)(P + kdep) * D;
        const half8 h1 = bitcast<half8>(r1), h2 = bitcast<half8>(r2);
        half8 o1, o2;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const float c = cs[2 * (c8 + e)], sn = cs[2 * (c8 + e) + 1];
          const float x1 = (float)h1[e], x2 = (float)h2[e];
          o1[e] = (_Float16)(x1 * c - x2 * sn);
          o2[e] = (_Float16)(x2 * c + x1 * sn);
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
      char* sb = kvs + (kr / kFastKeys) * L::kStage;
      const int key = kr % kFastKeys, ca = c8 / 8, cb = (c8 + HALF) / 8;
      *reinterpret_cast<u32x4*>(sb + L::k_off(key, ca)) = k1;
      *reinterpret_cast<u32x4*>(sb + L::k_off(key, cb)) = k2;
      *reinterpret_cast<u32x4*>(sb + L::v_off(key, ca)) = v1;
      *reinterpret_cast<u32x4*>(sb + L::v_off(key, cb)) = v2;
    }
    __syncthreads();
    compute(kvs, a.T, 0, std::true_type{}, std::true_type{});
    if (a.T > kFastKeys) compute(kvs + L::kStage, a.T - kFastKeys, kFastKeys, std::true_type{}, std::true_type{});
  } else {
    // step t: wait for stage t (this wave's loads; later stages may stay in
    // flight), barrier (every wave's loads of stage t have landed and every
    // wave is done with stage t - 1), refill stage t - 1's slot with stage
    // t + NS - 1, compute stage t (the last one masked past k_hi)
    // (every stage but the last is full: the loop has one unmasked body)
    for (int t = 0; t < ntiles - 1; ++t) {
      vm_wait_stages<LPW, NS - 2>(ntiles - 1 - t);
      lds_barrier();
      if (t + NS - 1 < ntiles) issue_tile(t + NS - 1);
      compute(kvs + (t % NS) * L::kStage, kFastKeys, 0, std::false_type{}, std::false_type{});
    }
    if (ntiles > 0) {
      const int t = ntiles - 1;
      vm_wait<0>();
      lds_barrier();
      compute(kvs + (t % NS) * L::kStage, k_hi - (k_lo + t * kFastKeys), 0, std::true_type{}, std::false_type{});
    }
  }

  // ---- publish this split's partial (merged by the next kernel) ----
#pragma unroll
  for (int t2 = 0; t2 < TPW; ++t2) {
    const int vw = TPW * wave + t2;
    float inv[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) inv[r] = ol[t2][r] > 0.f ? 1.0f / ol[t2][r] : 0.f;
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) {
      const uint32_t lo = (uint32_t)f2h(o[t2][dt][0] * inv[0]) | ((uint32_t)f2h(o[t2][dt][1] * inv[1]) << 16);
      const uint32_t hi = (uint32_t)f2h(o[t2][dt][2] * inv[2]) | ((uint32_t)f2h(o[t2][dt][3] * inv[3]) << 16);
      *reinterpret_cast<u32x2*>(mine + ((size_t)(vw * DT + dt) * kWave + lane) * 8) = u32x2{lo, hi};
    }
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const float mr = __shfl(m_ref[t2], 4 * kq + r, kWave);
      if (n16 == 0) lse[vw * 16 + 4 * kq + r] = ol[t2][r] > 0.f ? mr + __log2f(ol[t2][r]) : -INFINITY;
    }
  }
}

// query rows per workgroup of the target kernel: 32 per wave, up to 4 waves,
// or 8 (one workgroup per compute unit, each key and value stage landing once
// for all 256 rows of a KV head) when a head has more than 128 rows and the
// prefix may reach 16K keys, where streaming the cache dominates
static int fast_attn_waves(int R, int P_max) {
  return R <= 32 ? 1 : R <= 64 ? 2 : (R <= 128 || P_max < 16384) ? 4 : 8;
}
// 16-row tiles per wave of the target kernel: one where a head's rows and
// the prefix splits leave a single 4-wave workgroup per compute unit (the
// 70B shape: 8 KV heads x 256 rows, 16 parts), so that 8 waves of 16 rows
// each give every SIMD two waves over the same 128 rows and LDS stages;
// else two (32 rows per wave)
static int fast_attn_tiles(int R, int P_max, int Hkv, int nsplit) {
  const int W = fast_attn_waves(R, P_max);
  if (W != 4) return 2;
  const int RB = (R + 127) / 128;
  return (long)Hkv * RB * (nsplit + 1) <= 256 ? 1 : 2;
}

static int attn_waves(int R) { return R >= 128 ? 8 : 4; }

AttnPlan plan_tree_attention(int T, int Hq, int Hkv, int D, int S_max, bool draft) {
  AttnPlan p;
  const int G = Hq / Hkv;
  const int R = T * G;
  // rows per workgroup: draft kernel 16 per wave (4 or 8 waves), target
  // kernel 32 per wave (1, 2 or 4 waves); partials in 16-row virtual waves
  const int VW = draft ? attn_waves(R) : 2 * fast_attn_waves(R, S_max - T);
  const int RB = (R + 16 * VW - 1) / (16 * VW);
  const int groups = Hkv * RB;
  // about 256 workgroups in flight, at least two key tiles per prefix split
  // (four: no change at the 70B shapes, 2 us slower at prefixes of 500-1000
  // keys with few KV heads; one: slower at 1000 keys)
  // about two workgroups per compute unit for the target kernel with up to 4
  // waves (one for the 8-wave target workgroups and for the draft kernel)
  int ns = (draft || VW == 16 ? 256 : 512) / groups - 1;
  // the draft kernel's splits span at least two 64-key tiles; the target
  // kernel's at least one 32-key stage (the 1B layer, 512 keys and 8 KV
  // heads: 5 -> 16 parts, attention + merge 10.0 -> 9.2 us)
  const int max_splits = draft ? (S_max - T + kKeyTile - 1) / kKeyTile / 2 : (S_max - T + kFastKeys - 1) / kFastKeys;
  if (ns > max_splits) ns = max_splits;
  // at most 16 parts for the draft kernel, and for the target kernel when
  // workgroups of up to 4 waves cover at least 8 row groups (there the merge,
  // which re-reads every part, costs more than the longer splits)
  const int max_parts = draft || (VW <= 8 && groups >= 8) ? 16 : kMaxParts;
  if (ns > max_parts - 1) ns = max_parts - 1;
  if (ns < 1) ns = 1;
  p.nsplit = ns;
  p.chunk = 0;
  const size_t part_stride = D == 64 ? attn_part_bytes<64>(VW) : attn_part_bytes<128>(VW);
  p.part_bytes = (size_t)groups * (ns + 1) * part_stride;
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
  a.N = L.N;
  a.cache_parent = L.cache_parent;
  a.leaf_parent = L.leaf_parent;
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
  a.nsplit = L.nsplit;
  a.scale_log2 = L.scale * 1.4426950408889634f;
  const bool draft = L.N > 0 || L.leaf_parent != nullptr;
  if (!draft) {
    // target model: direct-to-LDS kernel, 32 rows per wave, partials in
    // 16-row virtual waves (2 per wave) for the merge kernel
    const int TPW = fast_attn_tiles(a.R, a.S_max - a.T, a.Hkv, a.nsplit);
    const int W = fast_attn_waves(a.R, a.S_max - a.T) * (2 / TPW);  // waves per workgroup
    a.RB = (a.R + 16 * TPW * W - 1) / (16 * TPW * W);
    const dim3 grid(L.Hkv * a.RB * (L.nsplit + 1));
#define SS_FAST(DD, WW, TT)                                                                          \
    hipLaunchKernelGGL((tree_attention_fast_kernel<DD, WW, TT>), grid, dim3(64 * WW), 0, st, a);         \
    launch_merge<DD, TT * WW>(a, st)
    if (L.D == 64) {
      if (W == 1) { SS_FAST(64, 1, 2); } else if (W == 2) { SS_FAST(64, 2, 2); } else if (W == 4) { SS_FAST(64, 4, 2); } else if (TPW == 1) { SS_FAST(64, 8, 1); } else { SS_FAST(64, 8, 2); }
    } else {
      if (W == 1) { SS_FAST(128, 1, 2); } else if (W == 2) { SS_FAST(128, 2, 2); } else if (W == 4) { SS_FAST(128, 4, 2); } else if (TPW == 1) { SS_FAST(128, 8, 1); } else { SS_FAST(128, 8, 2); }
    }
#undef SS_FAST
    return;
  }
  const int W = attn_waves(a.R);
  a.RB = (a.R + 16 * W - 1) / (16 * W);
  const dim3 grid(L.Hkv * a.RB * (L.nsplit + 1));
  if (W == 8) {
    if (L.D == 64) {
      hipLaunchKernelGGL((tree_attention_kernel<64, 8>), grid, dim3(512), 0, st, a);
      launch_merge<64, 8>(a, st);
    } else {
      hipLaunchKernelGGL((tree_attention_kernel<128, 8>), grid, dim3(512), 0, st, a);
      launch_merge<128, 8>(a, st);
    }
  } else {
    if (L.D == 64) {
      hipLaunchKernelGGL((tree_attention_kernel<64, 4>), grid, dim3(256), 0, st, a);
      launch_merge<64, 4>(a, st);
    } else {
      hipLaunchKernelGGL((tree_attention_kernel<128, 4>), grid, dim3(256), 0, st, a);
      launch_merge<128, 4>(a, st);
    }
  }
}

}  // namespace ss
