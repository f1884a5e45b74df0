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
constexpr int kMaxParts = 16;  // prefix splits + tree split, merged in one pass

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

// Merge of the S + 1 <= 16 partials of one 16-row x 16-column output tile,
// in split order: with L_s the log-sum-exp of a row in split s and O_s its
// normalised output, O = sum_s 2^(L_s - L) O_s, L = log2 sum_s 2^L_s (taken
// relative to max_s L_s).  One wave per tile (lane: rows 4 (lane / 16) + r,
// column lane % 16); every split's loads are issued at once, so the kernel
// is one memory round trip long.  Grid = Hkv x RB x W x D/16.  A row that no
// split saw (only when the attention kernel rejected the tree or the prefix
// and published empty partials) is not written.
template <int D, int W>
__global__ __launch_bounds__(64) void tree_attention_merge_kernel(AttnArgs a) {
  constexpr int DT = D / 16;
  const int lane = lane_id();
  const int n16 = lane & 15, kq = lane >> 4;
  const int dt = blockIdx.x % DT;
  const int wave = (blockIdx.x / DT) % W;
  const int grp = blockIdx.x / (DT * W);  // g * RB + rb
  const int g = grp / a.RB, rb = grp % a.RB;
  const int nparts = a.nsplit + 1;
  const size_t part_stride = attn_part_bytes<D>(W);
  const char* base = reinterpret_cast<const char*>(a.part) + (size_t)grp * nparts * part_stride;
  f32x4 ls[kMaxParts];
  u32x2 ov[kMaxParts];
#pragma unroll
  for (int j = 0; j < kMaxParts; ++j) {
    const char* src = base + (size_t)(j < nparts ? j : nparts - 1) * part_stride;
    ls[j] = *reinterpret_cast<const f32x4*>(src + (size_t)W * DT * kWave * 8 + (wave * 16 + 4 * kq) * 4);
    ov[j] = *reinterpret_cast<const u32x2*>(src + ((size_t)(wave * DT + dt) * kWave + lane) * 8);
  }
  float lmax[4] = {-INFINITY, -INFINITY, -INFINITY, -INFINITY};
#pragma unroll
  for (int j = 0; j < kMaxParts; ++j)
#pragma unroll
    for (int r = 0; r < 4; ++r)
      if (j < nparts) lmax[r] = fmaxf(lmax[r], ls[j][r]);
  float wsum[4] = {0.f, 0.f, 0.f, 0.f}, acc[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int j = 0; j < kMaxParts; ++j)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const float w = (j < nparts && ls[j][r] != -INFINITY) ? exp2f(ls[j][r] - lmax[r]) : 0.f;
      wsum[r] += w;
      acc[r] += w * h2f((uint16_t)(ov[j][r >> 1] >> (16 * (r & 1))));
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

static int attn_waves(int R) { return R >= 128 ? 8 : 4; }

AttnPlan plan_tree_attention(int T, int Hq, int Hkv, int D, int S_max) {
  AttnPlan p;
  const int G = Hq / Hkv;
  const int R = T * G;
  const int W = attn_waves(R);
  const int RB = (R + 16 * W - 1) / (16 * W);
  const int groups = Hkv * RB;
  // about 256 workgroups in flight, at least two key tiles per prefix split
  // (four: no change at the 70B shapes, 2 us slower at prefixes of 500-1000
  // keys with few KV heads; one: slower at 1000 keys)
  int ns = 256 / groups - 1;
  const int max_tiles = (S_max - T + kKeyTile - 1) / kKeyTile;
  if (ns > max_tiles / 2) ns = max_tiles / 2;
  if (ns > kMaxParts - 1) ns = kMaxParts - 1;
  if (ns < 1) ns = 1;
  p.nsplit = ns;
  p.chunk = 0;
  const size_t part_stride = D == 64 ? attn_part_bytes<64>(W) : attn_part_bytes<128>(W);
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
  const int W = attn_waves(a.R);
  a.RB = (a.R + 16 * W - 1) / (16 * W);
  a.nsplit = L.nsplit;
  a.scale_log2 = L.scale * 1.4426950408889634f;
  const dim3 grid(L.Hkv * a.RB * (L.nsplit + 1));
  const dim3 mgrid(L.Hkv * a.RB * W * (L.D / 16));
  if (W == 8) {
    if (L.D == 64) {
      hipLaunchKernelGGL((tree_attention_kernel<64, 8>), grid, dim3(512), 0, st, a);
      hipLaunchKernelGGL((tree_attention_merge_kernel<64, 8>), mgrid, dim3(64), 0, st, a);
    } else {
      hipLaunchKernelGGL((tree_attention_kernel<128, 8>), grid, dim3(512), 0, st, a);
      hipLaunchKernelGGL((tree_attention_merge_kernel<128, 8>), mgrid, dim3(64), 0, st, a);
    }
  } else {
    if (L.D == 64) {
      hipLaunchKernelGGL((tree_attention_kernel<64, 4>), grid, dim3(256), 0, st, a);
      hipLaunchKernelGGL((tree_attention_merge_kernel<64, 4>), mgrid, dim3(64), 0, st, a);
    } else {
      hipLaunchKernelGGL((tree_attention_kernel<128, 4>), grid, dim3(256), 0, st, a);
      hipLaunchKernelGGL((tree_attention_merge_kernel<128, 4>), mgrid, dim3(64), 0, st, a);
    }
  }
}

}  // namespace ss
