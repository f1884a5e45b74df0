// Host-side launch descriptors shared between the C-ABI layer and the
// kernel translation units.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace ss {

struct GemmLaunch {
  const void* w0;  // kernel-native (prepacked) weights
  const void* w1;  // up-projection of the fused SwiGLU
  int K, N;       // N = output columns
  const uint16_t* aprep;  // activations in the prepared layout
  int M;
  // non-null (plans with norm_in_kslice only): the input is RMSNorm(xnorm)
  // with weight gamma [K], computed in the GEMM; aprep is not read
  const uint16_t* xnorm = nullptr;
  int ldx = 0;
  const uint16_t* gamma = nullptr;
  float eps = 0.f;
  uint16_t* y;      // plain output (nullable)
  int ldy;
  uint16_t* yprep;  // prepared output for a following GEMM (nullable)
  const uint16_t* res;
  int ldr;
  int nw;       // N-tiles (16 columns) per block, counting gate and up tiles for SwiGLU
  int nblocks;  // column blocks
  int nwg;      // workgroups launched
  int ksw;      // > 0: one workgroup per column tile with ksw waves splitting K (no partials)
  bool swiglu;
  float* part;  // split-K partial slots (2 per workgroup)
};

// A K-split GEMM applies the RMSNorm of its input itself where no wave
// holds more than this many 128-wide groups (all its loads in registers).
constexpr int kNormMaxGroupsPerWave = 4;

struct GemmPlan {
  int nw, nblocks, nwg, ksw = 0;
  size_t part_bytes;  // split partials
  size_t prep_bytes;  // prepared activations of the input
};
GemmPlan plan_w4a16_gemm(int M, int K, int N, bool swiglu);
bool norm_in_kslice(const GemmPlan& p, int K);
void launch_w4a16_gemm(const GemmLaunch& L, hipStream_t st);
void launch_prepare_activations(const uint16_t* x, int M, int ldx, int K, uint16_t* out, hipStream_t st);
void launch_prepack_w4(const uint8_t* q, const uint16_t* s, const uint8_t* z, int K, int N, void* packed,
                       hipStream_t st);
inline size_t w4_packed_bytes(int K, int N) { return (size_t)K * N / 2 + (size_t)N * (K / 128) * 4; }

// VALU dot-product variant of the W4A16 GEMM (no matrix cores): one wave
// per (16-column tile, K slice), fp32 partial sums per slice, summed in
// slice order by a second kernel that also adds the residual.
struct ValuGemmPlan {
  int ksplit, gslice;  // K slices and groups per slice
  size_t part_bytes;   // [ksplit][M][N] fp32
};
ValuGemmPlan plan_w4a16_gemm_valu(int M, int K, int N);
void launch_w4a16_gemm_valu(const void* packed, int K, int N, const uint16_t* aprep, int M, uint16_t* y,
                            int ldy, const uint16_t* res, int ldr, float* part, const ValuGemmPlan& p,
                            hipStream_t st);

struct AttnLaunch {
  const uint16_t* q;
  int ldq;
  const uint16_t* k;
  const uint16_t* v;
  int ldkv;
  uint16_t* k_cache;
  uint16_t* v_cache;
  int S_max;
  const int32_t* prefix_len;
  const int32_t* parent;
  int T, Hq, Hkv, D;
  // draft model: N tree-cache rows after the prefix (forest cache_parent),
  // the T new tokens are leaves below leaf_parent[i]; target: 0, NULL, NULL
  int N = 0;
  const int32_t* cache_parent = nullptr;
  const int32_t* leaf_parent = nullptr;
  const float* rope;
  float scale;
  uint16_t* out;
  int ldo;
  uint16_t* out_prep;  // attention output also in the prepared layout (nullable)
  void* ws;         // header (error word, counters)
  float* part;      // split partials
  int nsplit;       // key splits per kv head
  int chunk;        // prefix keys per split (multiple of the key tile)
};
struct AttnPlan {
  int nsplit, chunk;
  size_t part_bytes;
};
// draft: the draft model's kernel (non-square mask); else the target kernel
AttnPlan plan_tree_attention(int T, int Hq, int Hkv, int D, int S_max, bool draft);
void launch_tree_attention(const AttnLaunch& L, hipStream_t st);

void launch_rmsnorm(const uint16_t* x, int M, int H, int ldx, const uint16_t* gamma, float eps,
                    uint16_t* out, int ldo, uint16_t* out_prep, hipStream_t st);

void launch_kv_commit(uint16_t* k_cache, uint16_t* v_cache, int n_layers, int64_t layer_stride,
                      int Hkv, int S_max, int D, int32_t* prefix_len, const int32_t* parent, int T,
                      const int32_t* accepted, int advance, void* ws, hipStream_t st);

void launch_tree_masks(const int32_t* parents, int n_trees, int T, uint64_t* anc, int32_t* depth,
                       int32_t* status, hipStream_t st);

void launch_clock_sample(uint64_t* out, uint32_t ticks, hipStream_t st);
void launch_ws_init(void* ws, size_t bytes, hipStream_t st);

void launch_kv_reorganize(uint16_t* k_cache, uint16_t* v_cache, int n_layers, int64_t layer_stride, int Hkv,
                          int S_max, int D, int32_t* prefix_len, const int32_t* parent, int N, const int32_t* d_last,
                          const int32_t* d_keep, int32_t* new_parent, int32_t* n_kept, int advance, void* ws,
                          hipStream_t st);
int greedy_accept_splits(int T);
int topk_logprobs_splits(int n);
size_t topk_logprobs_part_bytes(int n);
void launch_topk_logprobs(const uint16_t* logits, int ldl, int n, int V, int k, int32_t* tokens, float* logprobs,
                          void* ws, void* part, hipStream_t st);  // workgroups per logits row
void launch_greedy_accept(const uint16_t* logits, int ldl, int T, int V, const int32_t* tokens,
                          const int32_t* parent, int32_t* argmax, int32_t* accepted, int32_t* bonus,
                          int32_t* path_len, void* ws, void* part, hipStream_t st);
void launch_lm_head(const uint16_t* xn, int M, int H, const uint16_t* W, int V, uint16_t* logits, int ldl,
                    hipStream_t st);

}  // namespace ss
