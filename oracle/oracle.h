/*
 * fp64 reference checker for the tree-verification step (TEST INFRASTRUCTURE).
 *
 * Only the test-suite, the smoke check and the benchmark's CPU-baseline leg
 * may load this library.  The product path (the HIP library and its Python
 * binding) never calls it and shares no code with it.
 *
 * Everything is computed in double precision with plain loops, following
 * the definitions in the paper (SwiftSpec, arXiv 2506.11309):
 *   - target-side tree mask: a draft token attends to the whole prefix and,
 *     inside the tree, only to itself and its ancestors (Sec. 3.1, paragraph
 *     on non-square masks; square mask for the target model);
 *   - rotary position embedding fused into attention, position id from the
 *     node depth (Sec. 3.3, masked attention; Sec. 4 tree bookkeeping);
 *   - int4 AWQ-style weights, group size 128, 16-bit compute (Sec. 5.1);
 *   - SwiGLU MLP (Sec. 3.3, fused SwiGLU);
 *   - verified tokens moved into the contiguous prefix of the KV cache
 *     (Sec. 3.2 and Fig. 5 caption), the verified path starting at the
 *     current tree root (Sec. 3.1, Fig. 3 walk-through).
 *
 * fp16 values cross the interface as uint16 IEEE binary16 bit patterns.
 * fp16 rounding (round to nearest, ties to even) happens only at the
 * storage points of a decoder layer: normalised input, projection outputs,
 * rotated keys and values written to the cache, attention output, residual
 * sums and the SwiGLU product.  All arithmetic between them is fp64.
 *
 * All pointers are host pointers.  Functions returning int return 0 on
 * success and a negative value on invalid arguments or an invalid tree.
 */
#ifndef SWIFTSPEC_ORACLE_H
#define SWIFTSPEC_ORACLE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* binary16 <-> double */
double oracle_f16_to_f64(uint16_t h);
uint16_t oracle_f64_to_f16(double x);

/* Tree bookkeeping.  parent[0] = -1 and 0 <= parent[i] < i.
 * depth[i] = number of edges from the root; anc[i*T + j] = 1 iff j == i or
 * j is an ancestor of i.  Returns 0, or -1 for an invalid parent array. */
int oracle_tree(const int32_t* parent, int32_t T, int32_t* depth, uint8_t* anc);

/* W'[n][k] = (q[n][k] - z[n][k/128]) * s[n][k/128]; q packed two per byte,
 * low nibble = even k.  Returns the exact dequantised value. */
double oracle_dequant(const uint8_t* qweight, const uint16_t* scales, const uint8_t* zeros,
                      int32_t K, int32_t n, int32_t k);

/* y[m][n] = fp16( sum_k x[m][k] * W'[n][k]  (+ residual[m][n]) ). */
int oracle_w4a16_gemm(const uint8_t* qweight, const uint16_t* scales, const uint8_t* zeros,
                      int32_t K, int32_t N, const uint16_t* x, int32_t M, int32_t ldx,
                      const uint16_t* residual, int32_t ldr, uint16_t* y, int32_t ldy);

/* y[m][n] = fp16( silu(g) * u ),  g = x.Wg'^T, u = x.Wu'^T (fp64). */
int oracle_w4a16_swiglu(const uint8_t* qg, const uint16_t* sg, const uint8_t* zg,
                        const uint8_t* qu, const uint16_t* su, const uint8_t* zu, int32_t K,
                        int32_t N, const uint16_t* x, int32_t M, int32_t ldx, uint16_t* y,
                        int32_t ldy);

/* out[m][:] = fp16( x[m][:] / sqrt(mean(x[m][:]^2) + eps) * gamma ). */
int oracle_rmsnorm(const uint16_t* x, int32_t M, int32_t H, int32_t ldx, const uint16_t* gamma,
                   double eps, uint16_t* out, int32_t ldo);

/* Rotary embedding of one head vector (rotate-half pairs (d, d + D/2)),
 * angle pos * theta^(-2d/D), in place, fp64. */
void oracle_rope(double* vec, int32_t D, int64_t pos, double theta);

/* Tree-masked GQA attention of T draft tokens over the cache.
 * q [T][ldq] (Hq*D used), k, v [T][ldkv] (Hkv*D used), pre-rotation.
 * Caches [Hkv][S_max][D]; rows [P, P+T) receive fp16(rope(k)) and v.
 * out [T][ldo] (Hq*D used) = fp16(attention).  Query head h reads kv head
 * h / (Hq/Hkv).  Returns 0 or -1. */
int oracle_tree_attention(const uint16_t* q, int32_t ldq, const uint16_t* k, const uint16_t* v,
                          int32_t ldkv, uint16_t* k_cache, uint16_t* v_cache, int32_t S_max,
                          int32_t P, const int32_t* parent, int32_t T, int32_t Hq, int32_t Hkv,
                          int32_t D, double rope_theta, double softmax_scale, uint16_t* out,
                          int32_t ldo);

/* Commit the accepted root-to-node path: with path pi_0 = 0, ..., pi_{L-1} =
 * accepted, row P+i <- row P+pi_i (from a snapshot) for i < L, in every layer
 * and for K and V; other rows unchanged.  Layer l's caches start at
 * k_cache + l*layer_stride.  Returns L, or -1. */
int32_t oracle_kv_commit(uint16_t* k_cache, uint16_t* v_cache, int32_t n_layers,
                         int64_t layer_stride, int32_t Hkv, int32_t S_max, int32_t D, int32_t P,
                         const int32_t* parent, int32_t T, int32_t accepted);

/* Draft-model attention with a non-square mask (Sec. 3.1, paragraph on
 * non-square masks; Fig. 4): the draft model expands w leaves of its tree.
 * Cache rows [0, P) hold the verified prefix, rows [P, P+N) the draft tree
 * cache (a forest: cache_parent[j] in [-1, j), -1 = below the last prefix
 * token), all already rotated.  New token i (a leaf below cache node
 * leaf_parent[i], -1 = below the last prefix token) sits at position
 * P + depth, where a cached node below the last prefix token has depth 0
 * and a new token one more than its parent (so position P if its parent is
 * -1).  Its key, rotated at that position and rounded to fp16, and its
 * value enter rows P + N + i.  It attends to the whole prefix, to the cached
 * nodes on its parent's root path (parent included) and to itself: a
 * w x (N + w) mask over the tree region.  Returns 0 or -1. */
int oracle_draft_tree_attention(const uint16_t* q, int32_t ldq, const uint16_t* k, const uint16_t* v,
                                int32_t ldkv, uint16_t* k_cache, uint16_t* v_cache, int32_t S_max, int32_t P,
                                const int32_t* cache_parent, int32_t N, const int32_t* leaf_parent, int32_t w,
                                int32_t Hq, int32_t Hkv, int32_t D, double rope_theta, double softmax_scale,
                                uint16_t* out, int32_t ldo);

/* Draft-side KV reorganisation after re-rooting (Sec. 3.2, consistency
 * management of the draft model's cache; Fig. 5).  Rows [P, P+N) of every
 * cache hold a forest of draft nodes: parent[i] in [-1, i), -1 = a child of
 * the last prefix token.  last = the deepest forest node on the newly
 * verified path (-1: none).  path = the forest root ... last (L nodes, L = 0
 * if last = -1); kept = the nodes below last in index order (S nodes; none
 * unless keep).  Rows P + i take the old rows of (path ++ kept)[i]; other
 * rows are unchanged.  new_parent[j] (j < S) = position in kept of kept[j]'s
 * parent, or -1 if that parent is last.  Returns L (the prefix grows by L),
 * *n_kept = S; -1 for invalid arguments or forest. */
int32_t oracle_kv_reorganize(uint16_t* k_cache, uint16_t* v_cache, int32_t n_layers, int64_t layer_stride,
                             int32_t Hkv, int32_t S_max, int32_t D, int32_t P, const int32_t* parent,
                             int32_t N, int32_t last, int32_t keep, int32_t* new_parent, int32_t* n_kept);

/* Greedy acceptance of a verified tree (target-side verification with the
 * target's greedy choice; Sec. 3.1, Fig. 3 walk-through).  logits [T][ldl]
 * fp16: row i is the target's distribution after the path root -> node i.
 * argmax[i] = first index of the largest logit of row i.  From the root,
 * repeatedly step to the lowest-index child c with tokens[c] == argmax of
 * the current node; the node where no child matches is *accepted and its
 * argmax is the *bonus token.  tokens[0] (the root's own token) is not
 * used.  Returns L = depth(accepted) + 1 (accepted path length, root
 * included), or -1 for invalid arguments or tree. */
int32_t oracle_greedy_accept(const uint16_t* logits, int32_t T, int32_t V, int32_t ldl,
                             const int32_t* tokens, const int32_t* parent, int32_t* argmax,
                             int32_t* accepted, int32_t* bonus);

typedef struct {
  int32_t H, Hq, Hkv, D, F, S_max;
  double eps, rope_theta;
} oracle_dims;

typedef struct {
  const uint8_t* q;
  const uint16_t* s;
  const uint8_t* z;
} oracle_w4;

/* One Llama decoder layer over the draft tree:
 *   xn = fp16(rmsnorm(x, attn_norm))        qkv = fp16(xn . Wqkv'^T)
 *   o  = fp16(tree_attention(qkv))          h   = fp16(x + o . Wo'^T)
 *   hn = fp16(rmsnorm(h, mlp_norm))         m   = fp16(silu(hn.Wg'^T) * (hn.Wu'^T))
 *   out = fp16(h + m . Wd'^T)
 * hidden [T][H] is read as x and overwritten with out.  The caches receive
 * the tree's keys and values at rows [P, P+T).  Returns 0 or -1. */
int oracle_verify_layer(const oracle_dims* dims, const uint16_t* attn_norm,
                        const uint16_t* mlp_norm, oracle_w4 wqkv, oracle_w4 wo, oracle_w4 wgate,
                        oracle_w4 wup, oracle_w4 wdown, uint16_t* k_cache, uint16_t* v_cache,
                        uint16_t* hidden, int32_t T, int32_t P, const int32_t* parent);

/* logits[m][v] = fp16( rmsnorm(h[m], gamma) . W[v] ),  W [V][H] fp16. */
int oracle_lm_head(const uint16_t* h, int32_t M, int32_t H, const uint16_t* gamma, double eps,
                   const uint16_t* W, int32_t V, uint16_t* logits);

/* Draft-tree expansion (Sec. 3.1, maximum-likelihood expansion): for each
 * of n logits rows [V] fp16 (stride ldl), the k tokens of largest logit
 * (equal logits: lower index first) and their log-softmax values.  O(k V)
 * per row.  Returns 0 or -1. */
int32_t oracle_topk_logprobs(const uint16_t* logits, int32_t n, int32_t V, int32_t ldl, int32_t k,
                             int32_t* tokens, double* logprobs);

int oracle_num_threads(void);
void oracle_set_num_threads(int n);

#ifdef __cplusplus
}
#endif
#endif
