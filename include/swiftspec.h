/*
 * swiftspec -- tree-verification forward step for speculative decoding on
 * AMD Instinct MI355X (gfx950).  C ABI of libswiftspec.so.
 *
 * The operations follow SwiftSpec (arXiv 2506.11309):
 *   - the target model verifies a draft token tree by one batched forward
 *     pass (Algorithm 1, target-worker branch; Sec. 3.1);
 *   - inside the tree a token attends only to itself and its ancestors, and
 *     to the whole verified prefix (Sec. 3.1, paragraph on non-square masks,
 *     square mask of the target model);
 *   - rotary position embedding is fused into attention, a token's position
 *     being prefix length + its depth in the tree (Sec. 3.3, masked
 *     attention; Sec. 4, tree bookkeeping by depth and ancestor list);
 *   - weights are int4 AWQ-style with group size 128, compute is 16-bit
 *     (Sec. 5.1);
 *   - the MLP is a fused SwiGLU (Sec. 3.3, fused SwiGLU);
 *   - after verification the KV states of the verified tokens are kept as a
 *     contiguous prefix of the cache, the tree region following it
 *     (Sec. 3.2 and the caption of Fig. 5); the verified path begins at the
 *     current tree root (Sec. 3.1, walk-through of Fig. 3).
 *
 * Conventions
 *   - fp16 tensors are passed as uint16_t IEEE binary16 bit patterns.
 *   - Unless stated otherwise every tensor pointer is DEVICE memory owned by
 *     the caller (e.g. allocated by PyTorch).  The library never allocates
 *     device memory and never frees caller memory.
 *   - Row-major layouts; leading dimensions (ld*) are in elements.  Device
 *     tensors and leading dimensions must keep 16-byte alignment of every
 *     row (ld % 8 == 0 for fp16) unless stated otherwise.
 *   - Work is enqueued on `stream` (a hipStream_t passed as void*; NULL is
 *     the null stream).  No call synchronises the stream or reads device
 *     data on the host, so every compute call can be captured into a HIP
 *     graph.  Host-side argument checks happen before any launch; on error
 *     nothing is launched.
 *   - Scratch memory is a caller-provided device workspace whose size comes
 *     from the matching *_workspace_bytes query.  The first
 *     SWIFTSPEC_WS_HEADER_BYTES bytes of every workspace hold an error word
 *     and ticket counters that must be zero before first use (allocate it
 *     zero-filled or call swiftspec_workspace_init once); every call leaves
 *     them zero again.  Calls sharing one workspace must not overlap in
 *     time (use one stream per workspace).
 *   - Per-step data that lives in device memory (prefix length, parent
 *     array, accepted node) is validated on the device: an invalid value
 *     sets a bit of the workspace error word (swiftspec_read_device_error)
 *     and the affected kernels skip their writes; they never access memory
 *     out of bounds.
 *   - Thread safety: calls are stateless apart from a thread-local record of
 *     the last HIP error.
 */
#ifndef SWIFTSPEC_H
#define SWIFTSPEC_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* ---------------------------------------------------------------- status */
enum {
  SWIFTSPEC_OK = 0,
  SWIFTSPEC_INVALID_ARG = 1,         /* null pointer, bad dimension, bad leading dimension */
  SWIFTSPEC_UNSUPPORTED = 2,         /* D not 64/128, T > 64, K % 128, M > 64, Hq % Hkv ... */
  SWIFTSPEC_MISALIGNED = 3,          /* pointer or leading dimension breaks 16-byte alignment */
  SWIFTSPEC_WORKSPACE_TOO_SMALL = 4, /* ws_bytes below the *_workspace_bytes figure */
  SWIFTSPEC_BAD_TREE = 5,            /* host-side tree validation failed */
  SWIFTSPEC_HIP_ERROR = 6,           /* a HIP runtime call failed; see swiftspec_last_hip_error */
  SWIFTSPEC_CAPACITY = 7             /* a host-side draft tree would exceed its node capacity */
};

/* bits of the device error word */
#define SWIFTSPEC_DEVERR_BAD_TREE 1u     /* parent[0] != -1 or parent[i] outside [0, i) */
#define SWIFTSPEC_DEVERR_BAD_PREFIX 2u   /* prefix length < 0 or prefix + T > S_max */
#define SWIFTSPEC_DEVERR_BAD_ACCEPTED 4u /* accepted node outside [0, T) */

#define SWIFTSPEC_WS_HEADER_BYTES 65536u
#define SWIFTSPEC_MAX_TREE 64 /* one 64-lane wavefront builds the ancestor masks */
#define SWIFTSPEC_MAX_M 64    /* GEMM rows (tree tokens) per call */

const char* swiftspec_status_string(int status);
/* hipError_t of the last failing HIP call on this thread (0 if none). */
int swiftspec_last_hip_error(void);
/* Zero the workspace header on `stream` (a fill kernel, no memset). */
int swiftspec_workspace_init(void* ws, size_t ws_bytes, void* stream);
/* Synchronise `stream`, copy the error word to *out (host), then clear it. */
int swiftspec_read_device_error(void* ws, void* stream, uint32_t* out);

/* ------------------------------------------------------- int4 weights
 * AWQ-style int4 matrix W (N output rows x K inputs), group size 128
 * (Sec. 5.1).  Dequantised value W'[n][k] = (q[n][k] - z[n][k/128]) * s[n][k/128].
 *   qweight: [N][K/2] bytes, byte b of row n holds k = 2b (low nibble) and
 *            k = 2b + 1 (high nibble), values 0..15;
 *   scales : [N][K/128] fp16;
 *   zeros  : [N][K/128] uint8, values 0..15;
 *   packed : kernel-native copy of the same matrix written once by
 *            swiftspec_w4_prepack (swiftspec_w4_packed_bytes(K, N) bytes,
 *            16-byte aligned, device memory owned by the caller).  It holds
 *            the same nibbles regrouped so that every 16x128 (column x k)
 *            block is one contiguous kilobyte, followed by one 32-bit word
 *            (scale | zero << 16) per (column, group).  The compute entry
 *            points read only `packed`; qweight/scales/zeros are needed only
 *            by swiftspec_w4_prepack.
 * K % 128 == 0, N % 64 == 0 (four waves of 16 output columns), and the
 * kernel-native copy below 4 GiB (swiftspec_w4_packed_bytes(K, N) <= 2^32 - 1;
 * UNSUPPORTED otherwise). */
typedef struct {
  const uint8_t* qweight;
  const uint16_t* scales;
  const uint8_t* zeros;
  int32_t K, N;
  const void* packed;
} swiftspec_w4;

size_t swiftspec_w4_packed_bytes(int32_t K, int32_t N);
/* Write the kernel-native copy of W (qweight, scales, zeros) into `packed`
 * on `stream`.  A pure rearrangement of the same bits. */
int swiftspec_w4_prepack(const swiftspec_w4* W, void* packed, size_t packed_bytes, void* stream);

/* y[m][n] = fp16( sum_k x[m][k] * W'[n][k] + residual[m][n] ), fp32
 * accumulation, for m < M (1 <= M <= 64).  residual may be NULL; it may
 * alias y only if ldr == ldy.  x [M][ldx], y [M][ldy], residual [M][ldr].
 * The weight projections of a decoder layer at GEMM M = tree size
 * (Sec. 3.3; QKV, O, down projections). */
int swiftspec_w4a16_gemm(const swiftspec_w4* W, const uint16_t* x, int32_t M, int32_t ldx,
                         uint16_t* y, int32_t ldy, const uint16_t* residual, int32_t ldr,
                         void* ws, size_t ws_bytes, void* stream);
size_t swiftspec_w4a16_gemm_workspace_bytes(int32_t M, int32_t K, int32_t N);

/* Fused SwiGLU (Sec. 3.3): y[m][n] = fp16( silu(g) * u ), g = x.Wg'^T,
 * u = x.Wu'^T (fp32), silu(g) = g / (1 + exp(-g)).  Wg and Wu share K, N. */
int swiftspec_w4a16_swiglu(const swiftspec_w4* Wg, const swiftspec_w4* Wu, const uint16_t* x,
                           int32_t M, int32_t ldx, uint16_t* y, int32_t ldy, void* ws,
                           size_t ws_bytes, void* stream);
size_t swiftspec_w4a16_swiglu_workspace_bytes(int32_t M, int32_t K, int32_t N);

/* The same product as swiftspec_w4a16_gemm computed on the vector ALUs
 * only (v_dot2_f32_f16, no matrix cores): the comparison point for the
 * matrix-core kernel at M = tree size (Sec. 3.3, Sec. 5.1).  Same arguments,
 * constraints and result tolerance; fp32 partial sums per K slice are added
 * in slice order (deterministic).  Workspace from
 * swiftspec_w4a16_gemm_valu_workspace_bytes. */
int swiftspec_w4a16_gemm_valu(const swiftspec_w4* W, const uint16_t* x, int32_t M, int32_t ldx,
                              uint16_t* y, int32_t ldy, const uint16_t* residual, int32_t ldr,
                              void* ws, size_t ws_bytes, void* stream);
size_t swiftspec_w4a16_gemm_valu_workspace_bytes(int32_t M, int32_t K, int32_t N);

/* Activations in the matrix-core operand order the GEMMs read
 * ("prepared" layout: [ceil(M/16)][K/128][4][64][8] fp16, rows >= M zero,
 * values as given).  Chained GEMMs can keep
 * activations in this form and call the *_prepared entry points. */
size_t swiftspec_prepared_bytes(int32_t M, int32_t K);
int swiftspec_prepare_activations(const uint16_t* x, int32_t M, int32_t ldx, int32_t K, uint16_t* xp,
                                  void* stream);
/* As swiftspec_w4a16_gemm / swiftspec_w4a16_swiglu with prepared activations xp. */
int swiftspec_w4a16_gemm_prepared(const swiftspec_w4* W, const uint16_t* xp, int32_t M, uint16_t* y,
                                  int32_t ldy, const uint16_t* residual, int32_t ldr, void* ws,
                                  size_t ws_bytes, void* stream);
int swiftspec_w4a16_swiglu_prepared(const swiftspec_w4* Wg, const swiftspec_w4* Wu, const uint16_t* xp,
                                    int32_t M, uint16_t* y, int32_t ldy, void* ws, size_t ws_bytes,
                                    void* stream);

/* out[m][:] = fp16( x[m][:] / sqrt(mean(x[m][:]^2) + eps) * gamma ), M rows of H
 * (the RMSNorm in front of the attention and MLP blocks, and the final norm).
 * H % 32 == 0 (UNSUPPORTED otherwise); pointers 16-byte aligned, ldx and
 * ldo multiples of 8. */
int swiftspec_rmsnorm(const uint16_t* x, int32_t M, int32_t H, int32_t ldx, const uint16_t* gamma,
                      float eps, uint16_t* out, int32_t ldo, void* stream);

/* RMSNorm followed by a projection: the QKV projection of the attention
 * block and the fused SwiGLU of the MLP block read the normalised residual
 * stream (Sec. 2's decoder layer):
 *   swiftspec_rmsnorm_w4a16_gemm  : y = fp16( xn . W'^T )
 *   swiftspec_rmsnorm_w4a16_swiglu: y = fp16( silu(xn . Wg'^T) * (xn . Wu'^T) )
 * with xn[m] = x[m] / sqrt(mean_k x[m][k]^2 + eps) * gamma over the K
 * columns, xn rounded to fp16 (as swiftspec_rmsnorm computes it) and then
 * multiplied.  Where the GEMM's plan gives each workgroup all of K and each
 * of its waves at most 4 groups of 128 (up to 16 rows, SwiGLU up to 8;
 * matrices of at most 32 MB) the norm runs inside the GEMM, which sums the
 * rows' squares first and forms the fp16 operand values the same way;
 * otherwise the norm kernel writes them for the GEMM.  x [M][ldx], gamma [K]
 * fp16, 16-byte aligned, ldx % 8 == 0; no residual; the workspace of
 * swiftspec_w4a16_gemm_workspace_bytes / _swiglu_workspace_bytes.  Other
 * arguments and errors as swiftspec_w4a16_gemm / _swiglu. */
int swiftspec_rmsnorm_w4a16_gemm(const swiftspec_w4* W, const uint16_t* x, int32_t M, int32_t ldx,
                                 const uint16_t* gamma, float eps, uint16_t* y, int32_t ldy, void* ws,
                                 size_t ws_bytes, void* stream);
int swiftspec_rmsnorm_w4a16_swiglu(const swiftspec_w4* Wg, const swiftspec_w4* Wu, const uint16_t* x,
                                   int32_t M, int32_t ldx, const uint16_t* gamma, float eps, uint16_t* y,
                                   int32_t ldy, void* ws, size_t ws_bytes, void* stream);

/* ------------------------------------------------------- tree attention
 * Tree-masked grouped-query attention of the T draft tokens over the KV
 * cache (Sec. 3.1 target-side square mask; Sec. 3.3 masked attention with
 * the position embedding fused in).
 *   q       : [T][ldq]  query heads h = 0..Hq-1 at columns [h*D, (h+1)*D), before RoPE
 *   k, v    : [T][ldkv] kv heads at columns [g*D, (g+1)*D), k before RoPE
 *   k_cache, v_cache : [Hkv][S_max][D]; rows [0, P) hold the verified prefix
 *             (already rotated); rows [P, P+T) RECEIVE fp16(rope(k)) and v.
 *   d_prefix_len : device int32, P
 *   d_parent : device int32[T], parent[0] = -1, 0 <= parent[i] < i
 *   rope_cos_sin : device fp32 [S_max][D/2][2] (cos, sin) of pos * theta^(-2d/D),
 *             see swiftspec_rope_table; rotation pairs (d, d + D/2)
 *   out     : [T][ldo] fp16, query head h at columns [h*D, (h+1)*D)
 * Node i at position P + depth(i) attends to cache rows [0, P) and to the
 * tree rows P + j of its ancestors-or-self j; query head h reads kv head
 * h / (Hq / Hkv).  1 <= T <= 64, D in {64, 128}, Hq % Hkv == 0,
 * softmax_scale > 0 and finite (SWIFTSPEC_INVALID_ARG otherwise); q, k, v
 * and the cache rows read must be finite (NaN or infinite entries give
 * undefined results, not an error).  An invalid
 * tree or prefix length sets the device error word; then out and the cache
 * are left untouched. */
int swiftspec_tree_attention(const uint16_t* q, int32_t ldq, const uint16_t* k, const uint16_t* v,
                             int32_t ldkv, uint16_t* k_cache, uint16_t* v_cache, int32_t S_max,
                             const int32_t* d_prefix_len, const int32_t* d_parent, int32_t T,
                             int32_t Hq, int32_t Hkv, int32_t D, const float* rope_cos_sin,
                             float softmax_scale, uint16_t* out, int32_t ldo, void* ws,
                             size_t ws_bytes, void* stream);
/* Tree attention that allocates nothing, for callers that cannot allocate
 * device memory or hand over a workspace (work under HIP graph capture,
 * tight serving loops, harnesses that forbid allocation).  Same arguments
 * and results as swiftspec_tree_attention, without ws / ws_bytes: the split
 * partials live in a library-owned device array of
 * SWIFTSPEC_NOALLOC_SCRATCH_BYTES on each GPU the library runs on, held
 * until the process ends; nothing in it needs to start at zero.  d_error
 * (device uint32, nullable) receives the device error bits
 * (SWIFTSPEC_DEVERR_*, OR-ed in; the caller clears it).  A shape whose
 * partials do not fit returns SWIFTSPEC_WORKSPACE_TOO_SMALL before any
 * launch (the Llama-3 1B/8B/70B shapes at T <= 64 need at most 17.2 MB).
 * The first call on a device looks up the array's device address
 * (SWIFTSPEC_HIP_ERROR if that fails).  No call allocates or frees memory.
 * Every call on one GPU shares its array: calls that overlap in time on one
 * GPU (several streams or threads) race, and their results are undefined. */
#define SWIFTSPEC_NOALLOC_SCRATCH_BYTES (32u << 20)
int swiftspec_tree_attention_noalloc(const uint16_t* q, int32_t ldq, const uint16_t* k, const uint16_t* v,
                                     int32_t ldkv, uint16_t* k_cache, uint16_t* v_cache, int32_t S_max,
                                     const int32_t* d_prefix_len, const int32_t* d_parent, int32_t T,
                                     int32_t Hq, int32_t Hkv, int32_t D, const float* rope_cos_sin,
                                     float softmax_scale, uint16_t* out, int32_t ldo, uint32_t* d_error,
                                     void* stream);
size_t swiftspec_tree_attention_workspace_bytes(int32_t T, int32_t Hq, int32_t Hkv, int32_t D,
                                                int32_t S_max);

/* Host helper: (cos, sin) table [S_max][D/2][2] of angle pos * theta^(-2d/D),
 * evaluated in fp64 and rounded to fp32, into host memory. */
int swiftspec_rope_table(double theta, int32_t S_max, int32_t D, float* host_out);

/* Device ancestor masks: for each of n_trees parent arrays ([n_trees][T],
 * device), anc[t][i] bit j set iff j is i or an ancestor of i; depth[t][i];
 * status[t] = 0 (valid) or SWIFTSPEC_DEVERR_BAD_TREE (then anc = self bit,
 * depth = 0).  The same wavefront routine the attention and commit kernels
 * use.  T <= 64. */
int swiftspec_tree_masks(const int32_t* d_parents, int32_t n_trees, int32_t T, uint64_t* d_anc,
                         int32_t* d_depth, int32_t* d_status, void* stream);

/* Host helper: validates a host parent array; fills depth_out (host, may be NULL). */
int swiftspec_tree_validate(const int32_t* parent_host, int32_t T, int32_t* depth_out);

/* ------------------------------------------------------------ KV commit
 * Moves the KV states of the accepted path into the contiguous prefix
 * (Sec. 3.2, Fig. 5 caption; target side).  With the accepted node a and its
 * root-to-node path pi_0 = 0, ..., pi_{L-1} = a (L = depth(a) + 1), for every
 * layer l < n_layers, for K and V and every kv head:
 *     row P + i  <-  row P + pi_i   (i < L, all sources read before any write)
 * rows [P+L, P+T) are left unchanged.  Layer l's caches start at
 * k_cache + l * layer_stride_elems.  If advance != 0 the device prefix
 * length becomes P + L after the copy (stream-ordered).  ws may be NULL
 * (then device errors are not reported); otherwise its header receives the
 * error word. */
int swiftspec_kv_commit(uint16_t* k_cache, uint16_t* v_cache, int32_t n_layers,
                        int64_t layer_stride_elems, int32_t Hkv, int32_t S_max, int32_t D,
                        int32_t* d_prefix_len, const int32_t* d_parent, int32_t T,
                        const int32_t* d_accepted_node, int32_t advance, void* ws,
                        size_t ws_bytes, void* stream);

/* Draft-model tree attention with a non-square mask (Sec. 3.1, paragraph
 * on non-square masks; Fig. 4): the draft model expands w leaves of its
 * tree.  Cache rows [0, P) hold the verified prefix (P = *d_prefix_len),
 * rows [P, P+N) the draft tree cache, already rotated: a forest,
 * d_cache_parent[N] with parent[j] in [-1, j) (-1: below the last prefix
 * token).  New token i (q, k, v rows i, layouts as in
 * swiftspec_tree_attention, k pre-rotation) is a leaf below cache node
 * d_leaf_parent[i] (-1: below the last prefix token) at position P + depth
 * (a cached node below the last prefix token has depth 0, a new token one
 * more than its parent).  Its rotated key (fp16) and its value are written
 * to rows P + N + i, and it attends to the whole prefix, to the cached
 * nodes on its parent's root path (parent included) and to itself: a
 * w x (N + w) mask over the tree region.  1 <= w <= 64, 0 <= N <= 64,
 * P + N + w <= S_max (else the device error word gets
 * SWIFTSPEC_DEVERR_BAD_PREFIX), other requirements and the workspace
 * (swiftspec_tree_attention_workspace_bytes(w, Hq, Hkv, D, S_max)) as for
 * swiftspec_tree_attention.  An invalid forest or leaf parent sets
 * SWIFTSPEC_DEVERR_BAD_TREE and leaves output and cache untouched. */
int swiftspec_draft_tree_attention(const uint16_t* q, int32_t ldq, const uint16_t* k, const uint16_t* v,
                                   int32_t ldkv, uint16_t* k_cache, uint16_t* v_cache, int32_t S_max,
                                   const int32_t* d_prefix_len, const int32_t* d_cache_parent, int32_t N,
                                   const int32_t* d_leaf_parent, int32_t w, int32_t Hq, int32_t Hkv, int32_t D,
                                   const float* rope_cos_sin, float softmax_scale, uint16_t* out, int32_t ldo,
                                   void* ws, size_t ws_bytes, void* stream);

/* Draft-side KV reorganisation after re-rooting (Sec. 3.2, consistency
 * management of the draft model's cache; Fig. 5).  Rows [P, P+N) of each
 * [Hkv][S_max][D] cache (layer l at k_cache + l * layer_stride_elems) hold
 * the draft tree cache: a forest, d_parent[N] with parent[i] in [-1, i)
 * (-1: a child of the last prefix token).  *d_last = the deepest forest node
 * on the newly verified token sequence, or -1 if the first verified token
 * is not in the forest.  Rows P .. P+L-1 take the verified path (the forest
 * root above last, ..., last; L = 0 if last = -1); if *d_keep != 0 the nodes
 * below last follow in index order (S of them, rows P+L .. P+L+S-1), else
 * S = 0; all other rows are unchanged.  d_new_parent (nullable, N entries)
 * receives, for j < S, the new tree-cache index of kept node j's parent, or
 * -1 if that parent is last (now the last prefix token); *d_n_kept
 * (nullable) = S.  If advance != 0, *d_prefix_len becomes P + L after the
 * copy (stream-ordered).  With *d_keep == 0 and a single-root tree this is
 * swiftspec_kv_commit.  1 <= N <= 64, D % 8 == 0, D <= 256, caches 16-byte
 * aligned.  d_new_parent must not overlap d_parent[0 .. N) (the old forest
 * is read while the new one is written): SWIFTSPEC_INVALID_ARG.  Invalid
 * device data (forest, last, prefix) sets the error word (ws may be NULL:
 * then it is not reported) and nothing is written. */
int swiftspec_kv_reorganize(uint16_t* k_cache, uint16_t* v_cache, int32_t n_layers, int64_t layer_stride_elems,
                            int32_t Hkv, int32_t S_max, int32_t D, int32_t* d_prefix_len, const int32_t* d_parent,
                            int32_t N, const int32_t* d_last, const int32_t* d_keep, int32_t* d_new_parent,
                            int32_t* d_n_kept, int32_t advance, void* ws, size_t ws_bytes, void* stream);

/* ------------------------------------------------ draft tree expansion
 * The children of the leaves a draft step expands (Sec. 3.1, maximum-
 * likelihood tree expansion: a node's value is the log-softmax probability
 * of its token): for each of n logits rows [V] fp16 (row i at
 * logits + i * ldl, device), the k tokens of largest logit (equal logits:
 * lower index first) into d_tokens[n][k] (int32, device) and their
 * log-softmax values, computed in fp32, into d_logprobs[n][k] (float,
 * device), in decreasing order.  Logits are expected to be finite.
 * 1 <= n <= 64, 1 <= k <= 8, k <= V, ldl >= V, ldl % 8 == 0, logits 16-byte
 * aligned.  ws: swiftspec_topk_logprobs_workspace_bytes(n) bytes (per-range
 * partial lists after the header; the header's counters are used and left
 * zero). */
size_t swiftspec_topk_logprobs_workspace_bytes(int32_t n);
int swiftspec_topk_logprobs(const uint16_t* logits, int32_t ldl, int32_t n, int32_t V, int32_t k,
                            int32_t* d_tokens, float* d_logprobs, void* ws, size_t ws_bytes, void* stream);

/* ------------------------------------------------- draft tree (host)
 * The draft worker's tree of parallel tree generation (Sec. 3.1, Alg. 1;
 * re-rooting and the draft cache per Sec. 3.2 and Fig. 5).  HOST memory
 * and host computation only; no call touches the GPU.  Not thread-safe.
 *
 * Node 0 is the root; children get the next indices (parents precede
 * children).  A node's value is a log-probability (<= 0) and its weight the
 * sum of values from the root (double; the root's weight is 0).  The order
 * used everywhere: larger weight first, then lower index.
 * Draft cache: the root's keys and values are the last row of the draft's
 * prefix cache (once the root is expanded); every other node selected for
 * expansion owns one tree-cache row (rows 0, 1, ... in selection order; the
 * draft attention of those leaves writes them, swiftspec_draft_tree_attention
 * with the forest below as d_cache_parent).
 *
 * create: an empty tree of capacity nodes holding the root token (not yet
 *   expanded).  destroy: frees it.  size / rows: nodes / tree-cache rows
 *   (-1 for NULL).
 * nodes: copies token, parent, weight, row (-1: none) and expanded (0/1)
 *   of every node into the non-NULL host arrays of size() entries.
 * forest: parent_row[rows()] = the tree-cache row of each row's parent, -1
 *   for a child of the root.
 * select_leaves: the up to w unexpanded, unselected nodes first in the
 *   order (a priority queue, O(w log s)) into leaves[*n]; each non-root one
 *   gets the next tree-cache row; parent_row[j] = its parent's row (-1: the
 *   root).  They stay selected until expanded.
 * expand: for j < n, leaf leaves[j] (selected, not yet expanded) receives
 *   children tokens[j][0..k) with values logprobs[j][0..k) (each <= 0,
 *   e.g. the output of swiftspec_topk_logprobs copied to the host), appended
 *   in leaf order then child order.  Everything is checked first:
 *   SWIFTSPEC_INVALID_ARG (bad leaf, repeated leaf, value > 0 or NaN) or
 *   SWIFTSPEC_CAPACITY leaves the tree unchanged.
 * select_subgraph: the min(bs, size) nodes first in the order -- the most
 *   probable connected subgraph containing the root -- listed by node index
 *   into nodes[*n], with parent[j] = the position of node j's parent in that
 *   list (-1 for the root) and tokens[j] (nullable): a tree for
 *   swiftspec_verify_step.
 * reroot: verified[0 .. n_verified) = the target's output (root token
 *   first, then the accepted tokens and the token the target produced after
 *   them, as in the walk-through of Fig. 3; n_verified >= 2).  From the root the walk goes
 *   to the (lowest-index) child carrying the next verified token while there
 *   is one; *last = the tree-cache row of the deepest walked node owning one
 *   (-1: none) and *path_rows = the walked nodes owning rows (they move to
 *   the prefix).  If the walk consumed every verified token and ended on an
 *   expanded non-root node, that node becomes the root and its subtree is
 *   kept (nodes renumbered in index order, rows in row order, weights minus
 *   its weight): *keep = 1, *n_pending = 0.  Otherwise the tree restarts
 *   from a fresh root holding the last verified token: *keep = 0 and
 *   pending[*n_pending] (at most n_verified entries) = the tokens whose
 *   draft keys and values are still missing, in context order: the old root
 *   if it was never expanded, then the verified tokens after the walked
 *   nodes owning rows (the last is the new root).  *last, *keep and the
 *   forest before the call are the arguments of swiftspec_kv_reorganize for
 *   the draft cache.  SWIFTSPEC_INVALID_ARG if n_verified < 2, if
 *   verified[0] is not the root
 *   token, if a verified token other than the last is not found, or if
 *   selected leaves are still unexpanded; the tree is then unchanged. */
typedef struct swiftspec_draft_tree swiftspec_draft_tree;
int swiftspec_draft_tree_create(int32_t capacity, int32_t root_token, swiftspec_draft_tree** out);
void swiftspec_draft_tree_destroy(swiftspec_draft_tree* t);
int32_t swiftspec_draft_tree_size(const swiftspec_draft_tree* t);
int32_t swiftspec_draft_tree_rows(const swiftspec_draft_tree* t);
int swiftspec_draft_tree_nodes(const swiftspec_draft_tree* t, int32_t* token, int32_t* parent, double* weight,
                               int32_t* row, int32_t* expanded);
int swiftspec_draft_tree_forest(const swiftspec_draft_tree* t, int32_t* parent_row);
int swiftspec_draft_tree_select_leaves(swiftspec_draft_tree* t, int32_t w, int32_t* leaves, int32_t* parent_row,
                                       int32_t* n);
int swiftspec_draft_tree_expand(swiftspec_draft_tree* t, int32_t n, const int32_t* leaves, int32_t k,
                                const int32_t* tokens, const float* logprobs);
int swiftspec_draft_tree_select_subgraph(const swiftspec_draft_tree* t, int32_t bs, int32_t* nodes,
                                         int32_t* parent, int32_t* tokens, int32_t* n);
int swiftspec_draft_tree_reroot(swiftspec_draft_tree* t, const int32_t* verified, int32_t n_verified,
                                int32_t* last, int32_t* path_rows, int32_t* keep, int32_t* pending,
                                int32_t* n_pending);

/* ------------------------------------------------- greedy acceptance
 * Closes a verification step on the device (Sec. 3.1, Fig. 3 walk-through:
 * an iteration's output is the accepted root path followed by one token
 * the target produced after it), for the target's greedy choice.
 *   logits  [T][ldl] fp16 (device): row i = the target's scores for the
 *           token after the root path of node i (as written by
 *           swiftspec_verify_step / swiftspec_lm_head); V columns are read;
 *           values are expected to be finite.
 *   d_tokens[T] int32: the draft token of each node (d_tokens[0], the
 *           root's own token, is not read).
 *   d_parent[T] int32: the tree (parent[0] = -1, 0 <= parent[i] < i).
 * Outputs (device int32): d_argmax[i] = the first index of row i's largest
 * value (the target's choice after node i); *d_accepted = the node reached
 * from the root by repeatedly stepping to the lowest-index child whose
 * token equals the current node's choice, stopping where no child matches;
 * *d_bonus = d_argmax[*d_accepted]; *d_path_len (nullable) = depth of the
 * accepted node + 1 (the accepted path, root included).  The accepted node
 * can be passed straight to swiftspec_kv_commit (d_accepted_node) on the
 * same stream, so verify, accept and commit replay as one graph.
 * 1 <= T <= 64, ldl >= V, ldl % 8 == 0, logits 16-byte aligned.  ws: a
 * workspace of swiftspec_greedy_accept_workspace_bytes(T) bytes (per-range
 * partial maxima after the header; the header's first ticket counter is
 * used and left zero).  An invalid tree sets SWIFTSPEC_DEVERR_BAD_TREE;
 * d_argmax is still written, the other outputs are not. */
size_t swiftspec_greedy_accept_workspace_bytes(int32_t T);
int swiftspec_greedy_accept(const uint16_t* logits, int32_t ldl, int32_t T, int32_t V,
                            const int32_t* d_tokens, const int32_t* d_parent, int32_t* d_argmax,
                            int32_t* d_accepted, int32_t* d_bonus, int32_t* d_path_len, void* ws,
                            size_t ws_bytes, void* stream);

/* -------------------------------------------------------- decoder layer */
typedef struct {
  int32_t H, Hq, Hkv, D, F, S_max;
  float eps;        /* RMSNorm epsilon */
  float rope_theta; /* informational; the table passed in defines the rotation */
} swiftspec_dims;

typedef struct {
  const uint16_t* attn_norm; /* [H] fp16 */
  const uint16_t* mlp_norm;  /* [H] fp16 */
  swiftspec_w4 wqkv;         /* K = H, N = (Hq + 2 Hkv) D: rows [Q heads | K heads | V heads] */
  swiftspec_w4 wo;           /* K = Hq D, N = H */
  swiftspec_w4 wgate, wup;   /* K = H, N = F */
  swiftspec_w4 wdown;        /* K = F, N = H */
  uint16_t* k_cache;         /* [Hkv][S_max][D] */
  uint16_t* v_cache;
} swiftspec_layer;

/* One Llama decoder layer over the draft tree (Algorithm 1, batch verify):
 *   xn = rmsnorm(x, attn_norm); qkv = xn.Wqkv'^T; o = tree_attention(qkv)
 *   h = x + o.Wo'^T; hn = rmsnorm(h, mlp_norm); m = silu(hn.Wg'^T) * (hn.Wu'^T)
 *   out = h + m.Wd'^T
 * with fp16 storage of xn, qkv, o, h, hn, m, out (xn and hn as the operand
 * values of the projections that read them, swiftspec_rmsnorm_w4a16_gemm
 * and _swiglu, which keep them in the workspace only where the norm runs
 * as a kernel of its own).  The layer is
 * exactly the composition rmsnorm_w4a16_gemm, tree_attention, w4a16_gemm
 * (+ residual), rmsnorm_w4a16_swiglu, w4a16_gemm (+ residual).  hidden
 * [T][H] is read as x and overwritten with out.  The caches receive the tree's keys and values
 * at rows [P, P+T).  softmax scale 1/sqrt(D). */
int swiftspec_verify_layer(const swiftspec_layer* layer, const swiftspec_dims* dims,
                           uint16_t* hidden, int32_t T, const int32_t* d_prefix_len,
                           const int32_t* d_parent, const float* rope_cos_sin, void* ws,
                           size_t ws_bytes, void* stream);
size_t swiftspec_verify_layer_workspace_bytes(const swiftspec_dims* dims, int32_t T);
/* Byte offsets, inside the verify_layer workspace, of the layer's fp16
 * intermediates after a call: offsets[0..3] = qkv [T][(Hq+2Hkv)D],
 * o [T][Hq D], h [T][H], m [T][F] (row-major, dense).  For
 * inspection and stage-by-stage checking; the contents are valid until the
 * next call that uses the workspace. */
int swiftspec_verify_layer_workspace_layout(const swiftspec_dims* dims, int32_t T, size_t* offsets);

/* Final RMSNorm and fp16 LM head of the verification step (the logits of
 * every tree node, from which acceptance is decided; Sec. 3.1, Alg. 1):
 *   logits[m][v] = fp16( xn[m] . W[v] ),  xn = fp16(rmsnorm(h[m], gamma)),
 * fp32 accumulation.  h [M][H] fp16 (dense rows), gamma [H] fp16, W [V][H]
 * fp16 row-major (dense, not quantised), logits [M][V] fp16 (dense rows).
 * 1 <= M <= 64, H % 128 == 0, V % 16 == 0; pointers 16-byte aligned.  The
 * normalised rows are kept in the workspace (after its header). */
int swiftspec_lm_head(const uint16_t* h, int32_t M, int32_t H, const uint16_t* gamma, float eps,
                      const uint16_t* W, int32_t V, uint16_t* logits, void* ws, size_t ws_bytes,
                      void* stream);
size_t swiftspec_lm_head_workspace_bytes(int32_t M, int32_t H, int32_t V);

/* The target model's whole verification forward over the draft tree
 * (Alg. 1, batch verify; Sec. 3.1): decoder layers 0 .. n_layers-1 in order
 * (each exactly as swiftspec_verify_layer, with layers[l]'s weights and
 * caches), then, if V > 0, the final RMSNorm and LM head
 * (swiftspec_lm_head) into logits [T][V].  hidden [T][H] is the input
 * embedding of the tree tokens and holds the last layer's output on return.
 * All layers share dims, T, the device prefix length, the parent array and
 * the RoPE table.  Every argument of every layer is checked before the
 * first launch; nothing is enqueued if one fails.  V == 0 skips the head
 * (final_norm, lm_head and logits may then be NULL).  One call enqueues
 * 7 n_layers + 2 kernels (+ split fix-ups) and can be captured whole into
 * one graph. */
int swiftspec_verify_step(const swiftspec_layer* layers, int32_t n_layers, const swiftspec_dims* dims,
                          uint16_t* hidden, int32_t T, const int32_t* d_prefix_len,
                          const int32_t* d_parent, const float* rope_cos_sin,
                          const uint16_t* final_norm, const uint16_t* lm_head, int32_t V,
                          uint16_t* logits, void* ws, size_t ws_bytes, void* stream);
size_t swiftspec_verify_step_workspace_bytes(const swiftspec_dims* dims, int32_t T, int32_t V);

/* -------------------------------------------------------- clock sample
 * Measurement helper for benchmarks, not part of the verification path.
 * Enqueues on `stream` one single-wave kernel.  The kernel reads the shader
 * clock counter (s_memtime) and the 100 MHz real-time counter
 * (s_memrealtime).  It then polls until the real-time counter has advanced
 * by window_us microseconds (1..1000; it also stops after 2^22 polls), and
 * reads both counters again.  The four 64-bit values go to d_out[0..3]
 * (caller-owned device memory, 8-byte aligned): shader start, real start,
 * shader end, real end.  The shader clock in GHz is
 * (d_out[2] - d_out[0]) / (d_out[3] - d_out[1]) / 10.  Enqueued right
 * after a timed region, it reports the clock the chip held there (the
 * power management changes clocks over milliseconds, not microseconds).
 * Returns INVALID_ARG for a null or misaligned d_out or a window outside
 * 1..1000. */
int swiftspec_clock_sample(uint64_t* d_out, int32_t window_us, void* stream);

/* ---------------------------------------------------------- HIP graphs
 * Capture the calls issued on `stream` between begin and end into an
 * executable graph (hipStreamBeginCapture / hipGraphInstantiate) and replay
 * it with swiftspec_graph_launch.  Device-resident prefix length and parent
 * array make one graph valid for every step of a generation. */
typedef struct swiftspec_graph swiftspec_graph;
int swiftspec_graph_begin(void* stream);
int swiftspec_graph_end(void* stream, swiftspec_graph** out);
int swiftspec_graph_launch(swiftspec_graph* g, void* stream);
int swiftspec_graph_destroy(swiftspec_graph* g);

#ifdef __cplusplus
}
#endif
#endif
