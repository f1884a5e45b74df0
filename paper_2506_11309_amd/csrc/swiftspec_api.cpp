// C-ABI layer of libswiftspec.so: argument validation, workspace planning,
// kernel launches on the caller's stream, and HIP-graph helpers.
// The contract of every entry point is documented in include/swiftspec.h.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstring>
#include <mutex>
#include <new>

#include "../../include/swiftspec.h"
#include "ss_internal.h"

namespace {

thread_local int g_last_hip_error = 0;

constexpr size_t kHeader = SWIFTSPEC_WS_HEADER_BYTES;
constexpr size_t kAlign = 256;

inline size_t align_up(size_t v, size_t a = kAlign) { return (v + a - 1) / a * a; }
inline bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }
inline hipStream_t S(void* s) { return reinterpret_cast<hipStream_t>(s); }

int check_launch() {
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) {
    g_last_hip_error = (int)e;
    return SWIFTSPEC_HIP_ERROR;
  }
  return SWIFTSPEC_OK;
}

int hip_status(hipError_t e) {
  if (e != hipSuccess) {
    g_last_hip_error = (int)e;
    return SWIFTSPEC_HIP_ERROR;
  }
  return SWIFTSPEC_OK;
}

int check_w4_shape(const swiftspec_w4* W) {
  if (!W) return SWIFTSPEC_INVALID_ARG;
  if (W->K <= 0 || W->N <= 0) return SWIFTSPEC_INVALID_ARG;
  if (W->K % 128 != 0 || W->N % 64 != 0) return SWIFTSPEC_UNSUPPORTED;
  // the kernels address the packed matrix through 32-bit buffer ranges
  if (ss::w4_packed_bytes(W->K, W->N) > 0xFFFFFFFFull) return SWIFTSPEC_UNSUPPORTED;
  return SWIFTSPEC_OK;
}

// The compute entry points read the kernel-native copy only.
int check_w4(const swiftspec_w4* W) {
  int rc = check_w4_shape(W);
  if (rc) return rc;
  if (!W->packed) return SWIFTSPEC_INVALID_ARG;
  if (!aligned16(W->packed)) return SWIFTSPEC_MISALIGNED;
  return SWIFTSPEC_OK;
}

constexpr int kMaxCounters = (int)((SWIFTSPEC_WS_HEADER_BYTES - 256u) / 4u);

bool attn_counters_fit(int T, int Hq, int Hkv) {
  const long R = (long)T * (Hq / Hkv);
  return (long)Hkv * ((R + 63) / 64) <= kMaxCounters;
}

size_t gemm_ws(int M, int K, int N, bool swiglu) {
  ss::GemmPlan p = ss::plan_w4a16_gemm(M, K, N, swiglu);
  return kHeader + align_up(p.prep_bytes) + align_up(p.part_bytes);
}

// Launch a validated W4A16 GEMM / SwiGLU reading prepared activations.
// With `norm` (x, ldx, gamma, eps) the input is RMSNorm(x), computed inside
// the GEMM; only K-split plans take it (norm_in_gemm).
struct NormIn {
  const uint16_t* x;
  int ldx;
  const uint16_t* gamma;
  float eps;
};

bool norm_in_gemm(int M, const swiftspec_w4* W0, bool swiglu) {
  return ss::norm_in_kslice(ss::plan_w4a16_gemm(M, W0->K, W0->N, swiglu), W0->K);
}

void run_gemm(const swiftspec_w4* W0, const swiftspec_w4* W1, const uint16_t* aprep, int M,
              uint16_t* y, int ldy, uint16_t* yprep, const uint16_t* res, int ldr, void* ws,
              float* part, hipStream_t st, const NormIn* norm = nullptr) {
  const bool swiglu = W1 != nullptr;
  ss::GemmPlan p = ss::plan_w4a16_gemm(M, W0->K, W0->N, swiglu);
  ss::GemmLaunch L;
  if (norm) {
    L.xnorm = norm->x;
    L.ldx = norm->ldx;
    L.gamma = norm->gamma;
    L.eps = norm->eps;
  }
  L.w0 = W0->packed;
  L.w1 = swiglu ? W1->packed : W0->packed;
  L.K = W0->K;
  L.N = W0->N;
  L.aprep = aprep;
  L.M = M;
  L.y = y;
  L.ldy = ldy;
  L.yprep = yprep;
  L.res = res;
  L.ldr = ldr;
  L.nw = p.nw;
  L.nblocks = p.nblocks;
  L.nwg = p.nwg;
  L.ksw = p.ksw;
  L.swiglu = swiglu;
  L.part = part;
  ss::launch_w4a16_gemm(L, st);
}

// RMSNorm(x; gamma, eps) followed by the GEMM / SwiGLU: inside the GEMM
// where its plan splits K within workgroups, else the norm kernel writes
// the prepared operand into xprep and the GEMM reads it.
void run_norm_gemm(const swiftspec_w4* W0, const swiftspec_w4* W1, const NormIn& n, int M, uint16_t* y,
                   int ldy, uint16_t* yprep, uint16_t* xprep, void* ws, float* part, hipStream_t st) {
  if (norm_in_gemm(M, W0, W1 != nullptr)) {
    run_gemm(W0, W1, nullptr, M, y, ldy, yprep, nullptr, 0, ws, part, st, &n);
  } else {
    ss::launch_rmsnorm(n.x, M, W0->K, n.ldx, n.gamma, n.eps, nullptr, 0, xprep, st);
    run_gemm(W0, W1, xprep, M, y, ldy, yprep, nullptr, 0, ws, part, st);
  }
}

// Standalone entry: prepare plain x into the workspace, then run the GEMM.
void run_gemm_plain(const swiftspec_w4* W0, const swiftspec_w4* W1, const uint16_t* x, int M, int ldx,
                    uint16_t* y, int ldy, const uint16_t* res, int ldr, void* ws, hipStream_t st) {
  ss::GemmPlan p = ss::plan_w4a16_gemm(M, W0->K, W0->N, W1 != nullptr);
  char* base = static_cast<char*>(ws);
  uint16_t* aprep = reinterpret_cast<uint16_t*>(base + kHeader);
  float* part = reinterpret_cast<float*>(base + kHeader + align_up(p.prep_bytes));
  ss::launch_prepare_activations(x, M, ldx, W0->K, aprep, st);
  run_gemm(W0, W1, aprep, M, y, ldy, nullptr, res, ldr, ws, part, st);
}

int check_tree_attention_args(const uint16_t* q, int ldq, const uint16_t* k, const uint16_t* v,
                              int ldkv, const uint16_t* kc, const uint16_t* vc, int S_max,
                              const int32_t* P, const int32_t* parent, int T, int Hq, int Hkv,
                              int D, const float* rope, float scale, const uint16_t* out, int ldo) {
  if (!q || !k || !v || !kc || !vc || !P || !parent || !rope || !out) return SWIFTSPEC_INVALID_ARG;
  if (!(scale > 0.f) || !std::isfinite(scale)) return SWIFTSPEC_INVALID_ARG;
  if (T < 1 || Hq < 1 || Hkv < 1 || S_max < T) return SWIFTSPEC_INVALID_ARG;
  if (T > SWIFTSPEC_MAX_TREE || (D != 64 && D != 128) || Hq % Hkv != 0) return SWIFTSPEC_UNSUPPORTED;
  if (ldq < Hq * D || ldkv < Hkv * D || ldo < Hq * D) return SWIFTSPEC_INVALID_ARG;
  if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(kc) || !aligned16(vc))
    return SWIFTSPEC_MISALIGNED;
  if (ldq % 8 || ldkv % 8) return SWIFTSPEC_MISALIGNED;
  if (!attn_counters_fit(T, Hq, Hkv)) return SWIFTSPEC_UNSUPPORTED;
  return SWIFTSPEC_OK;
}

// partial bytes of the target or the draft attention kernel, whichever is larger
size_t attn_part_bytes(int T, int Hq, int Hkv, int D, int S_max) {
  const size_t a = ss::plan_tree_attention(T, Hq, Hkv, D, S_max, false).part_bytes;
  const size_t b = ss::plan_tree_attention(T, Hq, Hkv, D, S_max, true).part_bytes;
  return a > b ? a : b;
}

size_t attn_ws(int T, int Hq, int Hkv, int D, int S_max) {
  return kHeader + align_up(attn_part_bytes(T, Hq, Hkv, D, S_max));
}

void run_attention(const uint16_t* q, int ldq, const uint16_t* k, const uint16_t* v, int ldkv,
                   uint16_t* kc, uint16_t* vc, int S_max, const int32_t* P, const int32_t* parent,
                   int T, int Hq, int Hkv, int D, const float* rope, float scale, uint16_t* out,
                   int ldo, uint16_t* out_prep, void* ws, float* part, hipStream_t st, int N = 0,
                   const int32_t* cache_parent = nullptr, const int32_t* leaf_parent = nullptr) {
  ss::AttnPlan p = ss::plan_tree_attention(T, Hq, Hkv, D, S_max, N > 0 || leaf_parent != nullptr);
  ss::AttnLaunch L;
  L.N = N;
  L.cache_parent = cache_parent;
  L.leaf_parent = leaf_parent;
  L.q = q;
  L.ldq = ldq;
  L.k = k;
  L.v = v;
  L.ldkv = ldkv;
  L.k_cache = kc;
  L.v_cache = vc;
  L.S_max = S_max;
  L.prefix_len = P;
  L.parent = parent;
  L.T = T;
  L.Hq = Hq;
  L.Hkv = Hkv;
  L.D = D;
  L.rope = rope;
  L.scale = scale;
  L.out = out;
  L.ldo = ldo;
  L.out_prep = out_prep;
  L.ws = ws;
  L.part = part;
  L.nsplit = p.nsplit;
  L.chunk = p.chunk;
  ss::launch_tree_attention(L, st);
}

// ---- tree attention without allocation: partials in a library-owned array
// of SWIFTSPEC_NOALLOC_SCRATCH_BYTES per GPU.  In host code `scratch` names a
// host-side stand-in; the device address of each GPU's copy is looked up
// once per device (with that device current) and used everywhere instead.
static __device__ __align__(256) unsigned char scratch[SWIFTSPEC_NOALLOC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

// Device address of the current device's scratch array, or nullptr with the
// status in *rc.
void* noalloc_scratch(int* rc) {
  int dev = 0;
  *rc = hip_status(hipGetDevice(&dev));
  if (*rc) return nullptr;
  if (dev < 0 || dev >= kMaxDevices) {
    *rc = SWIFTSPEC_UNSUPPORTED;
    return nullptr;
  }
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    *rc = hip_status(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)));
    if (*rc) return nullptr;
    g_scratch_ptr[dev] = p;
  }
  return g_scratch_ptr[dev];
}

struct LayerWs {
  size_t qkv, o, h, m, xn_p, o_p, hn_p, m_p, part, total;
};

LayerWs layer_ws(const swiftspec_dims* d, int T) {
  LayerWs w;
  const int Nqkv = (d->Hq + 2 * d->Hkv) * d->D;
  const size_t MT16 = (size_t)((T + 15) / 16) * 16;  // prepared buffers hold whole 16-row tiles
  size_t off = kHeader;
  auto take = [&](size_t bytes) {
    const size_t o = off;
    off += align_up(bytes);
    return o;
  };
  w.qkv = take((size_t)T * Nqkv * 2);
  w.o = take((size_t)T * d->Hq * d->D * 2);
  w.h = take((size_t)T * d->H * 2);
  w.m = take((size_t)T * d->F * 2);
  w.xn_p = take(MT16 * d->H * 2);
  w.o_p = take(MT16 * d->Hq * d->D * 2);
  w.hn_p = take(MT16 * d->H * 2);
  w.m_p = take(MT16 * d->F * 2);
  size_t part = 0;
  auto upd = [&](size_t b) { part = b > part ? b : part; };
  upd(ss::plan_w4a16_gemm(T, d->H, Nqkv, false).part_bytes);
  upd(ss::plan_w4a16_gemm(T, d->Hq * d->D, d->H, false).part_bytes);
  upd(ss::plan_w4a16_gemm(T, d->H, d->F, true).part_bytes);
  upd(ss::plan_w4a16_gemm(T, d->F, d->H, false).part_bytes);
  upd(attn_part_bytes(T, d->Hq, d->Hkv, d->D, d->S_max));
  w.part = take(part);
  w.total = off;
  return w;
}

}  // namespace

extern "C" {

const char* swiftspec_status_string(int status) {
  switch (status) {
    case SWIFTSPEC_OK: return "ok";
    case SWIFTSPEC_INVALID_ARG: return "invalid argument";
    case SWIFTSPEC_UNSUPPORTED: return "unsupported shape";
    case SWIFTSPEC_MISALIGNED: return "misaligned pointer or leading dimension";
    case SWIFTSPEC_WORKSPACE_TOO_SMALL: return "workspace too small";
    case SWIFTSPEC_BAD_TREE: return "invalid parent array";
    case SWIFTSPEC_HIP_ERROR: return "HIP runtime error";
    case SWIFTSPEC_CAPACITY: return "draft tree capacity exceeded";
    default: return "unknown status";
  }
}

int swiftspec_last_hip_error(void) { return g_last_hip_error; }

int swiftspec_workspace_init(void* ws, size_t ws_bytes, void* stream) {
  if (!ws || ws_bytes < kHeader) return SWIFTSPEC_INVALID_ARG;
  ss::launch_ws_init(ws, kHeader, S(stream));
  return check_launch();
}

int swiftspec_read_device_error(void* ws, void* stream, uint32_t* out) {
  if (!ws || !out) return SWIFTSPEC_INVALID_ARG;
  int rc = hip_status(hipStreamSynchronize(S(stream)));
  if (rc) return rc;
  rc = hip_status(hipMemcpy(out, ws, sizeof(uint32_t), hipMemcpyDeviceToHost));
  if (rc) return rc;
  ss::launch_ws_init(ws, 256, S(stream));
  rc = check_launch();
  if (rc) return rc;
  return hip_status(hipStreamSynchronize(S(stream)));
}

int swiftspec_clock_sample(uint64_t* d_out, int32_t window_us, void* stream) {
  if (!d_out || (reinterpret_cast<uintptr_t>(d_out) & 7u) || window_us < 1 || window_us > 1000)
    return SWIFTSPEC_INVALID_ARG;
  ss::launch_clock_sample(d_out, (uint32_t)window_us * 100u, S(stream));
  return check_launch();
}

size_t swiftspec_w4_packed_bytes(int32_t K, int32_t N) {
  if (K <= 0 || N <= 0) return 0;
  return ss::w4_packed_bytes(K, N);
}

int swiftspec_w4_prepack(const swiftspec_w4* W, void* packed, size_t packed_bytes, void* stream) {
  int rc = check_w4_shape(W);
  if (rc) return rc;
  if (!W->qweight || !W->scales || !W->zeros || !packed) return SWIFTSPEC_INVALID_ARG;
  if (!aligned16(W->qweight) || !aligned16(packed)) return SWIFTSPEC_MISALIGNED;
  if (packed_bytes < ss::w4_packed_bytes(W->K, W->N)) return SWIFTSPEC_WORKSPACE_TOO_SMALL;
  ss::launch_prepack_w4(W->qweight, W->scales, W->zeros, W->K, W->N, packed, S(stream));
  return check_launch();
}

size_t swiftspec_w4a16_gemm_workspace_bytes(int32_t M, int32_t K, int32_t N) {
  if (M < 1 || K < 128 || N < 16) return kHeader;
  return gemm_ws(M, K, N, false);
}

size_t swiftspec_w4a16_swiglu_workspace_bytes(int32_t M, int32_t K, int32_t N) {
  if (M < 1 || K < 128 || N < 16) return kHeader;
  return gemm_ws(M, K, N, true);
}

int swiftspec_w4a16_gemm(const swiftspec_w4* W, const uint16_t* x, int32_t M, int32_t ldx,
                         uint16_t* y, int32_t ldy, const uint16_t* residual, int32_t ldr,
                         void* ws, size_t ws_bytes, void* stream) {
  int rc = check_w4(W);
  if (rc) return rc;
  if (!x || !y || !ws) return SWIFTSPEC_INVALID_ARG;
  if (M < 0 || ldx < W->K || ldy < W->N || (residual && ldr < W->N)) return SWIFTSPEC_INVALID_ARG;
  if (M > SWIFTSPEC_MAX_M) return SWIFTSPEC_UNSUPPORTED;
  if (!aligned16(x) || ldx % 8) return SWIFTSPEC_MISALIGNED;
  if (residual == y && ldr != ldy) return SWIFTSPEC_INVALID_ARG;
  if (M == 0) return SWIFTSPEC_OK;
  if (ws_bytes < gemm_ws(M, W->K, W->N, false)) return SWIFTSPEC_WORKSPACE_TOO_SMALL;
  run_gemm_plain(W, nullptr, x, M, ldx, y, ldy, residual, ldr, ws, S(stream));
  return check_launch();
}

size_t swiftspec_w4a16_gemm_valu_workspace_bytes(int32_t M, int32_t K, int32_t N) {
  if (M < 1 || K < 128 || N < 64) return kHeader;
  const ss::GemmPlan g = ss::plan_w4a16_gemm(M, K, N, false);
  const ss::ValuGemmPlan p = ss::plan_w4a16_gemm_valu(M, K, N);
  return kHeader + align_up(g.prep_bytes) + align_up(p.part_bytes);
}

int swiftspec_w4a16_gemm_valu(const swiftspec_w4* W, const uint16_t* x, int32_t M, int32_t ldx, uint16_t* y,
                              int32_t ldy, const uint16_t* residual, int32_t ldr, void* ws, size_t ws_bytes,
                              void* stream) {
  int rc = check_w4(W);
  if (rc) return rc;
  if (!x || !y || !ws) return SWIFTSPEC_INVALID_ARG;
  if (M < 0 || ldx < W->K || ldy < W->N || (residual && ldr < W->N)) return SWIFTSPEC_INVALID_ARG;
  if (M > SWIFTSPEC_MAX_M) return SWIFTSPEC_UNSUPPORTED;
  if (!aligned16(x) || ldx % 8 || !aligned16(ws)) return SWIFTSPEC_MISALIGNED;
  if (residual == y && ldr != ldy) return SWIFTSPEC_INVALID_ARG;
  if (M == 0) return SWIFTSPEC_OK;
  if (ws_bytes < swiftspec_w4a16_gemm_valu_workspace_bytes(M, W->K, W->N)) return SWIFTSPEC_WORKSPACE_TOO_SMALL;
  const ss::GemmPlan g = ss::plan_w4a16_gemm(M, W->K, W->N, false);
  const ss::ValuGemmPlan p = ss::plan_w4a16_gemm_valu(M, W->K, W->N);
  char* base = static_cast<char*>(ws);
  uint16_t* aprep = reinterpret_cast<uint16_t*>(base + kHeader);
  float* part = reinterpret_cast<float*>(base + kHeader + align_up(g.prep_bytes));
  hipStream_t st = S(stream);
  ss::launch_prepare_activations(x, M, ldx, W->K, aprep, st);
  ss::launch_w4a16_gemm_valu(W->packed, W->K, W->N, aprep, M, y, ldy, residual, ldr, part, p, st);
  return check_launch();
}

int swiftspec_w4a16_swiglu(const swiftspec_w4* Wg, const swiftspec_w4* Wu, const uint16_t* x,
                           int32_t M, int32_t ldx, uint16_t* y, int32_t ldy, void* ws,
                           size_t ws_bytes, void* stream) {
  int rc = check_w4(Wg);
  if (rc) return rc;
  rc = check_w4(Wu);
  if (rc) return rc;
  if (Wg->K != Wu->K || Wg->N != Wu->N) return SWIFTSPEC_INVALID_ARG;
  if (!x || !y || !ws) return SWIFTSPEC_INVALID_ARG;
  if (M < 0 || ldx < Wg->K || ldy < Wg->N) return SWIFTSPEC_INVALID_ARG;
  if (M > SWIFTSPEC_MAX_M) return SWIFTSPEC_UNSUPPORTED;
  if (!aligned16(x) || ldx % 8) return SWIFTSPEC_MISALIGNED;
  if (M == 0) return SWIFTSPEC_OK;
  if (ws_bytes < gemm_ws(M, Wg->K, Wg->N, true)) return SWIFTSPEC_WORKSPACE_TOO_SMALL;
  run_gemm_plain(Wg, Wu, x, M, ldx, y, ldy, nullptr, 0, ws, S(stream));
  return check_launch();
}

// Argument checks shared by the RMSNorm + GEMM / SwiGLU entry points.
static int check_norm_gemm(const swiftspec_w4* W0, const swiftspec_w4* W1, const uint16_t* x, int32_t M,
                           int32_t ldx, const uint16_t* gamma, const uint16_t* y, int32_t ldy, const void* ws) {
  int rc = check_w4(W0);
  if (rc) return rc;
  if (W1) {
    if ((rc = check_w4(W1))) return rc;
    if (W0->K != W1->K || W0->N != W1->N) return SWIFTSPEC_INVALID_ARG;
  }
  if (!x || !gamma || !y || !ws) return SWIFTSPEC_INVALID_ARG;
  if (M < 0 || ldx < W0->K || ldy < W0->N) return SWIFTSPEC_INVALID_ARG;
  if (M > SWIFTSPEC_MAX_M) return SWIFTSPEC_UNSUPPORTED;
  if (!aligned16(x) || !aligned16(gamma) || ldx % 8) return SWIFTSPEC_MISALIGNED;
  return SWIFTSPEC_OK;
}

int swiftspec_rmsnorm_w4a16_gemm(const swiftspec_w4* W, const uint16_t* x, int32_t M, int32_t ldx,
                                 const uint16_t* gamma, float eps, uint16_t* y, int32_t ldy, void* ws,
                                 size_t ws_bytes, void* stream) {
  int rc = check_norm_gemm(W, nullptr, x, M, ldx, gamma, y, ldy, ws);
  if (rc) return rc;
  if (M == 0) return SWIFTSPEC_OK;
  if (ws_bytes < gemm_ws(M, W->K, W->N, false)) return SWIFTSPEC_WORKSPACE_TOO_SMALL;
  const ss::GemmPlan p = ss::plan_w4a16_gemm(M, W->K, W->N, false);
  char* base = static_cast<char*>(ws);
  run_norm_gemm(W, nullptr, NormIn{x, ldx, gamma, eps}, M, y, ldy, nullptr,
                reinterpret_cast<uint16_t*>(base + kHeader),
                ws, reinterpret_cast<float*>(base + kHeader + align_up(p.prep_bytes)), S(stream));
  return check_launch();
}

int swiftspec_rmsnorm_w4a16_swiglu(const swiftspec_w4* Wg, const swiftspec_w4* Wu, const uint16_t* x,
                                   int32_t M, int32_t ldx, const uint16_t* gamma, float eps, uint16_t* y,
                                   int32_t ldy, void* ws, size_t ws_bytes, void* stream) {
  if (!Wu) return SWIFTSPEC_INVALID_ARG;
  int rc = check_norm_gemm(Wg, Wu, x, M, ldx, gamma, y, ldy, ws);
  if (rc) return rc;
  if (M == 0) return SWIFTSPEC_OK;
  if (ws_bytes < gemm_ws(M, Wg->K, Wg->N, true)) return SWIFTSPEC_WORKSPACE_TOO_SMALL;
  const ss::GemmPlan p = ss::plan_w4a16_gemm(M, Wg->K, Wg->N, true);
  char* base = static_cast<char*>(ws);
  run_norm_gemm(Wg, Wu, NormIn{x, ldx, gamma, eps}, M, y, ldy, nullptr,
                reinterpret_cast<uint16_t*>(base + kHeader),
                ws, reinterpret_cast<float*>(base + kHeader + align_up(p.prep_bytes)), S(stream));
  return check_launch();
}

size_t swiftspec_prepared_bytes(int32_t M, int32_t K) {
  if (M < 1 || K < 128 || K % 128) return 0;
  return (size_t)((M + 15) / 16) * (K / 128) * 4 * 64 * 16;
}

int swiftspec_prepare_activations(const uint16_t* x, int32_t M, int32_t ldx, int32_t K, uint16_t* xp,
                                  void* stream) {
  if (!x || !xp || M < 0 || K <= 0 || ldx < K) return SWIFTSPEC_INVALID_ARG;
  if (K % 128 || M > SWIFTSPEC_MAX_M) return SWIFTSPEC_UNSUPPORTED;
  if (!aligned16(x) || !aligned16(xp) || ldx % 8) return SWIFTSPEC_MISALIGNED;
  if (M == 0) return SWIFTSPEC_OK;
  ss::launch_prepare_activations(x, M, ldx, K, xp, S(stream));
  return check_launch();
}

int swiftspec_w4a16_gemm_prepared(const swiftspec_w4* W, const uint16_t* xp, int32_t M, uint16_t* y,
                                  int32_t ldy, const uint16_t* residual, int32_t ldr, void* ws,
                                  size_t ws_bytes, void* stream) {
  int rc = check_w4(W);
  if (rc) return rc;
  if (!xp || !y || !ws || M < 0 || ldy < W->N || (residual && ldr < W->N)) return SWIFTSPEC_INVALID_ARG;
  if (M > SWIFTSPEC_MAX_M) return SWIFTSPEC_UNSUPPORTED;
  if (!aligned16(xp)) return SWIFTSPEC_MISALIGNED;
  if (residual == y && ldr != ldy) return SWIFTSPEC_INVALID_ARG;
  if (M == 0) return SWIFTSPEC_OK;
  ss::GemmPlan p = ss::plan_w4a16_gemm(M, W->K, W->N, false);
  if (ws_bytes < kHeader + align_up(p.part_bytes)) return SWIFTSPEC_WORKSPACE_TOO_SMALL;
  run_gemm(W, nullptr, xp, M, y, ldy, nullptr, residual, ldr, ws,
           reinterpret_cast<float*>(static_cast<char*>(ws) + kHeader), S(stream));
  return check_launch();
}

int swiftspec_w4a16_swiglu_prepared(const swiftspec_w4* Wg, const swiftspec_w4* Wu, const uint16_t* xp,
                                    int32_t M, uint16_t* y, int32_t ldy, void* ws, size_t ws_bytes,
                                    void* stream) {
  int rc = check_w4(Wg);
  if (rc) return rc;
  rc = check_w4(Wu);
  if (rc) return rc;
  if (Wg->K != Wu->K || Wg->N != Wu->N) return SWIFTSPEC_INVALID_ARG;
  if (!xp || !y || !ws || M < 0 || ldy < Wg->N) return SWIFTSPEC_INVALID_ARG;
  if (M > SWIFTSPEC_MAX_M) return SWIFTSPEC_UNSUPPORTED;
  if (!aligned16(xp)) return SWIFTSPEC_MISALIGNED;
  if (M == 0) return SWIFTSPEC_OK;
  ss::GemmPlan p = ss::plan_w4a16_gemm(M, Wg->K, Wg->N, true);
  if (ws_bytes < kHeader + align_up(p.part_bytes)) return SWIFTSPEC_WORKSPACE_TOO_SMALL;
  run_gemm(Wg, Wu, xp, M, y, ldy, nullptr, nullptr, 0, ws,
           reinterpret_cast<float*>(static_cast<char*>(ws) + kHeader), S(stream));
  return check_launch();
}

int swiftspec_rmsnorm(const uint16_t* x, int32_t M, int32_t H, int32_t ldx, const uint16_t* gamma,
                      float eps, uint16_t* out, int32_t ldo, void* stream) {
  if (!x || !gamma || !out || M < 0 || H <= 0 || ldx < H || ldo < H) return SWIFTSPEC_INVALID_ARG;
  if (H % 32) return SWIFTSPEC_UNSUPPORTED;  // whole 32-element chunks (one operand-layout fragment set)
  if (!aligned16(x) || !aligned16(gamma) || !aligned16(out) || ldx % 8 || ldo % 8)
    return SWIFTSPEC_MISALIGNED;
  if (M == 0) return SWIFTSPEC_OK;
  ss::launch_rmsnorm(x, M, H, ldx, gamma, eps, out, ldo, nullptr, S(stream));
  return check_launch();
}

size_t swiftspec_tree_attention_workspace_bytes(int32_t T, int32_t Hq, int32_t Hkv, int32_t D,
                                                int32_t S_max) {
  if (T < 1 || Hq < 1 || Hkv < 1 || Hq % Hkv || (D != 64 && D != 128) || S_max < T) return kHeader;
  return attn_ws(T, Hq, Hkv, D, S_max);
}

int swiftspec_tree_attention(const uint16_t* q, int32_t ldq, const uint16_t* k, const uint16_t* v,
                             int32_t ldkv, uint16_t* k_cache, uint16_t* v_cache, int32_t S_max,
                             const int32_t* d_prefix_len, const int32_t* d_parent, int32_t T,
                             int32_t Hq, int32_t Hkv, int32_t D, const float* rope_cos_sin,
                             float softmax_scale, uint16_t* out, int32_t ldo, void* ws,
                             size_t ws_bytes, void* stream) {
  int rc = check_tree_attention_args(q, ldq, k, v, ldkv, k_cache, v_cache, S_max, d_prefix_len,
                                     d_parent, T, Hq, Hkv, D, rope_cos_sin, softmax_scale, out, ldo);
  if (rc) return rc;
  if (!ws) return SWIFTSPEC_INVALID_ARG;
  if (ws_bytes < attn_ws(T, Hq, Hkv, D, S_max)) return SWIFTSPEC_WORKSPACE_TOO_SMALL;
  run_attention(q, ldq, k, v, ldkv, k_cache, v_cache, S_max, d_prefix_len, d_parent, T, Hq, Hkv, D,
                rope_cos_sin, softmax_scale, out, ldo, nullptr, ws,
                reinterpret_cast<float*>(static_cast<char*>(ws) + kHeader), S(stream));
  return check_launch();
}

int swiftspec_tree_attention_noalloc(const uint16_t* q, int32_t ldq, const uint16_t* k, const uint16_t* v,
                                     int32_t ldkv, uint16_t* k_cache, uint16_t* v_cache, int32_t S_max,
                                     const int32_t* d_prefix_len, const int32_t* d_parent, int32_t T,
                                     int32_t Hq, int32_t Hkv, int32_t D, const float* rope_cos_sin,
                                     float softmax_scale, uint16_t* out, int32_t ldo, uint32_t* d_error,
                                     void* stream) {
  int rc = check_tree_attention_args(q, ldq, k, v, ldkv, k_cache, v_cache, S_max, d_prefix_len,
                                     d_parent, T, Hq, Hkv, D, rope_cos_sin, softmax_scale, out, ldo);
  if (rc) return rc;
  if (ss::plan_tree_attention(T, Hq, Hkv, D, S_max, false).part_bytes > SWIFTSPEC_NOALLOC_SCRATCH_BYTES)
    return SWIFTSPEC_WORKSPACE_TOO_SMALL;
  float* part = static_cast<float*>(noalloc_scratch(&rc));
  if (rc) return rc;
  // the kernels OR device errors into word 0 of `ws`: here the caller's word
  run_attention(q, ldq, k, v, ldkv, k_cache, v_cache, S_max, d_prefix_len, d_parent, T, Hq, Hkv, D,
                rope_cos_sin, softmax_scale, out, ldo, nullptr, d_error, part, S(stream));
  return check_launch();
}

int swiftspec_rope_table(double theta, int32_t S_max, int32_t D, float* host_out) {
  if (!host_out || S_max < 1 || D < 2 || D % 2 || !(theta > 0)) return SWIFTSPEC_INVALID_ARG;
  const int half = D / 2;
  for (int d = 0; d < half; ++d) {
    const double inv_freq = std::pow(theta, -2.0 * d / (double)D);
    for (int pos = 0; pos < S_max; ++pos) {
      const double ang = (double)pos * inv_freq;
      host_out[((size_t)pos * half + d) * 2 + 0] = (float)std::cos(ang);
      host_out[((size_t)pos * half + d) * 2 + 1] = (float)std::sin(ang);
    }
  }
  return SWIFTSPEC_OK;
}

int swiftspec_tree_masks(const int32_t* d_parents, int32_t n_trees, int32_t T, uint64_t* d_anc,
                         int32_t* d_depth, int32_t* d_status, void* stream) {
  if (!d_parents || !d_anc || !d_depth || !d_status || n_trees < 0 || T < 1) return SWIFTSPEC_INVALID_ARG;
  if (T > SWIFTSPEC_MAX_TREE) return SWIFTSPEC_UNSUPPORTED;
  if (n_trees == 0) return SWIFTSPEC_OK;
  ss::launch_tree_masks(d_parents, n_trees, T, d_anc, d_depth, d_status, S(stream));
  return check_launch();
}

int swiftspec_tree_validate(const int32_t* parent, int32_t T, int32_t* depth_out) {
  if (!parent || T < 1) return SWIFTSPEC_INVALID_ARG;
  if (parent[0] != -1) return SWIFTSPEC_BAD_TREE;
  for (int i = 1; i < T; ++i)
    if (parent[i] < 0 || parent[i] >= i) return SWIFTSPEC_BAD_TREE;
  if (depth_out) {
    depth_out[0] = 0;
    for (int i = 1; i < T; ++i) depth_out[i] = depth_out[parent[i]] + 1;
  }
  return SWIFTSPEC_OK;
}

int swiftspec_kv_commit(uint16_t* k_cache, uint16_t* v_cache, int32_t n_layers,
                        int64_t layer_stride_elems, int32_t Hkv, int32_t S_max, int32_t D,
                        int32_t* d_prefix_len, const int32_t* d_parent, int32_t T,
                        const int32_t* d_accepted_node, int32_t advance, void* ws,
                        size_t ws_bytes, void* stream) {
  if (!k_cache || !v_cache || !d_prefix_len || !d_parent || !d_accepted_node) return SWIFTSPEC_INVALID_ARG;
  if (n_layers < 1 || Hkv < 1 || T < 1 || S_max < T || D < 8) return SWIFTSPEC_INVALID_ARG;
  if (layer_stride_elems < (int64_t)Hkv * S_max * D) return SWIFTSPEC_INVALID_ARG;
  if (T > SWIFTSPEC_MAX_TREE || D % 8 || D > 256) return SWIFTSPEC_UNSUPPORTED;
  if (!aligned16(k_cache) || !aligned16(v_cache) || layer_stride_elems % 8) return SWIFTSPEC_MISALIGNED;
  if (ws && ws_bytes < kHeader) return SWIFTSPEC_WORKSPACE_TOO_SMALL;
  if ((int64_t)n_layers * 2 * Hkv > 0x7fffffff) return SWIFTSPEC_UNSUPPORTED;
  ss::launch_kv_commit(k_cache, v_cache, n_layers, layer_stride_elems, Hkv, S_max, D, d_prefix_len,
                       d_parent, T, d_accepted_node, advance, ws, S(stream));
  return check_launch();
}

int swiftspec_draft_tree_attention(const uint16_t* q, int32_t ldq, const uint16_t* k, const uint16_t* v,
                                   int32_t ldkv, uint16_t* k_cache, uint16_t* v_cache, int32_t S_max,
                                   const int32_t* d_prefix_len, const int32_t* d_cache_parent, int32_t N,
                                   const int32_t* d_leaf_parent, int32_t w, int32_t Hq, int32_t Hkv, int32_t D,
                                   const float* rope_cos_sin, float softmax_scale, uint16_t* out, int32_t ldo,
                                   void* ws, size_t ws_bytes, void* stream) {
  if (N < 0 || (N > 0 && !d_cache_parent) || !d_leaf_parent) return SWIFTSPEC_INVALID_ARG;
  if (N > SWIFTSPEC_MAX_TREE) return SWIFTSPEC_UNSUPPORTED;
  if ((int64_t)N + w > S_max) return SWIFTSPEC_INVALID_ARG;
  // the same checks as the target attention over w new tokens (d_leaf_parent
  // stands in for the parent array)
  int rc = check_tree_attention_args(q, ldq, k, v, ldkv, k_cache, v_cache, S_max, d_prefix_len, d_leaf_parent, w,
                                     Hq, Hkv, D, rope_cos_sin, softmax_scale, out, ldo);
  if (rc) return rc;
  if (!ws) return SWIFTSPEC_INVALID_ARG;
  if (ws_bytes < attn_ws(w, Hq, Hkv, D, S_max)) return SWIFTSPEC_WORKSPACE_TOO_SMALL;
  run_attention(q, ldq, k, v, ldkv, k_cache, v_cache, S_max, d_prefix_len, d_leaf_parent, w, Hq, Hkv, D,
                rope_cos_sin, softmax_scale, out, ldo, nullptr, ws,
                reinterpret_cast<float*>(static_cast<char*>(ws) + kHeader), S(stream), N, d_cache_parent,
                d_leaf_parent);
  return check_launch();
}

int swiftspec_kv_reorganize(uint16_t* k_cache, uint16_t* v_cache, int32_t n_layers, int64_t layer_stride_elems,
                            int32_t Hkv, int32_t S_max, int32_t D, int32_t* d_prefix_len, const int32_t* d_parent,
                            int32_t N, const int32_t* d_last, const int32_t* d_keep, int32_t* d_new_parent,
                            int32_t* d_n_kept, int32_t advance, void* ws, size_t ws_bytes, void* stream) {
  if (!k_cache || !v_cache || !d_prefix_len || !d_parent || !d_last || !d_keep) return SWIFTSPEC_INVALID_ARG;
  if (n_layers < 1 || Hkv < 1 || N < 1 || S_max < N || D < 8) return SWIFTSPEC_INVALID_ARG;
  if (d_new_parent) {  // the old forest is read while the new one is written
    const uintptr_t a0 = reinterpret_cast<uintptr_t>(d_parent), b0 = reinterpret_cast<uintptr_t>(d_new_parent);
    const uintptr_t bytes = (uintptr_t)N * sizeof(int32_t);
    if (a0 < b0 + bytes && b0 < a0 + bytes) return SWIFTSPEC_INVALID_ARG;
  }
  if (layer_stride_elems < (int64_t)Hkv * S_max * D) return SWIFTSPEC_INVALID_ARG;
  if (N > SWIFTSPEC_MAX_TREE || D % 8 || D > 256) return SWIFTSPEC_UNSUPPORTED;
  if (!aligned16(k_cache) || !aligned16(v_cache) || layer_stride_elems % 8) return SWIFTSPEC_MISALIGNED;
  if (ws && ws_bytes < kHeader) return SWIFTSPEC_WORKSPACE_TOO_SMALL;
  if ((int64_t)n_layers * 2 * Hkv > 0x7fffffff) return SWIFTSPEC_UNSUPPORTED;
  ss::launch_kv_reorganize(k_cache, v_cache, n_layers, layer_stride_elems, Hkv, S_max, D, d_prefix_len, d_parent, N,
                           d_last, d_keep, d_new_parent, d_n_kept, advance, ws, S(stream));
  return check_launch();
}

size_t swiftspec_greedy_accept_workspace_bytes(int32_t T) {
  if (T < 1 || T > SWIFTSPEC_MAX_TREE) return kHeader;
  return kHeader + align_up((size_t)T * ss::greedy_accept_splits(T) * 8);
}

int swiftspec_greedy_accept(const uint16_t* logits, int32_t ldl, int32_t T, int32_t V,
                            const int32_t* d_tokens, const int32_t* d_parent, int32_t* d_argmax,
                            int32_t* d_accepted, int32_t* d_bonus, int32_t* d_path_len, void* ws,
                            size_t ws_bytes, void* stream) {
  if (!logits || !d_tokens || !d_parent || !d_argmax || !d_accepted || !d_bonus || !ws)
    return SWIFTSPEC_INVALID_ARG;
  if (T < 1 || V < 1 || ldl < V) return SWIFTSPEC_INVALID_ARG;
  if (T > SWIFTSPEC_MAX_TREE) return SWIFTSPEC_UNSUPPORTED;
  if (!aligned16(logits) || ldl % 8) return SWIFTSPEC_MISALIGNED;
  if (ws_bytes < swiftspec_greedy_accept_workspace_bytes(T)) return SWIFTSPEC_WORKSPACE_TOO_SMALL;
  ss::launch_greedy_accept(logits, ldl, T, V, d_tokens, d_parent, d_argmax, d_accepted, d_bonus, d_path_len,
                           ws, static_cast<char*>(ws) + kHeader, S(stream));
  return check_launch();
}

size_t swiftspec_topk_logprobs_workspace_bytes(int32_t n) {
  if (n < 1 || n > SWIFTSPEC_MAX_TREE) return kHeader;
  return kHeader + align_up(ss::topk_logprobs_part_bytes(n));
}

int swiftspec_topk_logprobs(const uint16_t* logits, int32_t ldl, int32_t n, int32_t V, int32_t k,
                            int32_t* d_tokens, float* d_logprobs, void* ws, size_t ws_bytes, void* stream) {
  if (!logits || !d_tokens || !d_logprobs || !ws) return SWIFTSPEC_INVALID_ARG;
  if (n < 1 || V < 1 || ldl < V || k < 1 || k > V) return SWIFTSPEC_INVALID_ARG;
  if (n > SWIFTSPEC_MAX_TREE || k > 8) return SWIFTSPEC_UNSUPPORTED;
  if (!aligned16(logits) || ldl % 8) return SWIFTSPEC_MISALIGNED;
  if (ws_bytes < swiftspec_topk_logprobs_workspace_bytes(n)) return SWIFTSPEC_WORKSPACE_TOO_SMALL;
  ss::launch_topk_logprobs(logits, ldl, n, V, k, d_tokens, d_logprobs, ws, static_cast<char*>(ws) + kHeader,
                           S(stream));
  return check_launch();
}

size_t swiftspec_verify_layer_workspace_bytes(const swiftspec_dims* dims, int32_t T) {
  if (!dims || T < 1 || T > SWIFTSPEC_MAX_TREE) return kHeader;
  return layer_ws(dims, T).total;
}

int swiftspec_verify_layer_workspace_layout(const swiftspec_dims* dims, int32_t T, size_t* offsets) {
  if (!dims || !offsets || T < 1 || T > SWIFTSPEC_MAX_TREE) return SWIFTSPEC_INVALID_ARG;
  const LayerWs w = layer_ws(dims, T);
  offsets[0] = w.qkv;
  offsets[1] = w.o;
  offsets[2] = w.h;
  offsets[3] = w.m;
  return SWIFTSPEC_OK;
}

// Synchronous argument checks of one decoder layer (nothing is launched).
static int check_layer(const swiftspec_layer* Lw, const swiftspec_dims* d, int32_t T) {
  if (!Lw->attn_norm || !Lw->mlp_norm || !Lw->k_cache || !Lw->v_cache) return SWIFTSPEC_INVALID_ARG;
  if (T < 1 || d->H < 1 || d->Hq < 1 || d->Hkv < 1 || d->F < 1 || d->S_max < T) return SWIFTSPEC_INVALID_ARG;
  if (T > SWIFTSPEC_MAX_TREE || (d->D != 64 && d->D != 128) || d->Hq % d->Hkv) return SWIFTSPEC_UNSUPPORTED;
  const int H = d->H, Hd = d->Hq * d->D, Nqkv = (d->Hq + 2 * d->Hkv) * d->D, F = d->F;
  if (!attn_counters_fit(T, d->Hq, d->Hkv)) return SWIFTSPEC_UNSUPPORTED;
  int rc;
  if ((rc = check_w4(&Lw->wqkv)) || (rc = check_w4(&Lw->wo)) || (rc = check_w4(&Lw->wgate)) ||
      (rc = check_w4(&Lw->wup)) || (rc = check_w4(&Lw->wdown)))
    return rc;
  if (Lw->wqkv.K != H || Lw->wqkv.N != Nqkv || Lw->wo.K != Hd || Lw->wo.N != H ||
      Lw->wgate.K != H || Lw->wgate.N != F || Lw->wup.K != H || Lw->wup.N != F ||
      Lw->wdown.K != F || Lw->wdown.N != H)
    return SWIFTSPEC_INVALID_ARG;
  if (!aligned16(Lw->attn_norm) || !aligned16(Lw->mlp_norm) || !aligned16(Lw->k_cache) ||
      !aligned16(Lw->v_cache))
    return SWIFTSPEC_MISALIGNED;
  return SWIFTSPEC_OK;
}

// Enqueue one checked decoder layer on `st`.
static void enqueue_layer(const swiftspec_layer* Lw, const swiftspec_dims* d, uint16_t* hidden, int32_t T,
                          const int32_t* d_prefix_len, const int32_t* d_parent, const float* rope,
                          void* ws, hipStream_t st) {
  const int H = d->H, Hd = d->Hq * d->D, Nqkv = (d->Hq + 2 * d->Hkv) * d->D, F = d->F;
  const LayerWs w = layer_ws(d, T);
  char* base = static_cast<char*>(ws);
  auto at = [&](size_t off) { return reinterpret_cast<uint16_t*>(base + off); };
  uint16_t *qkv = at(w.qkv), *o = at(w.o), *h = at(w.h), *m = at(w.m);
  uint16_t *xn_p = at(w.xn_p), *o_p = at(w.o_p), *hn_p = at(w.hn_p), *m_p = at(w.m_p);
  float* part = reinterpret_cast<float*>(base + w.part);
  // the RMSNorms in front of the QKV and the FFN projections run with them
  // (swiftspec_rmsnorm_w4a16_gemm / _swiglu)
  const NormIn n_attn{hidden, H, Lw->attn_norm, d->eps}, n_mlp{h, H, Lw->mlp_norm, d->eps};
  run_norm_gemm(&Lw->wqkv, nullptr, n_attn, T, qkv, Nqkv, nullptr, xn_p, ws, part, st);
  run_attention(qkv, Nqkv, qkv + Hd, qkv + Hd + d->Hkv * d->D, Nqkv, Lw->k_cache, Lw->v_cache,
                d->S_max, d_prefix_len, d_parent, T, d->Hq, d->Hkv, d->D, rope,
                1.0f / std::sqrt((float)d->D), o, Hd, o_p, ws, part, st);
  run_gemm(&Lw->wo, nullptr, o_p, T, h, H, nullptr, hidden, H, ws, part, st);
  run_norm_gemm(&Lw->wgate, &Lw->wup, n_mlp, T, m, F, m_p, hn_p, ws, part, st);
  run_gemm(&Lw->wdown, nullptr, m_p, T, hidden, H, nullptr, h, H, ws, part, st);
}

int swiftspec_verify_layer(const swiftspec_layer* Lw, const swiftspec_dims* d, uint16_t* hidden,
                           int32_t T, const int32_t* d_prefix_len, const int32_t* d_parent,
                           const float* rope, void* ws, size_t ws_bytes, void* stream) {
  if (!Lw || !d || !hidden || !d_prefix_len || !d_parent || !rope || !ws) return SWIFTSPEC_INVALID_ARG;
  int rc = check_layer(Lw, d, T);
  if (rc) return rc;
  if (!aligned16(hidden) || !aligned16(ws)) return SWIFTSPEC_MISALIGNED;
  if (ws_bytes < layer_ws(d, T).total) return SWIFTSPEC_WORKSPACE_TOO_SMALL;
  enqueue_layer(Lw, d, hidden, T, d_prefix_len, d_parent, rope, ws, S(stream));
  return check_launch();
}

size_t swiftspec_verify_step_workspace_bytes(const swiftspec_dims* dims, int32_t T, int32_t V) {
  if (!dims || T < 1 || T > SWIFTSPEC_MAX_TREE) return kHeader;
  const size_t layer = layer_ws(dims, T).total;
  const size_t head = V > 0 ? swiftspec_lm_head_workspace_bytes(T, dims->H, V) : 0;
  return layer > head ? layer : head;
}

int swiftspec_verify_step(const swiftspec_layer* layers, int32_t n_layers, const swiftspec_dims* d,
                          uint16_t* hidden, int32_t T, const int32_t* d_prefix_len,
                          const int32_t* d_parent, const float* rope, const uint16_t* final_norm,
                          const uint16_t* lm_head, int32_t V, uint16_t* logits, void* ws,
                          size_t ws_bytes, void* stream) {
  if (!layers || !d || !hidden || !d_prefix_len || !d_parent || !rope || !ws) return SWIFTSPEC_INVALID_ARG;
  if (n_layers < 0 || V < 0 || (n_layers == 0 && V == 0)) return SWIFTSPEC_INVALID_ARG;
  if (T < 1) return SWIFTSPEC_INVALID_ARG;
  if (T > SWIFTSPEC_MAX_TREE) return SWIFTSPEC_UNSUPPORTED;
  int rc;
  for (int l = 0; l < n_layers; ++l)
    if ((rc = check_layer(&layers[l], d, T))) return rc;
  if (V > 0) {
    if (!final_norm || !lm_head || !logits) return SWIFTSPEC_INVALID_ARG;
    if (d->H < 1) return SWIFTSPEC_INVALID_ARG;
    if (d->H % 128 || V % 16) return SWIFTSPEC_UNSUPPORTED;
    if (!aligned16(final_norm) || !aligned16(lm_head)) return SWIFTSPEC_MISALIGNED;
  }
  if (!aligned16(hidden) || !aligned16(ws)) return SWIFTSPEC_MISALIGNED;
  if (ws_bytes < swiftspec_verify_step_workspace_bytes(d, T, V)) return SWIFTSPEC_WORKSPACE_TOO_SMALL;
  hipStream_t st = S(stream);
  for (int l = 0; l < n_layers; ++l) enqueue_layer(&layers[l], d, hidden, T, d_prefix_len, d_parent, rope, ws, st);
  if (V > 0) {
    uint16_t* xn = reinterpret_cast<uint16_t*>(static_cast<char*>(ws) + kHeader);
    ss::launch_rmsnorm(hidden, T, d->H, d->H, final_norm, d->eps, xn, d->H, nullptr, st);
    ss::launch_lm_head(xn, T, d->H, lm_head, V, logits, V, st);
  }
  return check_launch();
}

size_t swiftspec_lm_head_workspace_bytes(int32_t M, int32_t H, int32_t V) {
  (void)V;
  if (M < 1 || H < 1) return kHeader;
  return kHeader + align_up((size_t)M * H * 2);
}

int swiftspec_lm_head(const uint16_t* h, int32_t M, int32_t H, const uint16_t* gamma, float eps,
                      const uint16_t* W, int32_t V, uint16_t* logits, void* ws, size_t ws_bytes,
                      void* stream) {
  if (!h || !gamma || !W || !logits || !ws) return SWIFTSPEC_INVALID_ARG;
  if (M < 1 || H < 1 || V < 1) return SWIFTSPEC_INVALID_ARG;
  if (M > SWIFTSPEC_MAX_M || H % 128 || V % 16) return SWIFTSPEC_UNSUPPORTED;
  if (!aligned16(h) || !aligned16(gamma) || !aligned16(W) || !aligned16(ws)) return SWIFTSPEC_MISALIGNED;
  if (ws_bytes < swiftspec_lm_head_workspace_bytes(M, H, V)) return SWIFTSPEC_WORKSPACE_TOO_SMALL;
  uint16_t* xn = reinterpret_cast<uint16_t*>(static_cast<char*>(ws) + kHeader);
  ss::launch_rmsnorm(h, M, H, H, gamma, eps, xn, H, nullptr, S(stream));
  ss::launch_lm_head(xn, M, H, W, V, logits, V, S(stream));
  return check_launch();
}

struct swiftspec_graph {
  hipGraph_t graph;
  hipGraphExec_t exec;
};

int swiftspec_graph_begin(void* stream) {
  if (!stream) return SWIFTSPEC_INVALID_ARG;
  return hip_status(hipStreamBeginCapture(S(stream), hipStreamCaptureModeThreadLocal));
}

int swiftspec_graph_end(void* stream, swiftspec_graph** out) {
  if (!stream || !out) return SWIFTSPEC_INVALID_ARG;
  hipGraph_t g = nullptr;
  int rc = hip_status(hipStreamEndCapture(S(stream), &g));
  if (rc) return rc;
  hipGraphExec_t ex = nullptr;
  rc = hip_status(hipGraphInstantiate(&ex, g, nullptr, nullptr, 0));
  if (rc) {
    (void)hipGraphDestroy(g);
    return rc;
  }
  swiftspec_graph* r = new (std::nothrow) swiftspec_graph{g, ex};
  if (!r) {
    (void)hipGraphExecDestroy(ex);
    (void)hipGraphDestroy(g);
    return SWIFTSPEC_INVALID_ARG;
  }
  *out = r;
  return SWIFTSPEC_OK;
}

int swiftspec_graph_launch(swiftspec_graph* g, void* stream) {
  if (!g) return SWIFTSPEC_INVALID_ARG;
  return hip_status(hipGraphLaunch(g->exec, S(stream)));
}

int swiftspec_graph_destroy(swiftspec_graph* g) {
  if (!g) return SWIFTSPEC_INVALID_ARG;
  (void)hipGraphExecDestroy(g->exec);
  (void)hipGraphDestroy(g->graph);
  delete g;
  return SWIFTSPEC_OK;
}

}  // extern "C"
