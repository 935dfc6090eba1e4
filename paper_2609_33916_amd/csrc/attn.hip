// C ABI of the attention library (declared in include/attn_mi355x.h):
// argument validation, kernel selection by (dtype, d, causal) and launches.
// Validation happens entirely on the host before any HIP call, so every
// error code can be exercised without a GPU.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <atomic>
#include <cmath>
#include <cstdint>
#include <limits>
#include <mutex>
#include <type_traits>

#include "attn_mi355x.h"
#include "kernels.hpp"
#include "launch.hpp"

namespace {

using attn::bf16;

constexpr int kFwdBQ = attn::kDqBQ;  // queries per forward / dQ workgroup
constexpr int kFwdPpBQ = 256;        // queries per ping-pong forward workgroup
constexpr int kDkvBKV = 128;  // keys per float32 dK/dV workgroup

bool aligned(const void* p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) & (a - 1)) == 0; }

int check_common(int B, int H, int n, int d, float scale, int causal, int dtype) {
  if (B < 1 || H < 1 || n < 1) return ATTN_E_SHAPE;
  if (dtype != ATTN_BF16 && dtype != ATTN_F32) return ATTN_E_UNSUPPORTED;
  if (d != 32 && d != 64 && d != 128) return ATTN_E_UNSUPPORTED;
  if (!std::isfinite(scale)) return ATTN_E_ARG;
  if (causal != 0 && causal != 1) return ATTN_E_ARG;
  // grid sizes and per-head element offsets must fit in int
  const long long heads = (long long)B * H;
  const long long tiles = (n + 63) / 64;
  if ((long long)n * d > std::numeric_limits<int>::max()) return ATTN_E_SHAPE;
  if (heads * tiles > std::numeric_limits<int>::max()) return ATTN_E_SHAPE;
  return ATTN_OK;
}

struct ScaleParts {
  float sl2;
  float abs_scale;
  uint32_t qflip;  // per-dword sign mask for Q elements
};

ScaleParts split_scale(float scale, int dtype) {
  ScaleParts s;
  s.abs_scale = std::fabs(scale);
  // a zero scale would turn masked scores (-inf) into NaN; a floor far below
  // any representable score difference keeps them at -inf and leaves P exact
  s.sl2 = std::fmax(s.abs_scale * attn::kLog2e, 1e-30f);
  const bool neg = std::signbit(scale) && scale != 0.f;
  s.qflip = neg ? (dtype == ATTN_BF16 ? 0x80008000u : 0x80000000u) : 0u;
  return s;
}

// bf16 at d = 128: the ping-pong forward (256 queries per eight-wave
// workgroup); otherwise the four-wave forward (128 queries per workgroup).
// At d <= 64 a tile's softmax arithmetic outlasts its products, so the
// ping-pong phases would wait on the softmax.
template <typename T, int D, bool CAUSAL>
void launch_fwd(attn::FwdArgs a, int heads, hipStream_t st) {
  if constexpr (std::is_same<T, bf16>::value && D == 128) {
    a.ntiles = (a.n + kFwdPpBQ - 1) / kFwdPpBQ;
    a.nblocks = heads * a.ntiles;
    hipLaunchKernelGGL((attn::fwd_pp_kernel<D, CAUSAL>), dim3(a.nblocks), dim3(512), 0, st, a);
  } else {
    a.ntiles = (a.n + kFwdBQ - 1) / kFwdBQ;
    a.nblocks = heads * a.ntiles;
    hipLaunchKernelGGL((attn::fwd_kernel<T, D, CAUSAL>), dim3(a.nblocks), dim3(256), 0, st, a);
  }
}

// bf16 dK/dV and dQ launch from dkdv.hip and bwd.hip (launch.hpp); float32
// uses the 32-key-per-wave dK/dV kernel and the dQ kernel instantiated here.
template <typename T, int D, bool CAUSAL, bool MAT = false>
void launch_dkdv(attn::BwdArgs a, int heads, hipStream_t st) {
  if constexpr (std::is_same<T, bf16>::value) {
    attn::launch_dkdv16<D, CAUSAL, MAT, false>(a, heads, st);
  } else {
    a.ntiles = (a.n + kDkvBKV - 1) / kDkvBKV;
    a.nblocks = heads * a.ntiles;
    hipLaunchKernelGGL((attn::dkdv_kernel<T, D, CAUSAL, MAT>), dim3(a.nblocks), dim3(256), 0, st, a);
  }
}

template <typename T, int D, bool CAUSAL, bool MAT = false>
void launch_dq(attn::BwdArgs a, int heads, hipStream_t st) {
  if constexpr (std::is_same<T, bf16>::value) {
    attn::launch_dq16<D, CAUSAL, MAT>(a, heads, st);
  } else {
    a.ntiles = (a.n + kFwdBQ - 1) / kFwdBQ;
    a.nblocks = heads * a.ntiles;
    hipLaunchKernelGGL((attn::dq_kernel<T, D, CAUSAL, MAT>), dim3(a.nblocks), dim3(256), 0, st, a);
  }
}

// atomic-dQ backward (bfloat16): the dK/dV kernel also accumulates dQ. It
// is compiled here, with the default scheduler: under the iterative-ILP
// strategy its n = 2048, d = 128 unmasked case runs 1.4x slower.
template <typename T, int D, bool CAUSAL>
void launch_dkdv_aq(attn::BwdArgs a, int heads, hipStream_t st) {
  if constexpr (std::is_same<T, bf16>::value) {
    constexpr int nw = attn::dkdv16_nw(D, false, true), bkv = attn::dkdv16_bkv(D, false, true);
    a.ntiles = (a.n + bkv - 1) / bkv;
    a.nblocks = heads * a.ntiles;
    hipLaunchKernelGGL((attn::dkdv16_kernel<D, CAUSAL, nw, attn::kDkv16BQ, false, true, 1>), dim3(a.nblocks),
                       dim3(64 * nw), 0, st, a);
  }
}

template <typename T, int D, bool CAUSAL>
void launch_mat_fwd(attn::FwdArgs a, int heads, hipStream_t st) {
  a.ntiles = (a.n + kFwdBQ - 1) / kFwdBQ;
  a.nblocks = heads * a.ntiles;
  hipLaunchKernelGGL((attn::mat_fwd_kernel<T, D, CAUSAL>), dim3(a.nblocks), dim3(256), 0, st, a);
}

template <typename T, int D, bool C>
struct PrepL {
  static void run(attn::PrepArgs a, int, hipStream_t st) {
    constexpr int rpb = 256 / (D / attn::Elem<T>::CH);
    const long long blocks = (a.rows + rpb - 1) / rpb;
    hipLaunchKernelGGL((attn::bwd_prep_kernel<T, D>), dim3((unsigned)blocks), dim3(256), 0, st, a);
  }
};
template <typename T, int D, bool C>
struct FwdL { static void run(attn::FwdArgs a, int heads, hipStream_t st) { launch_fwd<T, D, C>(a, heads, st); } };
template <typename T, int D, bool C>
struct DkvL { static void run(attn::BwdArgs a, int heads, hipStream_t st) { launch_dkdv<T, D, C>(a, heads, st); } };
template <typename T, int D, bool C>
struct DqL { static void run(attn::BwdArgs a, int heads, hipStream_t st) { launch_dq<T, D, C>(a, heads, st); } };

template <typename T, int D, bool C>
struct MatFwdL { static void run(attn::FwdArgs a, int heads, hipStream_t st) { launch_mat_fwd<T, D, C>(a, heads, st); } };
template <typename T, int D, bool C>
struct MatDkvL { static void run(attn::BwdArgs a, int heads, hipStream_t st) { launch_dkdv<T, D, C, true>(a, heads, st); } };
template <typename T, int D, bool C>
struct MatDqL { static void run(attn::BwdArgs a, int heads, hipStream_t st) { launch_dq<T, D, C, true>(a, heads, st); } };

template <typename T, int D, bool C>
struct DkvAqL { static void run(attn::BwdArgs a, int heads, hipStream_t st) { launch_dkdv_aq<T, D, C>(a, heads, st); } };

template <template <typename, int, bool> class F, typename T, typename Args>
void by_d(int d, int causal, Args a, int heads, hipStream_t st) {
  if (d == 32) { causal ? F<T, 32, true>::run(a, heads, st) : F<T, 32, false>::run(a, heads, st); }
  else if (d == 64) { causal ? F<T, 64, true>::run(a, heads, st) : F<T, 64, false>::run(a, heads, st); }
  else { causal ? F<T, 128, true>::run(a, heads, st) : F<T, 128, false>::run(a, heads, st); }
}

template <template <typename, int, bool> class F, typename Args>
void run_dispatch(int dtype, int d, int causal, Args a, int heads, hipStream_t st) {
  if (dtype == ATTN_BF16) by_d<F, bf16>(d, causal, a, heads, st);
  else by_d<F, float>(d, causal, a, heads, st);
}

// Decode: split plan. A workgroup owns (batch, cache head, up to 32 query
// heads, one split of the keys); the keys are split until there are about two
// workgroups per compute unit, each split a whole number of 128-key tiles.
struct DecodePlan {
  int qchunks, nsplit, chunk;
};
constexpr int kDecodeTargetWGs = 512;
DecodePlan decode_plan(int B, int Hq, int Hkv, int n, int append) {
  DecodePlan p;
  const int G = Hq / Hkv;
  p.qchunks = (G + 31) / 32;
  const long long groups = (long long)B * Hkv * p.qchunks;
  const long long keys = (long long)n + append;
  const long long tiles = std::max<long long>(1, (keys + 127) / 128);
  long long ns = std::max<long long>(1, (kDecodeTargetWGs + groups - 1) / groups);
  ns = std::min(ns, tiles);
  const long long per = (tiles + ns - 1) / ns;     // tiles per split
  p.chunk = (int)(per * 128);
  p.nsplit = (int)((tiles + per - 1) / per);
  return p;
}

// Scratch of attn_fwd_bwd_noalloc: the two float32 rows per query (D and
// the base-2 log-sum-exp) that attn_fwd_bwd keeps in the caller's workspace,
// in a fixed device array instead. Each GPU holds its own copy from the
// library's first use on it until the process ends. In host code the name
// `scratch` is only a stand-in for the symbol: its device address (one per
// GPU) comes from hipGetSymbolAddress and is the only form passed to kernels.
constexpr size_t kScratchBytes = size_t(16) << 20;
static __device__ __align__(256) float scratch[kScratchBytes / sizeof(float)];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
std::atomic<void*> g_scratch_ptr[kMaxDevices];

// Device address of the current GPU's scratch array (looked up once per
// device, with that device current); nullptr if the lookup failed.
void* scratch_ptr() {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return nullptr;
  void* p = g_scratch_ptr[dev].load(std::memory_order_acquire);
  if (p) return p;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  p = g_scratch_ptr[dev].load(std::memory_order_relaxed);
  if (!p) {
    void* q = nullptr;
    if (hipGetSymbolAddress(&q, HIP_SYMBOL(scratch)) != hipSuccess || !q) return nullptr;
    p = q;
    g_scratch_ptr[dev].store(p, std::memory_order_release);
  }
  return p;
}

// Row stride of the materialised attention matrix: n rounded up to a
// multiple of 128, so every key tile the kernels touch lies inside the row.
constexpr int kMatMaxN = 1 << 20;
long long mat_lda(int n) { return ((long long)n + 127) / 128 * 128; }

}  // namespace

extern "C" {

size_t attn_workspace_bytes(int B, int H, int n, int d) {
  (void)d;
  if (B < 1 || H < 1 || n < 1) return 0;
  return 2 * (size_t)B * (size_t)H * (size_t)n * sizeof(float);
}

int attn_fwd(const void* Q, const void* K, const void* V, void* O, float* L,
             int B, int H, int n, int d, float scale, int causal, int dtype, void* stream) {
  if (!Q || !K || !V || !O || !L) return ATTN_E_NULL;
  int rc = check_common(B, H, n, d, scale, causal, dtype);
  if (rc != ATTN_OK) return rc;
  if (!aligned(Q, 16) || !aligned(K, 16) || !aligned(V, 16) || !aligned(O, 16) || !aligned(L, 4))
    return ATTN_E_ALIGN;
  const ScaleParts sp = split_scale(scale, dtype);
  attn::FwdArgs a{};
  a.q = Q; a.k = K; a.v = V; a.dout = nullptr;
  a.o = O; a.lse = L; a.dvec = nullptr; a.lse2 = nullptr;
  a.head_stride = (long long)n * d;
  a.n = n;
  a.sl2 = sp.sl2;
  a.qflip = sp.qflip;
  hipStream_t st = static_cast<hipStream_t>(stream);
  (void)hipGetLastError();
  run_dispatch<FwdL>(dtype, d, causal, a, B * H, st);
  if (hipGetLastError() != hipSuccess) return ATTN_E_HIP;
  return ATTN_OK;
}

static int fwd_bwd_impl(const void* Q, const void* K, const void* V, const void* dO,
                        void* O, float* L, void* dQ, void* dK, void* dV,
                        void* workspace, size_t workspace_bytes,
                        int B, int H, int n, int d, float scale, int causal, int dtype,
                        void* stream, void* const* events) {
  if (!Q || !K || !V || !dO || !O || !L || !dQ || !dK || !dV || !workspace) return ATTN_E_NULL;
  int rc = check_common(B, H, n, d, scale, causal, dtype);
  if (rc != ATTN_OK) return rc;
  if (!aligned(Q, 16) || !aligned(K, 16) || !aligned(V, 16) || !aligned(dO, 16) ||
      !aligned(O, 16) || !aligned(dQ, 16) || !aligned(dK, 16) || !aligned(dV, 16) ||
      !aligned(L, 4) || !aligned(workspace, 4))
    return ATTN_E_ALIGN;
  if (workspace_bytes < attn_workspace_bytes(B, H, n, d)) return ATTN_E_WORKSPACE;
  if (events) {
    for (int i = 0; i < 4; ++i)
      if (!events[i]) return ATTN_E_NULL;
  }
  const ScaleParts sp = split_scale(scale, dtype);
  float* dvec = static_cast<float*>(workspace);
  float* lse2 = dvec + (size_t)B * H * n;
  hipStream_t st = static_cast<hipStream_t>(stream);
  (void)hipGetLastError();
  auto mark = [&](int i) {
    return !events || hipEventRecord(static_cast<hipEvent_t>(events[i]), st) == hipSuccess;
  };

  attn::FwdArgs f{};
  f.q = Q; f.k = K; f.v = V; f.dout = dO;
  f.o = O; f.lse = L; f.dvec = dvec; f.lse2 = lse2;
  f.head_stride = (long long)n * d;
  f.n = n;
  f.sl2 = sp.sl2;
  f.qflip = sp.qflip;

  attn::BwdArgs b{};
  b.q = Q; b.k = K; b.v = V; b.dout = dO;
  b.lse2 = lse2; b.dvec = dvec;
  b.dq = dQ; b.dk = dK; b.dv = dV;
  b.head_stride = (long long)n * d;
  b.n = n;
  b.sl2 = sp.sl2;
  b.dk_scale = scale;
  b.dq_scale = scale;
  b.qflip = sp.qflip;

  if (!mark(0)) return ATTN_E_HIP;
  run_dispatch<FwdL>(dtype, d, causal, f, B * H, st);
  if (hipGetLastError() != hipSuccess || !mark(1)) return ATTN_E_HIP;
  run_dispatch<DkvL>(dtype, d, causal, b, B * H, st);
  if (hipGetLastError() != hipSuccess || !mark(2)) return ATTN_E_HIP;
  run_dispatch<DqL>(dtype, d, causal, b, B * H, st);
  if (hipGetLastError() != hipSuccess || !mark(3)) return ATTN_E_HIP;
  return ATTN_OK;
}

int attn_fwd_bwd(const void* Q, const void* K, const void* V, const void* dO,
                 void* O, float* L, void* dQ, void* dK, void* dV,
                 void* workspace, size_t workspace_bytes,
                 int B, int H, int n, int d, float scale, int causal, int dtype, void* stream) {
  return fwd_bwd_impl(Q, K, V, dO, O, L, dQ, dK, dV, workspace, workspace_bytes,
                      B, H, n, d, scale, causal, dtype, stream, nullptr);
}

size_t attn_noalloc_max_rows(void) { return kScratchBytes / (2 * sizeof(float)); }

int attn_fwd_bwd_noalloc(const void* Q, const void* K, const void* V, const void* dO,
                         void* O, float* L, void* dQ, void* dK, void* dV,
                         int B, int H, int n, int d, float scale, int causal, int dtype, void* stream) {
  // the same argument checks as attn_fwd_bwd, before the size limit and the
  // first HIP call
  if (!Q || !K || !V || !dO || !O || !L || !dQ || !dK || !dV) return ATTN_E_NULL;
  int rc = check_common(B, H, n, d, scale, causal, dtype);
  if (rc != ATTN_OK) return rc;
  if ((long long)B * H * (long long)n > (long long)attn_noalloc_max_rows()) return ATTN_E_SCRATCH;
  void* ws = scratch_ptr();
  if (!ws) return ATTN_E_HIP;
  return fwd_bwd_impl(Q, K, V, dO, O, L, dQ, dK, dV, ws, kScratchBytes, B, H, n, d, scale, causal, dtype,
                      stream, nullptr);
}

int attn_bwd(const void* Q, const void* K, const void* V, const void* O, const float* L,
             const void* dO, void* dQ, void* dK, void* dV,
             void* workspace, size_t workspace_bytes,
             int B, int H, int n, int d, float scale, int causal, int dtype, void* stream) {
  if (!Q || !K || !V || !O || !L || !dO || !dQ || !dK || !dV || !workspace) return ATTN_E_NULL;
  int rc = check_common(B, H, n, d, scale, causal, dtype);
  if (rc != ATTN_OK) return rc;
  if (!aligned(Q, 16) || !aligned(K, 16) || !aligned(V, 16) || !aligned(O, 16) ||
      !aligned(dO, 16) || !aligned(dQ, 16) || !aligned(dK, 16) || !aligned(dV, 16) ||
      !aligned(L, 4) || !aligned(workspace, 4))
    return ATTN_E_ALIGN;
  if (workspace_bytes < attn_workspace_bytes(B, H, n, d)) return ATTN_E_WORKSPACE;
  const ScaleParts sp = split_scale(scale, dtype);
  float* dvec = static_cast<float*>(workspace);
  float* lse2 = dvec + (size_t)B * H * n;
  hipStream_t st = static_cast<hipStream_t>(stream);
  (void)hipGetLastError();

  attn::PrepArgs p{};
  p.o = O; p.dout = dO; p.lse = L; p.dvec = dvec; p.lse2 = lse2;
  p.rows = (long long)B * H * n;
  run_dispatch<PrepL>(dtype, d, causal, p, B * H, st);
  if (hipGetLastError() != hipSuccess) return ATTN_E_HIP;

  attn::BwdArgs b{};
  b.q = Q; b.k = K; b.v = V; b.dout = dO;
  b.lse2 = lse2; b.dvec = dvec;
  b.dq = dQ; b.dk = dK; b.dv = dV;
  b.head_stride = (long long)n * d;
  b.n = n;
  b.sl2 = sp.sl2;
  b.dk_scale = scale;
  b.dq_scale = scale;
  b.qflip = sp.qflip;
  run_dispatch<DkvL>(dtype, d, causal, b, B * H, st);
  if (hipGetLastError() != hipSuccess) return ATTN_E_HIP;
  run_dispatch<DqL>(dtype, d, causal, b, B * H, st);
  if (hipGetLastError() != hipSuccess) return ATTN_E_HIP;
  return ATTN_OK;
}

int attn_fwd_bwd_timed(const void* Q, const void* K, const void* V, const void* dO,
                       void* O, float* L, void* dQ, void* dK, void* dV,
                       void* workspace, size_t workspace_bytes,
                       int B, int H, int n, int d, float scale, int causal, int dtype,
                       void* stream, void* const* events) {
  return fwd_bwd_impl(Q, K, V, dO, O, L, dQ, dK, dV, workspace, workspace_bytes,
                      B, H, n, d, scale, causal, dtype, stream, events);
}

size_t attn_mat_bytes(int B, int H, int n, int dtype) {
  if (B < 1 || H < 1 || n < 1 || n > kMatMaxN) return 0;
  if (dtype != ATTN_BF16 && dtype != ATTN_F32) return 0;
  const size_t e = dtype == ATTN_BF16 ? 2 : 4;
  return (size_t)B * (size_t)H * (size_t)n * (size_t)mat_lda(n) * e;
}

static int check_mat(const void* P, size_t p_bytes, int B, int H, int n, int dtype) {
  if (n > kMatMaxN) return ATTN_E_SHAPE;
  if (!aligned(P, 16)) return ATTN_E_ALIGN;
  if (p_bytes < attn_mat_bytes(B, H, n, dtype)) return ATTN_E_WORKSPACE;
  return ATTN_OK;
}

static attn::FwdArgs mat_fwd_args(const void* Q, const void* K, const void* V, const void* dO, void* O,
                                  float* L, void* P, float* dvec, float* lse2, int n, int d, float scale,
                                  int dtype) {
  const ScaleParts sp = split_scale(scale, dtype);
  attn::FwdArgs f{};
  f.q = Q; f.k = K; f.v = V; f.dout = dO;
  f.o = O; f.lse = L; f.dvec = dvec; f.lse2 = lse2;
  f.head_stride = (long long)n * d;
  f.n = n;
  f.sl2 = sp.sl2;
  f.qflip = sp.qflip;
  f.amat = P;
  f.lda = mat_lda(n);
  return f;
}

static attn::BwdArgs mat_bwd_args(const void* Q, const void* K, const void* V, const void* dO,
                                  const void* P, float* dvec, void* dQ, void* dK, void* dV, int n, int d,
                                  float scale, int dtype) {
  const ScaleParts sp = split_scale(scale, dtype);
  attn::BwdArgs b{};
  b.q = Q; b.k = K; b.v = V; b.dout = dO;
  b.lse2 = nullptr; b.dvec = dvec;
  b.dq = dQ; b.dk = dK; b.dv = dV;
  b.head_stride = (long long)n * d;
  b.n = n;
  b.sl2 = sp.sl2;
  b.dk_scale = scale;
  b.dq_scale = scale;
  b.qflip = sp.qflip;
  b.amat = P;
  b.lda = mat_lda(n);
  return b;
}

int attn_mat_fwd(const void* Q, const void* K, const void* V, void* O, float* L, void* P, size_t p_bytes,
                 int B, int H, int n, int d, float scale, int causal, int dtype, void* stream) {
  if (!Q || !K || !V || !O || !L || !P) return ATTN_E_NULL;
  int rc = check_common(B, H, n, d, scale, causal, dtype);
  if (rc != ATTN_OK) return rc;
  if (!aligned(Q, 16) || !aligned(K, 16) || !aligned(V, 16) || !aligned(O, 16) || !aligned(L, 4))
    return ATTN_E_ALIGN;
  rc = check_mat(P, p_bytes, B, H, n, dtype);
  if (rc != ATTN_OK) return rc;
  const attn::FwdArgs f = mat_fwd_args(Q, K, V, nullptr, O, L, P, nullptr, nullptr, n, d, scale, dtype);
  hipStream_t st = static_cast<hipStream_t>(stream);
  (void)hipGetLastError();
  run_dispatch<MatFwdL>(dtype, d, causal, f, B * H, st);
  if (hipGetLastError() != hipSuccess) return ATTN_E_HIP;
  return ATTN_OK;
}

int attn_mat_bwd(const void* Q, const void* K, const void* V, const void* O, const void* dO,
                 const void* P, size_t p_bytes, void* dQ, void* dK, void* dV,
                 void* workspace, size_t workspace_bytes,
                 int B, int H, int n, int d, float scale, int causal, int dtype, void* stream) {
  if (!Q || !K || !V || !O || !dO || !P || !dQ || !dK || !dV || !workspace) return ATTN_E_NULL;
  int rc = check_common(B, H, n, d, scale, causal, dtype);
  if (rc != ATTN_OK) return rc;
  if (!aligned(Q, 16) || !aligned(K, 16) || !aligned(V, 16) || !aligned(O, 16) ||
      !aligned(dO, 16) || !aligned(dQ, 16) || !aligned(dK, 16) || !aligned(dV, 16) ||
      !aligned(workspace, 4))
    return ATTN_E_ALIGN;
  rc = check_mat(P, p_bytes, B, H, n, dtype);
  if (rc != ATTN_OK) return rc;
  if (workspace_bytes < attn_workspace_bytes(B, H, n, d)) return ATTN_E_WORKSPACE;
  float* dvec = static_cast<float*>(workspace);
  hipStream_t st = static_cast<hipStream_t>(stream);
  (void)hipGetLastError();

  attn::PrepArgs p{};
  p.o = O; p.dout = dO; p.lse = nullptr; p.dvec = dvec; p.lse2 = nullptr;
  p.rows = (long long)B * H * n;
  run_dispatch<PrepL>(dtype, d, causal, p, B * H, st);
  if (hipGetLastError() != hipSuccess) return ATTN_E_HIP;
  const attn::BwdArgs b = mat_bwd_args(Q, K, V, dO, P, dvec, dQ, dK, dV, n, d, scale, dtype);
  run_dispatch<MatDkvL>(dtype, d, causal, b, B * H, st);
  if (hipGetLastError() != hipSuccess) return ATTN_E_HIP;
  run_dispatch<MatDqL>(dtype, d, causal, b, B * H, st);
  if (hipGetLastError() != hipSuccess) return ATTN_E_HIP;
  return ATTN_OK;
}

int attn_mat_fwd_bwd(const void* Q, const void* K, const void* V, const void* dO,
                     void* O, float* L, void* P, size_t p_bytes, void* dQ, void* dK, void* dV,
                     void* workspace, size_t workspace_bytes,
                     int B, int H, int n, int d, float scale, int causal, int dtype, void* stream) {
  if (!Q || !K || !V || !dO || !O || !L || !P || !dQ || !dK || !dV || !workspace) return ATTN_E_NULL;
  int rc = check_common(B, H, n, d, scale, causal, dtype);
  if (rc != ATTN_OK) return rc;
  if (!aligned(Q, 16) || !aligned(K, 16) || !aligned(V, 16) || !aligned(dO, 16) ||
      !aligned(O, 16) || !aligned(dQ, 16) || !aligned(dK, 16) || !aligned(dV, 16) ||
      !aligned(L, 4) || !aligned(workspace, 4))
    return ATTN_E_ALIGN;
  rc = check_mat(P, p_bytes, B, H, n, dtype);
  if (rc != ATTN_OK) return rc;
  if (workspace_bytes < attn_workspace_bytes(B, H, n, d)) return ATTN_E_WORKSPACE;
  float* dvec = static_cast<float*>(workspace);
  float* lse2 = dvec + (size_t)B * H * n;
  hipStream_t st = static_cast<hipStream_t>(stream);
  (void)hipGetLastError();
  const attn::FwdArgs f = mat_fwd_args(Q, K, V, dO, O, L, P, dvec, lse2, n, d, scale, dtype);
  run_dispatch<MatFwdL>(dtype, d, causal, f, B * H, st);
  if (hipGetLastError() != hipSuccess) return ATTN_E_HIP;
  const attn::BwdArgs b = mat_bwd_args(Q, K, V, dO, P, dvec, dQ, dK, dV, n, d, scale, dtype);
  run_dispatch<MatDkvL>(dtype, d, causal, b, B * H, st);
  if (hipGetLastError() != hipSuccess) return ATTN_E_HIP;
  run_dispatch<MatDqL>(dtype, d, causal, b, B * H, st);
  if (hipGetLastError() != hipSuccess) return ATTN_E_HIP;
  return ATTN_OK;
}

size_t attn_workspace_bytes_atomic(int B, int H, int n, int d) {
  if (B < 1 || H < 1 || n < 1 || (d != 32 && d != 64 && d != 128)) return 0;
  return attn_workspace_bytes(B, H, n, d) + (size_t)B * (size_t)H * (size_t)n * (size_t)d * sizeof(float);
}

int attn_fwd_bwd_atomic(const void* Q, const void* K, const void* V, const void* dO,
                        void* O, float* L, void* dQ, void* dK, void* dV,
                        void* workspace, size_t workspace_bytes,
                        int B, int H, int n, int d, float scale, int causal, int dtype, void* stream) {
  if (!Q || !K || !V || !dO || !O || !L || !dQ || !dK || !dV || !workspace) return ATTN_E_NULL;
  int rc = check_common(B, H, n, d, scale, causal, dtype);
  if (rc != ATTN_OK) return rc;
  if (dtype != ATTN_BF16) return ATTN_E_UNSUPPORTED;
  if (!aligned(Q, 16) || !aligned(K, 16) || !aligned(V, 16) || !aligned(dO, 16) ||
      !aligned(O, 16) || !aligned(dQ, 16) || !aligned(dK, 16) || !aligned(dV, 16) ||
      !aligned(L, 4) || !aligned(workspace, 16))
    return ATTN_E_ALIGN;
  if (workspace_bytes < attn_workspace_bytes_atomic(B, H, n, d)) return ATTN_E_WORKSPACE;
  const ScaleParts sp = split_scale(scale, dtype);
  const size_t rows = (size_t)B * H * n;
  // accumulator first: 16-byte aligned for the vector fill and finalize
  float* dqacc = static_cast<float*>(workspace);
  float* dvec = dqacc + rows * d;
  float* lse2 = dvec + rows;
  hipStream_t st = static_cast<hipStream_t>(stream);
  (void)hipGetLastError();

  const long long n8 = (long long)(rows * d / 8);
  hipLaunchKernelGGL(attn::zero_f32_kernel, dim3((unsigned)((n8 + 255) / 256)), dim3(256), 0, st, dqacc, n8);
  if (hipGetLastError() != hipSuccess) return ATTN_E_HIP;

  attn::FwdArgs f{};
  f.q = Q; f.k = K; f.v = V; f.dout = dO;
  f.o = O; f.lse = L; f.dvec = dvec; f.lse2 = lse2;
  f.head_stride = (long long)n * d;
  f.n = n;
  f.sl2 = sp.sl2;
  f.qflip = sp.qflip;
  run_dispatch<FwdL>(dtype, d, causal, f, B * H, st);
  if (hipGetLastError() != hipSuccess) return ATTN_E_HIP;

  attn::BwdArgs b{};
  b.q = Q; b.k = K; b.v = V; b.dout = dO;
  b.lse2 = lse2; b.dvec = dvec;
  b.dq = dQ; b.dk = dK; b.dv = dV;
  b.head_stride = (long long)n * d;
  b.n = n;
  b.sl2 = sp.sl2;
  b.dk_scale = scale;
  b.dq_scale = scale;
  b.qflip = sp.qflip;
  b.dqacc = dqacc;
  run_dispatch<DkvAqL>(dtype, d, causal, b, B * H, st);
  if (hipGetLastError() != hipSuccess) return ATTN_E_HIP;

  hipLaunchKernelGGL((attn::dq_finalize_kernel<bf16>), dim3((unsigned)((n8 + 255) / 256)), dim3(256), 0, st,
                     dqacc, static_cast<bf16*>(dQ), n8, scale);
  if (hipGetLastError() != hipSuccess) return ATTN_E_HIP;
  return ATTN_OK;
}

size_t attn_decode_workspace_bytes(int B, int Hq, int Hkv, int n, int d, int append) {
  if (B < 1 || Hq < 1 || Hkv < 1 || Hq % Hkv != 0 || n < 0 || (d != 32 && d != 64 && d != 128)) return 0;
  const DecodePlan p = decode_plan(B, Hq, Hkv, n, append ? 1 : 0);
  if (p.nsplit == 1) return 0;
  return (size_t)B * Hq * p.nsplit * (size_t)(d + 2) * sizeof(float);
}

int attn_decode(const void* q, const void* k_new, const void* v_new, void* k_cache, void* v_cache,
                const int* cache_lens, void* O, float* L, void* workspace, size_t workspace_bytes,
                int B, int Hq, int Hkv, int n, int n_cap, int d, float scale, int dtype, void* stream) {
  if (!q || !k_cache || !v_cache || !O) return ATTN_E_NULL;
  if ((k_new == nullptr) != (v_new == nullptr)) return ATTN_E_NULL;
  const int append = k_new ? 1 : 0;
  if (B < 1 || Hq < 1 || Hkv < 1 || n < 0 || n_cap < 1 || n_cap < n + append) return ATTN_E_SHAPE;
  if (Hq % Hkv != 0) return ATTN_E_SHAPE;
  if (dtype != ATTN_BF16 && dtype != ATTN_F32) return ATTN_E_UNSUPPORTED;
  if (dtype != ATTN_BF16) return ATTN_E_UNSUPPORTED;
  if (d != 32 && d != 64 && d != 128) return ATTN_E_UNSUPPORTED;
  if (!std::isfinite(scale)) return ATTN_E_ARG;
  if ((long long)B * Hkv * (long long)n_cap * d > (1LL << 46)) return ATTN_E_SHAPE;
  if ((long long)B * Hq * Hkv > std::numeric_limits<int>::max()) return ATTN_E_SHAPE;
  if (!aligned(q, 16) || !aligned(k_cache, 16) || !aligned(v_cache, 16) || !aligned(O, 16) ||
      (k_new && (!aligned(k_new, 16) || !aligned(v_new, 16))) || (L && !aligned(L, 4)) ||
      (cache_lens && !aligned(cache_lens, 4)))
    return ATTN_E_ALIGN;
  const DecodePlan plan = decode_plan(B, Hq, Hkv, n, append);
  const size_t need = attn_decode_workspace_bytes(B, Hq, Hkv, n, d, append);
  if (need > 0) {
    if (!workspace) return ATTN_E_NULL;
    if (!aligned(workspace, 16)) return ATTN_E_ALIGN;
    if (workspace_bytes < need) return ATTN_E_WORKSPACE;
  }
  if ((long long)B * Hkv * plan.qchunks > 65535) return ATTN_E_SHAPE;   // grid y limit
  const ScaleParts sp = split_scale(scale, dtype);
  attn::DecArgs a{};
  a.q = q; a.kc = k_cache; a.vc = v_cache; a.k_new = k_new; a.v_new = v_new;
  a.lens = cache_lens;
  a.part = static_cast<float*>(workspace);
  a.o = O; a.lse = L;
  a.rows = B * Hq;
  a.Hq = Hq; a.Hkv = Hkv; a.G = Hq / Hkv; a.n = n; a.n_cap = n_cap; a.append = append;
  a.chunk = plan.chunk; a.nsplit = plan.nsplit; a.qchunks = plan.qchunks;
  a.sl2 = sp.sl2;
  a.qflip = sp.qflip;
  hipStream_t st = static_cast<hipStream_t>(stream);
  (void)hipGetLastError();
  const dim3 grid(plan.nsplit, B * Hkv * plan.qchunks);
  a.fuse_append = append && plan.qchunks == 1;
  auto launch = [&](auto dtag) {
    constexpr int D = decltype(dtag)::value;
    if (append && !a.fuse_append) {
      const long long chunks = 2LL * B * Hkv * (D / 8);
      hipLaunchKernelGGL((attn::decode_append_kernel<bf16, D>), dim3((unsigned)((chunks + 255) / 256)), dim3(256),
                         0, st, a, B);
    }
    hipLaunchKernelGGL((attn::decode_kernel<D>), grid, dim3(256), 0, st, a);
    if (plan.nsplit > 1)
      hipLaunchKernelGGL((attn::decode_combine_kernel<bf16, D>), dim3((unsigned)(B * Hq)), dim3(256), 0,
                         st, a.part, O, L, B * Hq, plan.nsplit);
  };
  if (d == 32) launch(std::integral_constant<int, 32>{});
  else if (d == 64) launch(std::integral_constant<int, 64>{});
  else launch(std::integral_constant<int, 128>{});
  if (hipGetLastError() != hipSuccess) return ATTN_E_HIP;
  return ATTN_OK;
}

const char* attn_strerror(int code) {
  switch (code) {
    case ATTN_OK: return "success";
    case ATTN_E_NULL: return "a required pointer is NULL";
    case ATTN_E_SHAPE: return "B, H or n < 1, or the problem is too large to index";
    case ATTN_E_UNSUPPORTED: return "unsupported head dimension (d must be 32, 64 or 128) or dtype";
    case ATTN_E_ALIGN: return "a tensor is not 16-byte aligned (L and workspace: 4-byte)";
    case ATTN_E_WORKSPACE: return "workspace smaller than attn_workspace_bytes(), or P smaller than attn_mat_bytes()";
    case ATTN_E_HIP: return "the HIP runtime rejected a kernel launch";
    case ATTN_E_ARG: return "scale is not finite, or causal is not 0 or 1";
    case ATTN_E_SCRATCH:
      return "B * H * n exceeds attn_noalloc_max_rows(), the rows the fixed scratch of attn_fwd_bwd_noalloc holds";
    default: return "unknown attn status code";
  }
}

}  // extern "C"
