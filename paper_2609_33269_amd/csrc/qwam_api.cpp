// C ABI of libqwam: argument validation and dispatch to the HIP kernels.
// Every check runs on the host before any HIP call; device memory is never
// dereferenced here.
#include <hip/hip_runtime.h>

#include <atomic>
#include <cstdarg>
#include <cstdint>
#include <cstdio>

#include "../../include/qwam.h"
#include "qwam_internal.h"

namespace {

thread_local char g_err[512] = "";

qwam_status fail(qwam_status s, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  std::vsnprintf(g_err, sizeof(g_err), fmt, ap);
  va_end(ap);
  return s;
}

qwam_status ok() {
  g_err[0] = '\0';
  return QWAM_OK;
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

#define QWAM_REQUIRE_PTR(p)                                                              \
  do {                                                                                   \
    if ((p) == nullptr) return fail(QWAM_ERR_INVALID_ARG, "%s: %s is NULL", fn, #p);     \
    if (!aligned16(p)) return fail(QWAM_ERR_MISALIGNED, "%s: %s is not 16-byte aligned", fn, #p); \
  } while (0)

constexpr int32_t kMaxK = 65536;
constexpr int32_t kMaxN = 1 << 20;
constexpr int32_t kMaxM = 1 << 20;

qwam_status check_kn(const char* fn, int32_t K, int32_t N, int32_t group) {
  if (group != QWAM_GROUP && group != 32)
    return fail(QWAM_ERR_INVALID_ARG, "%s: group must be 64 or 32 (got %d)", fn, group);
  if (K <= 0 || K % QWAM_GROUP != 0) return fail(QWAM_ERR_INVALID_ARG, "%s: K must be a positive multiple of 64 (got %d)", fn, K);
  if (N <= 0 || N % 16 != 0) return fail(QWAM_ERR_INVALID_ARG, "%s: N must be a positive multiple of 16 (got %d)", fn, N);
  if (K > kMaxK) return fail(QWAM_ERR_UNSUPPORTED, "%s: K = %d exceeds %d", fn, K, kMaxK);
  if (N > kMaxN) return fail(QWAM_ERR_UNSUPPORTED, "%s: N = %d exceeds %d", fn, N, kMaxN);
  return QWAM_OK;
}

qwam_status check_layer(const char* fn, const qwam_layer* L, bool need_branch) {
  if (L == nullptr) return fail(QWAM_ERR_INVALID_ARG, "%s: layer is NULL", fn);
  qwam_status s = check_kn(fn, L->K, L->N, L->group);
  if (s != QWAM_OK) return s;
  if (need_branch && !(L->r == 16 || L->r == 32 || L->r == 48 || L->r == 64))
    return fail(QWAM_ERR_UNSUPPORTED, "%s: rank r must be 16, 32, 48 or 64 (got %d)", fn, L->r);
  const int32_t B = L->hadamard;
  if (B != 0 && (B < 16 || B > 1024 || (B & (B - 1)) != 0 || L->K % B != 0))
    return fail(QWAM_ERR_INVALID_ARG, "%s: hadamard must be 0 or a power of two in [16, 1024] dividing K (got %d)",
                fn, B);
  return QWAM_OK;
}

qwam_status check_m(const char* fn, int32_t M) {
  if (M <= 0) return fail(QWAM_ERR_INVALID_ARG, "%s: M must be >= 1 (got %d)", fn, M);
  if (M > kMaxM) return fail(QWAM_ERR_UNSUPPORTED, "%s: M = %d exceeds %d", fn, M, kMaxM);
  return QWAM_OK;
}

// The device count is queried once per process (a query per call would add
// host time to every launch, which small layers notice).
qwam_status check_device(const char* fn) {
  static std::atomic<int> visible{-1};
  int n = visible.load(std::memory_order_relaxed);
  if (n < 0) {
    int c = 0;
    if (hipGetDeviceCount(&c) != hipSuccess) {
      (void)hipGetLastError();
      c = 0;
    }
    visible.store(c, std::memory_order_relaxed);
    n = c;
  }
  if (n <= 0) return fail(QWAM_ERR_NO_DEVICE, "%s: no HIP device visible", fn);
  return QWAM_OK;
}

qwam_status launched(const char* fn, hipError_t e) {
  if (e != hipSuccess) return fail(QWAM_ERR_HIP, "%s: kernel launch failed: %s", fn, hipGetErrorString(e));
  return ok();
}

}  // namespace

extern "C" {

qwam_status qwam_pack_weights(int32_t K, int32_t N, int32_t group, const float* R, const float* smooth,
                              uint8_t* wq, float* ws, uint32_t* wsp, float* inv_smooth, void* stream) {
  const char* fn = "qwam_pack_weights";
  qwam_status s = check_kn(fn, K, N, group);
  if (s != QWAM_OK) return s;
  QWAM_REQUIRE_PTR(R);
  QWAM_REQUIRE_PTR(smooth);
  QWAM_REQUIRE_PTR(wq);
  QWAM_REQUIRE_PTR(ws);
  QWAM_REQUIRE_PTR(wsp);
  QWAM_REQUIRE_PTR(inv_smooth);
  if ((s = check_device(fn)) != QWAM_OK) return s;
  return launched(fn, qwam::launch_pack_weights(K, N, group, R, smooth, wq, ws, wsp, inv_smooth,
                                                static_cast<hipStream_t>(stream)));
}

}  // extern "C"

namespace {

qwam_status quantize_act_common(const char* fn, bool deflate, const qwam_layer* L, int32_t M,
                                const uint16_t* x, uint8_t* xq, float* xs, uint16_t* t, void* stream) {
  qwam_status s = check_layer(fn, L, true);
  if (s != QWAM_OK) return s;
  if ((s = check_m(fn, M)) != QWAM_OK) return s;
  QWAM_REQUIRE_PTR(L->inv_smooth);
  QWAM_REQUIRE_PTR(L->L1t);
  QWAM_REQUIRE_PTR(L->L1f);
  if (deflate) QWAM_REQUIRE_PTR(L->L1);
  QWAM_REQUIRE_PTR(x);
  QWAM_REQUIRE_PTR(xq);
  QWAM_REQUIRE_PTR(xs);
  QWAM_REQUIRE_PTR(t);
  if ((s = check_device(fn)) != QWAM_OK) return s;
  const hipStream_t st = static_cast<hipStream_t>(stream);
  if (L->hadamard != 0)
    return launched(fn, qwam::launch_quantize_act_rotated(M, L->K, L->r, L->group, L->hadamard, deflate, x,
                                                          L->inv_smooth, L->L1t, L->L1f, deflate ? L->L1 : nullptr,
                                                          xq, xs, t, st));
  if (deflate)
    return launched(fn, qwam::launch_quantize_act_deflated(M, L->K, L->r, L->group, x, L->inv_smooth, L->L1f, L->L1,
                                                           xq, xs, t, st));
  return launched(fn, qwam::launch_quantize_act(M, L->K, L->r, L->group, x, L->inv_smooth, L->L1f, xq, xs, t, st));
}

}  // namespace

extern "C" {

qwam_status qwam_quantize_act(const qwam_layer* L, int32_t M, const uint16_t* x, uint8_t* xq, float* xs,
                              uint16_t* t, void* stream) {
  return quantize_act_common("qwam_quantize_act", false, L, M, x, xq, xs, t, stream);
}

qwam_status qwam_quantize_act_deflated(const qwam_layer* L, int32_t M, const uint16_t* x, uint8_t* xq,
                                       float* xs, uint16_t* t, void* stream) {
  return quantize_act_common("qwam_quantize_act_deflated", true, L, M, x, xq, xs, t, stream);
}

qwam_status qwam_asp_linear(const qwam_layer* L, int32_t M, const uint8_t* xq, const float* xs,
                            const uint16_t* t, uint16_t* y, void* stream) {
  const char* fn = "qwam_asp_linear";
  qwam_status s = check_layer(fn, L, true);
  if (s != QWAM_OK) return s;
  if ((s = check_m(fn, M)) != QWAM_OK) return s;
  QWAM_REQUIRE_PTR(L->wq);
  QWAM_REQUIRE_PTR(L->ws);
  QWAM_REQUIRE_PTR(L->wsp);
  QWAM_REQUIRE_PTR(L->L2t);
  if (L->bias != nullptr && !aligned16(L->bias))
    return fail(QWAM_ERR_MISALIGNED, "%s: bias is not 16-byte aligned", fn);
  QWAM_REQUIRE_PTR(xq);
  QWAM_REQUIRE_PTR(xs);
  QWAM_REQUIRE_PTR(t);
  QWAM_REQUIRE_PTR(y);
  // the kernel addresses each scale array with 32-bit byte offsets
  if (static_cast<int64_t>(M) * (L->K / L->group) >= (int64_t(1) << 29) ||
      static_cast<int64_t>(L->N) * (L->K / L->group) >= (int64_t(1) << 29))
    return fail(QWAM_ERR_UNSUPPORTED, "%s: M*K/group and N*K/group must be below 2^29", fn);
  if ((s = check_device(fn)) != QWAM_OK) return s;
  return launched(fn, qwam::launch_asp_gemm(M, L->N, L->K, L->r, L->group, xq, xs, t, L->wq, L->ws, L->wsp, L->L2t,
                                            L->bias, y, static_cast<hipStream_t>(stream)));
}

qwam_status qwam_debug_group_partials(const qwam_layer* L, int32_t M, const uint8_t* xq, int32_t* P,
                                      void* stream) {
  const char* fn = "qwam_debug_group_partials";
  qwam_status s = check_layer(fn, L, false);
  if (s != QWAM_OK) return s;
  if ((s = check_m(fn, M)) != QWAM_OK) return s;
  QWAM_REQUIRE_PTR(L->wq);
  QWAM_REQUIRE_PTR(xq);
  QWAM_REQUIRE_PTR(P);
  if (static_cast<int64_t>(M) * L->N * (L->K / L->group) > (int64_t(1) << 34))
    return fail(QWAM_ERR_UNSUPPORTED, "%s: M*N*K/group too large for a partials dump", fn);
  if ((s = check_device(fn)) != QWAM_OK) return s;
  return launched(fn, qwam::launch_group_partials(M, L->N, L->K, L->group, xq, L->wq, P,
                                                  static_cast<hipStream_t>(stream)));
}

qwam_status qwam_asp_layer(const qwam_layer* L, int32_t M, const uint16_t* x, uint16_t* y, uint8_t* xq, float* xs,
                           uint16_t* t, void* stream) {
  const char* fn = "qwam_asp_layer";
  qwam_status s = check_layer(fn, L, true);
  if (s != QWAM_OK) return s;
  if ((s = check_m(fn, M)) != QWAM_OK) return s;
  if (M > qwam::kSmallM) return fail(QWAM_ERR_UNSUPPORTED, "%s: M = %d exceeds %d", fn, M, qwam::kSmallM);
  if (L->r != 16 && L->r != 32) return fail(QWAM_ERR_UNSUPPORTED, "%s: rank r must be 16 or 32 (got %d)", fn, L->r);
  if (L->group != QWAM_GROUP || L->hadamard != 0)
    return fail(QWAM_ERR_UNSUPPORTED, "%s: group 64 without rotation only", fn);
  if (L->K > 16384) return fail(QWAM_ERR_UNSUPPORTED, "%s: K = %d exceeds 16384", fn, L->K);
  QWAM_REQUIRE_PTR(L->wq);
  QWAM_REQUIRE_PTR(L->ws);
  QWAM_REQUIRE_PTR(L->inv_smooth);
  QWAM_REQUIRE_PTR(L->L1t);
  QWAM_REQUIRE_PTR(L->L2t);
  if (L->bias != nullptr && !aligned16(L->bias))
    return fail(QWAM_ERR_MISALIGNED, "%s: bias is not 16-byte aligned", fn);
  QWAM_REQUIRE_PTR(x);
  QWAM_REQUIRE_PTR(y);
  const int given = (xq != nullptr) + (xs != nullptr) + (t != nullptr);
  if (given != 0 && given != 3) return fail(QWAM_ERR_INVALID_ARG, "%s: xq, xs and t must be all NULL or all set", fn);
  if (given == 3) {
    QWAM_REQUIRE_PTR(xq);
    QWAM_REQUIRE_PTR(xs);
    QWAM_REQUIRE_PTR(t);
  }
  if ((s = check_device(fn)) != QWAM_OK) return s;
  return launched(fn, qwam::launch_asp_layer_small(M, L->N, L->K, L->r, x, L->inv_smooth, L->L1t, L->wq, L->ws,
                                                   L->L2t, L->bias, y, xq, xs, t, static_cast<hipStream_t>(stream)));
}

qwam_status qwam_aog_accumulate(int32_t d, int32_t n, const uint16_t* gT, float* A, void* stream) {
  const char* fn = "qwam_aog_accumulate";
  if (d < 16 || d % 16 != 0)
    return fail(QWAM_ERR_INVALID_ARG, "%s: d must be a positive multiple of 16 (got %d)", fn, d);
  if (n < 64 || n % 64 != 0)
    return fail(QWAM_ERR_INVALID_ARG, "%s: n must be a positive multiple of 64 (got %d)", fn, n);
  if (d > 16384) return fail(QWAM_ERR_UNSUPPORTED, "%s: d = %d exceeds 16384", fn, d);
  if (static_cast<int64_t>(d) * n >= (int64_t(1) << 30))
    return fail(QWAM_ERR_UNSUPPORTED, "%s: d * n must be below 2^30", fn);
  QWAM_REQUIRE_PTR(gT);
  QWAM_REQUIRE_PTR(A);
  qwam_status s = check_device(fn);
  if (s != QWAM_OK) return s;
  return launched(fn, qwam::launch_aog_accumulate(d, n, gT, A, static_cast<hipStream_t>(stream)));
}

}  // extern "C"

namespace {

qwam_status check_eig(const char* fn, int32_t d, int32_t r, int32_t iters, float scale, int32_t hadamard) {
  if (d < 128 || d % 64 != 0)
    return fail(QWAM_ERR_INVALID_ARG, "%s: d must be a multiple of 64, at least 128 (got %d)", fn, d);
  if (d > 16384) return fail(QWAM_ERR_UNSUPPORTED, "%s: d = %d exceeds 16384", fn, d);
  if (r < 1 || r > qwam::kEigMaxRank)
    return fail(QWAM_ERR_UNSUPPORTED, "%s: r must be in [1, %d] (got %d)", fn, qwam::kEigMaxRank, r);
  if (iters < 0 || iters > 1000) return fail(QWAM_ERR_INVALID_ARG, "%s: iters must be in [0, 1000] (got %d)", fn, iters);
  if (!(scale > 0.0f) || !(scale < 3.0e38f))
    return fail(QWAM_ERR_INVALID_ARG, "%s: scale must be positive and finite", fn);
  if (hadamard != 0 && (hadamard < 16 || hadamard > 1024 || (hadamard & (hadamard - 1)) != 0 || d % hadamard != 0))
    return fail(QWAM_ERR_INVALID_ARG, "%s: hadamard must be 0 or a power of two in [16, 1024] dividing d (got %d)",
                fn, hadamard);
  return QWAM_OK;
}

}  // namespace

extern "C" {

int64_t qwam_aog_protected_basis_workspace(int32_t d, int32_t r) {
  if (check_eig("qwam_aog_protected_basis_workspace", d, r, 0, 1.0f, 0) != QWAM_OK) return -1;
  ok();
  return qwam::eig_workspace_bytes(d, r);
}

qwam_status qwam_aog_protected_basis(int32_t d, int32_t r, int32_t iters, const float* A, float scale,
                                     const float* lam, int32_t hadamard, float* V, float* evals, void* workspace,
                                     int64_t workspace_bytes, void* stream) {
  const char* fn = "qwam_aog_protected_basis";
  qwam_status s = check_eig(fn, d, r, iters, scale, hadamard);
  if (s != QWAM_OK) return s;
  QWAM_REQUIRE_PTR(A);
  QWAM_REQUIRE_PTR(V);
  QWAM_REQUIRE_PTR(evals);
  QWAM_REQUIRE_PTR(workspace);
  if (lam != nullptr && !aligned16(lam)) return fail(QWAM_ERR_MISALIGNED, "%s: lam is not 16-byte aligned", fn);
  const int64_t need = qwam::eig_workspace_bytes(d, r);
  if (workspace_bytes < need)
    return fail(QWAM_ERR_INVALID_ARG, "%s: workspace of %lld bytes is below the %lld needed", fn,
                static_cast<long long>(workspace_bytes), static_cast<long long>(need));
  if ((s = check_device(fn)) != QWAM_OK) return s;
  return launched(fn, qwam::launch_aog_eig(d, r, iters, A, scale, lam, hadamard, V, evals, workspace,
                                           static_cast<hipStream_t>(stream)));
}

const char* qwam_last_error(void) { return g_err; }

const char* qwam_status_string(qwam_status s) {
  switch (s) {
    case QWAM_OK: return "QWAM_OK";
    case QWAM_ERR_INVALID_ARG: return "QWAM_ERR_INVALID_ARG";
    case QWAM_ERR_UNSUPPORTED: return "QWAM_ERR_UNSUPPORTED";
    case QWAM_ERR_MISALIGNED: return "QWAM_ERR_MISALIGNED";
    case QWAM_ERR_NO_DEVICE: return "QWAM_ERR_NO_DEVICE";
    case QWAM_ERR_HIP: return "QWAM_ERR_HIP";
  }
  return "QWAM_ERR_UNKNOWN";
}

int32_t qwam_abi_version(void) { return QWAM_ABI_VERSION; }

}  // extern "C"
