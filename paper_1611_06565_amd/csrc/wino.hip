// libwino device side: argument checks of the entry points of
// include/wino.h that enqueue work, and the choice of a size's launches.
// Plans, sizes and launch grids come from the host-side planner (plan.cpp);
// the kernels are instantiated per size in the sizes_*.hip units.
#include <hip/hip_runtime.h>

#include <cstdint>
#include <mutex>

#include "kernels.hpp"
#include "launch.hpp"
#include "plan.hpp"
#include "wino.h"

using namespace wino;

namespace wino {

// Compute units of the current device (cached per device); the planner sizes
// the product's tail split with it.
int device_cu_count() {
  static int cached[64] = {0};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 0;
  if (cached[dev] == 0) {
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return 0;
    cached[dev] = n;
  }
  return cached[dev];
}

}  // namespace wino

// Scratch of wino_forward_noalloc: the forward's workspace (V, then the
// product's partial outputs) for callers that cannot allocate device memory.
// One copy per device, held until the process ends.  In host code `scratch`
// names a host-side stand-in, so only its device address (from
// hipGetSymbolAddress, kept per device below) is ever passed to kernels.
static __device__ __align__(256) float scratch[WINO_NOALLOC_SCRATCH_BYTES / sizeof(float)];

namespace {

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

// Device address of `scratch` on the current device, looked up once per
// device (with that device current) and kept.
std::mutex scratch_mu;
void* scratch_dev[64] = {};

wino_status scratch_address(void** out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return WINO_EDEVICE;
  std::lock_guard<std::mutex> lock(scratch_mu);
  if (scratch_dev[dev] == nullptr) {
    void* ptr = nullptr;
    if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || ptr == nullptr) return WINO_EDEVICE;
    scratch_dev[dev] = ptr;
  }
  *out = scratch_dev[dev];
  return WINO_OK;
}

// The launch table of a plan's size (the planner only makes plans of
// compiled sizes).
const SizeOps* ops_of(const wino_plan_s& p) {
  if (p.aniso) return size_ops_ax(p.mv[0], p.mv[1]);
#define WINO_PICK(N_, M_, R_) \
  if (p.N == N_ && p.m == M_ && p.r == R_) return size_ops_##N_##_##M_##_##R_(p.const_mats);
  WINO_SIZES(WINO_PICK)
#undef WINO_PICK
  if (p.kind == 4) return size_ops_a8(p.m, p.r, p.const_mats);
  return nullptr;
}

}  // namespace

extern "C" {

wino_status wino_transform_filter(const wino_plan_t* p, const float* w, float* U, void* stream) {
  if (p == nullptr || w == nullptr || U == nullptr) return WINO_EINVAL;
  if (!aligned16(w) || !aligned16(U)) return WINO_EINVAL;
  const hipStream_t s = static_cast<hipStream_t>(stream);
  const SizeOps* ops = ops_of(*p);
  return ops ? ops->filter(*p, w, U, false, s) : WINO_EUNSUPPORTED;
}

wino_status wino_weight_gradient(const wino_plan_t* p, const float* x, const float* dy, float* dw, void* ws,
                                 size_t ws_bytes, void* stream) {
  if (p == nullptr || x == nullptr || dy == nullptr || dw == nullptr || ws == nullptr) return WINO_EINVAL;
  if (!aligned16(x) || !aligned16(dy) || !aligned16(dw) || !aligned16(ws)) return WINO_EINVAL;
  if (!p->wgrad_ok) return WINO_EUNSUPPORTED;
  if (ws_bytes < wino_weight_gradient_workspace_bytes(p)) return WINO_EWORKSPACE;
  const hipStream_t s = static_cast<hipStream_t>(stream);
  float* w = static_cast<float*>(ws);
  const SizeOps* ops = ops_of(*p);
  return ops ? ops->wgrad(*p, x, dy, dw, w, s) : WINO_EUNSUPPORTED;
}

wino_status wino_transform_filter_adjoint(const wino_plan_t* p, const float* w, float* U, void* stream) {
  if (p == nullptr || w == nullptr || U == nullptr) return WINO_EINVAL;
  if (!aligned16(w) || !aligned16(U)) return WINO_EINVAL;
  const hipStream_t s = static_cast<hipStream_t>(stream);
  const SizeOps* ops = ops_of(*p);
  return ops ? ops->filter(*p, w, U, true, s) : WINO_EUNSUPPORTED;
}

wino_status wino_transform_input(const wino_plan_t* p, const float* x, void* ws, size_t ws_bytes,
                                 void* stream) {
  if (p == nullptr || x == nullptr || ws == nullptr) return WINO_EINVAL;
  if (!aligned16(x) || !aligned16(ws)) return WINO_EINVAL;
  if (ws_bytes < wino_workspace_bytes(p)) return WINO_EWORKSPACE;
  const hipStream_t s = static_cast<hipStream_t>(stream);
  float* V = static_cast<float*>(ws);
  const SizeOps* ops = ops_of(*p);
  return ops ? ops->input(*p, x, V, s) : WINO_EUNSUPPORTED;
}

wino_status wino_gemm_inverse_ex(const wino_plan_t* p, void* ws, size_t ws_bytes, const float* U,
                                 const float* bias, float* y, void* stream) {
  if (p == nullptr || ws == nullptr || U == nullptr || y == nullptr) return WINO_EINVAL;
  if (!aligned16(ws) || !aligned16(U) || !aligned16(y)) return WINO_EINVAL;
  if (bias != nullptr && (reinterpret_cast<uintptr_t>(bias) & 3u) != 0) return WINO_EINVAL;
  if (ws_bytes < wino_workspace_bytes(p)) return WINO_EWORKSPACE;
  const hipStream_t s = static_cast<hipStream_t>(stream);
  const float* V = static_cast<const float*>(ws);
  float* part = p->nparts > 1 ? static_cast<float*>(ws) + p->v_floats : nullptr;
  const SizeOps* ops = ops_of(*p);
  return ops ? ops->gemm(*p, V, part, U, bias, y, s) : WINO_EUNSUPPORTED;
}

wino_status wino_gemm_inverse(const wino_plan_t* p, void* ws, size_t ws_bytes, const float* U,
                              float* y, void* stream) {
  return wino_gemm_inverse_ex(p, ws, ws_bytes, U, nullptr, y, stream);
}

wino_status wino_forward_ex(const wino_plan_t* p, const float* x, const float* U, const float* bias,
                            float* y, void* ws, size_t ws_bytes, void* stream) {
  if (p == nullptr || x == nullptr || U == nullptr || y == nullptr) return WINO_EINVAL;
  if (!aligned16(x) || !aligned16(U) || !aligned16(y)) return WINO_EINVAL;
  if (bias != nullptr && (reinterpret_cast<uintptr_t>(bias) & 3u) != 0) return WINO_EINVAL;
  if (p->fused) {
    // the input transform runs inside the product: no workspace
    const SizeOps* ops = ops_of(*p);
    if (ops == nullptr || ops->fused == nullptr) return WINO_EUNSUPPORTED;
    return ops->fused(*p, x, U, bias, y, static_cast<hipStream_t>(stream));
  }
  if (ws == nullptr) return WINO_EINVAL;
  if (!aligned16(ws)) return WINO_EINVAL;
  if (ws_bytes < wino_workspace_bytes(p)) return WINO_EWORKSPACE;
  wino_status st = wino_transform_input(p, x, ws, ws_bytes, stream);
  if (st != WINO_OK) return st;
  return wino_gemm_inverse_ex(p, ws, ws_bytes, U, bias, y, stream);
}

wino_status wino_forward(const wino_plan_t* p, const float* x, const float* U, float* y, void* ws,
                         size_t ws_bytes, void* stream) {
  return wino_forward_ex(p, x, U, nullptr, y, ws, ws_bytes, stream);
}

wino_status wino_forward_noalloc(const wino_plan_t* p, const float* x, const float* U, const float* bias,
                                 float* y, void* stream) {
  if (p == nullptr || x == nullptr || U == nullptr || y == nullptr) return WINO_EINVAL;
  if (!aligned16(x) || !aligned16(U) || !aligned16(y)) return WINO_EINVAL;
  if (bias != nullptr && (reinterpret_cast<uintptr_t>(bias) & 3u) != 0) return WINO_EINVAL;
  if (wino_forward_workspace_bytes(p) > WINO_NOALLOC_SCRATCH_BYTES) return WINO_EWORKSPACE;
  void* ws = nullptr;
  const wino_status st = scratch_address(&ws);
  if (st != WINO_OK) return st;
  // every word of V and of the partial outputs that the product reads is
  // written first by this call's own kernels: nothing needs clearing
  return wino_forward_ex(p, x, U, bias, y, ws, WINO_NOALLOC_SCRATCH_BYTES, stream);
}

wino_status wino_forward_pool(const wino_plan_t* p, const float* x, const float* U, const float* bias,
                              const int32_t* window, float* y, void* ws, size_t ws_bytes, void* stream) {
  if (p == nullptr || x == nullptr || U == nullptr || y == nullptr || window == nullptr) return WINO_EINVAL;
  if (!aligned16(x) || !aligned16(U) || !aligned16(y)) return WINO_EINVAL;
  if (bias != nullptr && (reinterpret_cast<uintptr_t>(bias) & 3u) != 0) return WINO_EINVAL;
  for (int i = 0; i < 3; ++i)
    if (window[i] < 1) return WINO_EINVAL;
  int pool = 0;
  if (window[0] == 1 && window[1] == 2 && window[2] == 2) pool = 1;
  else if (window[0] == 2 && window[1] == 2 && window[2] == 2) pool = 2;
  else return WINO_EUNSUPPORTED;
  if (p->N != 3) return WINO_EUNSUPPORTED;
  const SizeOps* ops = ops_of(*p);
  if (ops == nullptr) return WINO_EUNSUPPORTED;
  // the max-pool rides on the F(4^3) forward's epilogue (fused, or the
  // two-stage product) or on the F(2^3) product's (window (2, 2, 2): one tile)
  if (p->fused ? ops->fused == nullptr : ops->gemm_pool == nullptr) return WINO_EUNSUPPORTED;
  if (p->m == 2 && pool != 2) return WINO_EUNSUPPORTED;
  for (int i = 0; i < 3; ++i)
    if (p->Y[i] / window[i] < 1) return WINO_EINVAL;
  const hipStream_t s = static_cast<hipStream_t>(stream);
  if (p->fused) return launch_fused43(*p, p->const_mats, x, U, bias, y, s, pool);
  if (ws == nullptr) return WINO_EINVAL;
  if (!aligned16(ws)) return WINO_EINVAL;
  if (ws_bytes < wino_workspace_bytes(p)) return WINO_EWORKSPACE;
  float* V = static_cast<float*>(ws);
  float* part = p->nparts > 1 ? V + p->v_floats : nullptr;
  const wino_status st = ops->input(*p, x, V, s);
  if (st != WINO_OK) return st;
  return ops->gemm_pool(*p, V, part, U, bias, y, pool, s);
}

wino_status wino_maxpool3d(const int64_t* dims, const int32_t* window, const float* x, float* y,
                           void* stream) {
  if (dims == nullptr || window == nullptr || x == nullptr || y == nullptr) return WINO_EINVAL;
  if (!aligned16(x) || !aligned16(y)) return WINO_EINVAL;
  PoolGeom q{};
  const wino_status st = pool_geometry(dims, window, &q);
  if (st != WINO_OK) return st;
  PoolArgs a{};
  a.lead = q.lead;
  for (int i = 0; i < 3; ++i) { a.X[i] = q.X[i]; a.Y[i] = q.Y[i]; a.p[i] = q.p[i]; }
  a.total = q.total;
  const hipStream_t s = static_cast<hipStream_t>(stream);
  if (q.pair) hipLaunchKernelGGL(k_maxpool3d_pair, dim3(q.grid), dim3(256), 0, s, x, y, a);
  else hipLaunchKernelGGL(k_maxpool3d, dim3(q.grid), dim3(256), 0, s, x, y, a);
  return wino::launch_status();
}

}  // extern "C"
