// The allocation-free variant of the head entry point, for callers that cannot allocate device
// memory (code under HIP graph capture, tight serving loops, harnesses that forbid hipMalloc): its
// temporaries (pooled features, logit gradients and per-sample losses, B (C + K + 1) floats) live in
// a fixed file-scope device array instead of the caller's scratch workspace.
//
// Each GPU the library runs on holds its own copy of the array until the process ends.  Host code
// never passes the array's name to a kernel (on the host it is only a stand-in for the symbol):
// the first call on a device, with that device current, looks up the array's device address with
// hipGetSymbolAddress and keeps it per device; every later call on that device uses that address.
// Calls on one GPU share the array, so calls that overlap in time on one GPU race.  Nothing in the
// array has to start at zero: the head's first kernel writes every value its second kernel reads.
#include <hip/hip_runtime.h>

#include <cstdint>
#include <mutex>

#include "pnn.h"
#include "pnn_internal.h"

namespace {

constexpr size_t SCRATCH_FLOATS = size_t(1) << 20;   // 4 MiB per device
constexpr int MAX_DEVICES = 64;

}  // namespace

static __device__ __align__(256) float scratch[SCRATCH_FLOATS];

namespace {

std::mutex g_lock;
float* g_scratch_ptr[MAX_DEVICES] = {};

// Device address of this device's copy of `scratch`, looked up once per device (the device must be
// current); nullptr when the lookup fails.
float* device_scratch() {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= MAX_DEVICES) return nullptr;
  std::lock_guard<std::mutex> g(g_lock);
  if (g_scratch_ptr[dev] == nullptr) {
    void* ptr = nullptr;
    if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || ptr == nullptr) return nullptr;
    g_scratch_ptr[dev] = (float*)ptr;
  }
  return g_scratch_ptr[dev];
}

inline bool al(const void* p, uintptr_t a) { return ((uintptr_t)p & (a - 1)) == 0; }

}  // namespace

extern "C" pnn_status pnn_head_fwd_bwd_noalloc(pnn_plan* plan, const void* ytilde, const float* eps,
                                               const int32_t* labels, float* logits, float* loss,
                                               void* D_N, float* deps, void* stream) {
  if (plan == nullptr || ytilde == nullptr || eps == nullptr || labels == nullptr || loss == nullptr ||
      D_N == nullptr || deps == nullptr)
    return PNN_ERR_NULL;
  if (!al(ytilde, 16) || !al(eps, 16) || !al(D_N, 16) || !al(deps, 16) || !al(labels, 4) ||
      !al(logits, 4) || !al(loss, 4))
    return PNN_ERR_ALIGN;
  int B = 0, HW = 0, C = 0, K = 0, dtype = 0;
  pnn::head_geometry(plan, &B, &HW, &C, &K, &dtype);
  if (K > 4096 || C > 8192) return PNN_ERR_UNSUPPORTED;
  if ((size_t)B * ((size_t)C + K + 1) > SCRATCH_FLOATS) return PNN_ERR_TOO_LARGE;
  float* s = device_scratch();
  if (s == nullptr) return PNN_ERR_HIP;
  const int e = pnn::launch_head(ytilde, eps, labels, logits, loss, D_N, deps, s, B, HW, C, K, dtype,
                                 nullptr, (hipStream_t)stream);
  return e ? PNN_ERR_HIP : PNN_OK;
}
