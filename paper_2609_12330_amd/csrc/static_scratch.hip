// Split-KV attention for callers that cannot allocate device memory (code
// under HIP graph capture, tight serving loops, harnesses that forbid
// hipMalloc): the same validation and kernels as ef_attention_splitkv, with
// the partial states and arrival counters placed in a scratch array of static
// device storage instead of a caller workspace.
//
// Each device the library runs on holds its own copy of the array from the
// moment this code object is loaded on it until the process ends; it is zero
// at load, so the arrival counters start at zero, and every completed call
// leaves them at zero again. In host code the array's name is only a
// host-side stand-in: its device address is looked up once per device (with
// that device current) and only that address is handed to the kernels.
#include <hip/hip_runtime.h>

#include <mutex>

#include "ef_attention.h"

namespace ef {
ef_status splitkv_into(const void* q, const void* k, const void* v, float* o, int B, int Hq,
                       int Hkv, int Sq, int Skv, int D, float scale, int causal,
                       int partition_size, void* workspace, size_t workspace_bytes, void* stream);
}  // namespace ef

namespace {

constexpr size_t kScratchBytes = EF_STATIC_SCRATCH_BYTES;
constexpr int kMaxDevices = 64;

__device__ __align__(256) unsigned char scratch[kScratchBytes];

std::mutex g_mutex;
void* g_scratch[kMaxDevices];  // device address of `scratch` per device; null until looked up

// Device address of the current device's scratch array.
hipError_t current_scratch(void** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_mutex);
  if (g_scratch[dev] == nullptr) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    g_scratch[dev] = p;
  }
  *out = g_scratch[dev];
  return hipSuccess;
}

}  // namespace

extern "C" {

ef_status ef_attention_splitkv_noalloc(const void* q, const void* k, const void* v, float* o,
                                       int B, int Hq, int Hkv, int Sq, int Skv, int D,
                                       float scale, int causal, int partition_size,
                                       void* stream) {
  // Validation without a workspace: an argument error is returned as such, a
  // call that needs no workspace (no query rows, or no keys) runs completely,
  // and any other call stops at the workspace check before anything is enqueued.
  const ef_status st = ef::splitkv_into(q, k, v, o, B, Hq, Hkv, Sq, Skv, D, scale, causal,
                                        partition_size, nullptr, 0, stream);
  if (st != EF_ERR_WORKSPACE_TOO_SMALL) return st;
  if (ef_attention_splitkv_workspace_size(B, Hq, Hkv, Sq, Skv, D, partition_size) > kScratchBytes)
    return EF_ERR_SCRATCH_TOO_SMALL;
  void* ws = nullptr;
  if (current_scratch(&ws) != hipSuccess) return EF_ERR_HIP;
  return ef::splitkv_into(q, k, v, o, B, Hq, Hkv, Sq, Skv, D, scale, causal, partition_size, ws,
                          kScratchBytes, stream);
}

}  // extern "C"
