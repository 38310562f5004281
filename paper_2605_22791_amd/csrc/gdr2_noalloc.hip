// Allocation-free chunkwise forward, for callers that cannot allocate device
// memory (code under HIP graph capture, tight serving loops, harnesses that
// forbid allocation): gdr2_chunk_fwd with its workspace in one fixed array per
// device instead of a caller's buffer.
//
// The array is a file-scope __device__ object, so every GPU the library runs
// on holds its own copy (GDR2_NOALLOC_SCRATCH_BYTES) until the process ends.
// In host code its name stands for a host-side shadow, not a device address:
// the device address is looked up once per device with hipGetSymbolAddress,
// with that device current, and only that pointer is ever handed to kernels.
// The forward's kernels write every workspace byte they later read, so
// nothing in the array has to start at zero.  All calls on one GPU share its
// array: calls that overlap on one GPU (different streams or threads without
// ordering) race on it.

#include <hip/hip_runtime.h>

#include <cstdint>
#include <mutex>

#include "gdr2.h"

namespace {

constexpr size_t kScratchBytes = GDR2_NOALLOC_SCRATCH_BYTES;
constexpr int kMaxDevices = 64;

__device__ __align__(256) unsigned char scratch[kScratchBytes];

std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

bool ptr_ok(const void* x) { return x != nullptr && (reinterpret_cast<uintptr_t>(x) & 15u) == 0; }
bool opt_ptr_ok(const void* x) { return x == nullptr || (reinterpret_cast<uintptr_t>(x) & 15u) == 0; }

// Device address of the current device's array (looked up on its first use).
hipError_t scratch_ptr(void** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (g_scratch_ptr[dev] == nullptr) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (p == nullptr) return hipErrorInvalidSymbol;
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return hipSuccess;
}

}  // namespace

extern "C" gdr2_status gdr2_chunk_fwd_noalloc(const gdr2_problem* problem, const void* q, const void* k,
                                              const void* v, const float* log_alpha, const void* b,
                                              const void* w, const float* S0, void* o, float* S_T,
                                              hipStream_t stream) {
  // every argument is checked before the first HIP call, as in gdr2_chunk_fwd
  size_t need = 0;
  const gdr2_status s = gdr2_chunk_workspace_bytes(problem, 0, &need);
  if (s != GDR2_OK) return s;
  if (!ptr_ok(q) || !ptr_ok(k) || !ptr_ok(v) || !ptr_ok(log_alpha) || !ptr_ok(b) || !ptr_ok(w) || !ptr_ok(o) ||
      !opt_ptr_ok(S0) || !opt_ptr_ok(S_T))
    return GDR2_EINVAL;
  if (need > kScratchBytes) return GDR2_EWORKSPACE;
  void* ws = nullptr;
  if (scratch_ptr(&ws) != hipSuccess) return GDR2_EHIP;
  return gdr2_chunk_fwd(problem, q, k, v, log_alpha, b, w, S0, o, S_T, ws, kScratchBytes, stream);
}
