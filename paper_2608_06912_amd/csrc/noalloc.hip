// lapsum_forward_noalloc: the full-sort forward with its workspace in a
// file-scope device array instead of caller memory, for callers that cannot
// allocate (code under HIP graph capture, serving loops, harnesses that
// forbid hipMalloc).  It runs exactly the kernels of lapsum_forward.
//
// The array lives in this code object: every GPU the library runs on holds
// one copy of kScratchBytes at its own address until the process ends.  In
// host code the array's name is only a host-side stand-in, so its device
// address is looked up once per device with hipGetSymbolAddress (with that
// device current) and only that address is ever handed to kernels.
#include <hip/hip_runtime.h>
#include <math.h>

#include <mutex>

#include "../../include/lapsum.h"

namespace {

constexpr size_t kScratchBytes = static_cast<size_t>(LAPSUM_NOALLOC_SCRATCH_BYTES);
static_assert(kScratchBytes % 256 == 0, "scratch is a whole number of 256-byte blocks");

static __device__ __align__(256) unsigned char scratch[kScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_mu;
void* g_scratch_ptr[kMaxDevices] = {};

// The device address of `scratch` on the current device (looked up on the
// first call there and kept), or null on a runtime error.
void* scratch_on_current_device() {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return nullptr;
  std::lock_guard<std::mutex> g(g_mu);
  if (!g_scratch_ptr[dev]) {
    void* ptr = nullptr;
    if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || ptr == nullptr)
      return nullptr;
    g_scratch_ptr[dev] = ptr;
  }
  return g_scratch_ptr[dev];
}

}  // namespace

extern "C" int lapsum_forward_noalloc(const float* scores, int64_t batch, int64_t n, double k,
                                      double alpha, float* p, double* b, int32_t* perm_out,
                                      hipStream_t stream) {
  // the scalar checks of lapsum_forward come first, so that an invalid call
  // reports INVALID_ARG whatever its size
  if (!scores || !p || !b || batch < 1 || n < 1 || n > 2147483647LL) return LAPSUM_ERR_INVALID_ARG;
  if (!isfinite(k) || !(k > 0.0) || !(k < static_cast<double>(n)) || !isfinite(alpha) ||
      !(alpha < 0.0))
    return LAPSUM_ERR_INVALID_ARG;
  const size_t need = lapsum_forward_workspace_size(batch, n, perm_out != nullptr);
  if (need > kScratchBytes) return LAPSUM_ERR_WORKSPACE;
  void* ws = scratch_on_current_device();
  if (!ws) return LAPSUM_ERR_HIP;
  // the workspace's content on entry does not matter to lapsum_forward, so
  // nothing is cleared; no allocation happens below this point
  return lapsum_forward(scores, batch, n, k, alpha, p, b, perm_out, ws, kScratchBytes, stream);
}
