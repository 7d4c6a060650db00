// stca_forward_noalloc: stca_forward with its workspace in a file-scope
// device array of this library instead of a caller-provided buffer, for
// callers that cannot allocate device memory.
//
// The array exists once per GPU (each device holds its own copy from the
// first call on it until the process ends).  Host code never passes the
// array's name to a kernel: its device address is looked up once per device
// with hipGetSymbolAddress, with that device current, and the forward runs on
// that address exactly as on a caller's workspace.  Nothing here allocates.
#include <mutex>

#include "common.h"

namespace {

constexpr size_t kScratchBytes = STCA_NOALLOC_SCRATCH_BYTES;
static_assert(kScratchBytes % 256 == 0, "scratch size keeps the workspace alignment");

static __device__ __align__(256) unsigned char scratch[kScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_mu;
void* g_ptr[kMaxDevices] = {};

// Device address of this device's scratch array (nullptr on failure).
void* scratch_ptr(int dev) {
  std::lock_guard<std::mutex> lock(g_mu);
  if (!g_ptr[dev]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || p == nullptr) return nullptr;
    g_ptr[dev] = p;
  }
  return g_ptr[dev];
}

}  // namespace

extern "C" stca_status_t stca_forward_noalloc(const stca_dims_t* dims, const stca_batch_t* batch, const void* hist,
                                              const void* tgt, const stca_weights_t* w, void* out, void* saved,
                                              hipStream_t stream) {
  // sizes first: a call that does not fit is rejected before anything is
  // looked up or launched (0 = invalid or unsupported arguments, which
  // stca_forward itself reports below)
  const size_t need = stca_workspace_size(dims, batch, 0);
  if (need > kScratchBytes) return STCA_ERR_WORKSPACE;
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess) return STCA_ERR_HIP;
  if (dev < 0 || dev >= kMaxDevices) return STCA_ERR_UNSUPPORTED;
  void* ws = scratch_ptr(dev);
  if (!ws) return STCA_ERR_HIP;
  return stca_forward(dims, batch, hist, tgt, w, out, saved, ws, kScratchBytes, stream);
}
