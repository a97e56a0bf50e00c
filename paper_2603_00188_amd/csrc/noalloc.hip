// stlite_select_topk_noalloc: the integrated score and flat top-B of
// stlite_select_topk with its workspace in a library-owned static device
// array instead of a caller-allocated buffer, for callers that cannot
// allocate device memory.
//
// `scratch` is a file-scope __device__ array: every GPU the library runs on
// holds its own copy, at its own address, from module load until the process
// ends.  In host code the name `scratch` is only a host-side stand-in, so the
// address handed to kernels is the one hipGetSymbolAddress returns for the
// current device, looked up once per device on the first call there and kept
// in `g_scratch`.  The selection's workspace needs no clearing between calls
// (every pass writes the words the next one reads), so the array is never
// zeroed; it keeps what the last call left in it.
#include <stdio.h>

#include <atomic>
#include <mutex>

#include "stlite.h"
#include "stlite_internal.h"

namespace stlite {
stlite_status report_error(stlite_status st, const char* msg);  // stlite_abi.hip
}

namespace {

constexpr size_t kScratchBytes = size_t(STLITE_NOALLOC_SCRATCH_BYTES);
constexpr int kMaxDevices = 64;

static __device__ __align__(256) unsigned char scratch[kScratchBytes];

std::atomic<void*> g_scratch[kMaxDevices];
std::mutex g_scratch_mutex;

// Device address of `scratch` on the current device (nullptr on failure,
// with *err set).  Looked up once per device.
void* scratch_address(hipError_t* err) {
  int dev = -1;
  *err = hipGetDevice(&dev);
  if (*err != hipSuccess) return nullptr;
  if (dev < 0 || dev >= kMaxDevices) {
    *err = hipErrorInvalidDevice;
    return nullptr;
  }
  void* ptr = g_scratch[dev].load(std::memory_order_acquire);
  if (ptr) return ptr;
  std::lock_guard<std::mutex> lock(g_scratch_mutex);
  ptr = g_scratch[dev].load(std::memory_order_relaxed);
  if (!ptr) {
    *err = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (*err != hipSuccess || !ptr) return nullptr;
    g_scratch[dev].store(ptr, std::memory_order_release);
  }
  return ptr;
}

}  // namespace

extern "C" stlite_status stlite_select_topk_noalloc(const stlite_problem* p, const float* a_base,
                                                     const float* phi, const uint8_t* gate, float alpha,
                                                     int32_t* kept, float* score, void* stream) {
  size_t need = 0;
  stlite_status st = stlite_workspace_size(p, STLITE_CALL_SELECT_TOPK, &need);
  if (st != STLITE_OK) return st;
  char msg[256];
  if (need > kScratchBytes) {
    snprintf(msg, sizeof(msg), "the selection needs %zu bytes of scratch; the static buffer holds %zu",
             need, kScratchBytes);
    return stlite::report_error(STLITE_ERR_WORKSPACE, msg);
  }
  hipError_t err = hipSuccess;
  void* ws = scratch_address(&err);
  if (!ws) {
    snprintf(msg, sizeof(msg), "static scratch address: %s", hipGetErrorString(err));
    return stlite::report_error(STLITE_ERR_HIP, msg);
  }
  return stlite_select_topk(p, a_base, phi, gate, alpha, kept, score, ws, kScratchBytes, stream);
}
