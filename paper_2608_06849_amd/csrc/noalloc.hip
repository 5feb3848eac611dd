// Fused decode step for callers that cannot allocate device memory: the
// split-K partial results live in a static device array of this library
// instead of a caller workspace.  Same validation, split plan and kernels as
// aoh_decode_step, so the results are bit-identical to it.
//
// The array is a file-scope static device variable.  Its host-side name is
// only a symbol handle: the device address of each GPU's copy comes from
// hipGetSymbolAddress, looked up once per device on the first call that runs
// with that device current, and only that address is handed to kernels.
#include <cstdio>
#include <mutex>

#include "aoh.h"
#include "aoh_internal.h"

// Largest workspace a call may need (a batch-8 x 131072-token, 32-query-head,
// d_head-128 step needs about 32 MiB).
constexpr size_t kScratchBytes = size_t(64) << 20;

static __device__ __align__(256) unsigned char scratch[kScratchBytes];

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_mu;
void* g_scratch[kMaxDevices] = {};

// Device address of the current device's array (nullptr on failure, with
// the reason in msg).
void* scratch_address(char* msg, size_t len) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) {
    snprintf(msg, len, "hipGetDevice: %s", hipGetErrorString(e));
    return nullptr;
  }
  if (dev < 0 || dev >= kMaxDevices) {
    snprintf(msg, len, "device %d outside [0, %d)", dev, kMaxDevices);
    return nullptr;
  }
  std::lock_guard<std::mutex> lock(g_mu);
  if (!g_scratch[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p) {
      snprintf(msg, len, "hipGetSymbolAddress(scratch) on device %d: %s", dev, hipGetErrorString(e));
      return nullptr;
    }
    g_scratch[dev] = p;
  }
  return g_scratch[dev];
}

}  // namespace

extern "C" aoh_status aoh_decode_step_noalloc(const aoh_tensor* q, const aoh_tensor* k_new, const aoh_tensor* v_new,
                                              const aoh_paged_cache* kv_full, const aoh_ring_cache* kv_ring,
                                              const uint8_t* head_is_streaming, const int32_t* lens, int32_t n_sink,
                                              int32_t window, aoh_tensor* out, void* stream) {
  size_t need = 0;
  aoh_status st = aoh::decode_step_workspace_need(q, k_new, v_new, kv_full, kv_ring, head_is_streaming, lens, n_sink,
                                                  window, out, &need);
  if (st != AOH_OK) return st;
  char msg[256];
  if (need > kScratchBytes) {
    snprintf(msg, sizeof(msg), "the step needs %zu bytes of workspace; the static scratch area holds %zu", need,
             kScratchBytes);
    return aoh::report(AOH_ERR_UNSUPPORTED, msg);
  }
  void* ws = scratch_address(msg, sizeof(msg));
  if (!ws) return aoh::report(AOH_ERR_HIP, msg);
  return aoh_decode_step(q, k_new, v_new, kv_full, kv_ring, head_is_streaming, lens, n_sink, window, out, ws,
                         kScratchBytes, stream);
}
