// The one-call step (mpa_append_attention) for callers that cannot allocate
// device memory: code under HIP graph capture, tight serving loops, harnesses
// that forbid hipMalloc.  The split-K partial results, which the ordinary
// entry point keeps in a caller workspace, live here in one fixed device
// array of the library, `scratch`.
//
// In host code `scratch` names a host-side stand-in for the array, not its
// device address: the address comes from hipGetSymbolAddress, looked up once
// per device (with that device current, on the entry point's first call
// there) and kept per device, and only that pointer is ever handed to a
// kernel.  Every call on a device shares that device's array; nothing in it
// has to start at zero (every partial result is written by the step's
// attention kernels before its merge reads it), and calls that overlap on
// one device race on it.
#include <hip/hip_runtime.h>

#include <atomic>
#include <mutex>

#include "mpa.h"

namespace {

constexpr size_t kScratchBytes = MPA_SCRATCH_BYTES;
constexpr int kMaxDevices = 64;

static __device__ __align__(256) unsigned char scratch[kScratchBytes];

std::atomic<void*> g_scratch_ptr[kMaxDevices];
std::mutex g_scratch_lock;

// The current device's address of `scratch` (MPA_ERR_HIP when the lookup fails).
int scratch_on_current_device(void** ptr) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return MPA_ERR_HIP;
  void* p = g_scratch_ptr[dev].load(std::memory_order_acquire);
  if (!p) {
    std::lock_guard<std::mutex> guard(g_scratch_lock);
    p = g_scratch_ptr[dev].load(std::memory_order_relaxed);
    if (!p) {
      if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return MPA_ERR_HIP;
      g_scratch_ptr[dev].store(p, std::memory_order_release);
    }
  }
  *ptr = p;
  return MPA_OK;
}

}  // namespace

extern "C" int mpa_append_attention_noalloc(const mpa_shape* shape, const void* q, const void* k_new,
                                            const void* v_new, void* k_cache, void* v_cache,
                                            const int32_t* block_tables, const int32_t* seq_lens,
                                            const int32_t* query_start_loc, const int32_t* seq_lens_host,
                                            const int32_t* query_start_loc_host, const int32_t* block_tables_host,
                                            void* out, float* lse, void* stream) {
  if (!shape) return MPA_ERR_INVALID;
  // A batch whose partial results do not fit is refused before anything
  // runs; an invalid batch (size 0) gets its own error from the step's checks.
  if (mpa_workspace_size(shape, seq_lens_host, query_start_loc_host) > kScratchBytes) return MPA_ERR_SCRATCH;
  void* ws = nullptr;
  const int rc = scratch_on_current_device(&ws);
  if (rc != MPA_OK) return rc;
  return mpa_append_attention(shape, q, k_new, v_new, k_cache, v_cache, block_tables, seq_lens, query_start_loc,
                              seq_lens_host, query_start_loc_host, block_tables_host, out, lse, ws, kScratchBytes,
                              stream);
}
