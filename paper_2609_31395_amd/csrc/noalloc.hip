// actkv_step_noalloc: the whole step with no allocation by anyone, for callers that cannot
// call hipMalloc (code under HIP graph capture, tight serving loops, harnesses that forbid
// it).  Its workspace is a static device array of fixed size in this library's code object:
// every GPU the library runs on holds its own copy until the process ends.  The array's
// device address is looked up once per device, with that device current, on the entry
// point's first call there; host code uses only that address, never the array's name.
#include <atomic>
#include <mutex>

#include "actkv.h"
#include "actkv_internal.h"

namespace {

constexpr int kMaxDevices = 64;

__device__ __align__(256) char scratch[ACTKV_NOALLOC_SCRATCH_BYTES];

std::atomic<void*> g_scratch[kMaxDevices];   // the array's address on each device
std::mutex g_scratch_mu;

// The scratch array's device address on the current device (looked up on first use).
actkv_status current_scratch(void** out) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return ACTKV_ERR_HIP;
  if (dev < 0 || dev >= kMaxDevices) return ACTKV_ERR_UNSUPPORTED;
  void* ptr = g_scratch[dev].load(std::memory_order_acquire);
  if (!ptr) {
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    ptr = g_scratch[dev].load(std::memory_order_relaxed);
    if (!ptr) {
      if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || !ptr)
        return ACTKV_ERR_HIP;
      g_scratch[dev].store(ptr, std::memory_order_release);
    }
  }
  *out = ptr;
  return ACTKV_OK;
}

}  // namespace

extern "C" actkv_status actkv_step_noalloc(const actkv_problem* p, const void* q,
                                           void* kv_cache, int32_t* block_table,
                                           const float* lse, const int32_t* free_pages,
                                           int64_t num_free, float* scores, float* pooled,
                                           int32_t* kept, int32_t* freed_pages,
                                           int32_t* new_lens, void* stream) {
  // the size check first: a problem past the array's size is refused before any HIP call
  size_t need = 0;
  actkv_status st = actkv_query(p, &need, nullptr, nullptr, nullptr);
  if (st != ACTKV_OK) return st;
  if (need > (size_t)ACTKV_NOALLOC_SCRATCH_BYTES) return ACTKV_ERR_WORKSPACE_TOO_SMALL;
  void* ptr = nullptr;
  st = current_scratch(&ptr);
  if (st != ACTKV_OK) return st;
  return actkv::step_impl(p, q, kv_cache, block_table, lse, free_pages, num_free, scores,
                          pooled, kept, freed_pages, new_lens, ptr,
                          (size_t)ACTKV_NOALLOC_SCRATCH_BYTES, stream, false);
}
