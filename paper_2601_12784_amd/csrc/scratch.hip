// The decode step for callers that cannot allocate device memory: the
// split-K partial results live in a device array of the library's own,
// `scratch`, instead of a workspace the caller passes in.
//
// Host code never passes the array's name to a kernel or a copy: in host
// code that name stands for a host-side placeholder, not the device
// address. The address is looked up once per device with
// hipGetSymbolAddress (each device holds its own copy of the array) and kept.
#include <hip/hip_runtime.h>

#include <atomic>
#include <mutex>

#include "sf_internal.h"

namespace {

constexpr uint64_t kScratchBytes = SF_SCRATCH_BYTES;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

constexpr int kMaxDevices = 64;
std::atomic<void*> g_scratch_ptr[kMaxDevices];
std::mutex g_scratch_mu;

// The array's address on the current device (looked up on first use there).
sf_status scratch_on_current_device(void** ptr) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0) return SF_ERR_HIP;
  if (dev >= kMaxDevices) return SF_ERR_UNSUPPORTED;
  void* p = g_scratch_ptr[dev].load(std::memory_order_acquire);
  if (!p) {
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    p = g_scratch_ptr[dev].load(std::memory_order_relaxed);
    if (!p) {
      if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return SF_ERR_HIP;
      g_scratch_ptr[dev].store(p, std::memory_order_release);
    }
  }
  *ptr = p;
  return SF_OK;
}

}  // namespace

extern "C" sf_status sf_decode_attn_scratch(const sf_attn_desc* desc, const sf_plan_info* info,
                                            const int32_t* work_dev, const void* q, const void* k_pool,
                                            const void* v_pool, const int32_t* block_table, float* out,
                                            float* lse, void* stream) {
  // Everything is checked before the first HIP call.
  const sf_status chk = sf::check_step_args(desc, info, work_dev, q, k_pool, v_pool, block_table, out, lse,
                                            nullptr, nullptr, nullptr, nullptr, nullptr);
  if (chk != SF_OK) return chk;
  if (info->workspace_bytes > kScratchBytes) return SF_ERR_CAPACITY;
  void* ws = nullptr;
  if (info->workspace_bytes > 0 && info->num_workers > 0) {
    const sf_status st = scratch_on_current_device(&ws);
    if (st != SF_OK) return st;
  }
  return sf::decode_attn_and_combine(desc, info, work_dev, q, k_pool, v_pool, block_table, out, lse, ws,
                                     kScratchBytes, stream);
}
