// Allocation-free entry point of the typed eviction order: the same kernels
// as mori_evict_order, with the workspace in a device array of the library
// instead of a caller buffer.  For callers that cannot allocate device memory
// (code under HIP graph capture, serving loops that forbid it).
//
// The array lives for the process on every GPU the library's code is loaded
// on; each GPU holds its own copy at its own address, which is looked up once
// per device (with that device current) and kept.  Host code never passes
// the array's name to a kernel or a copy: only that looked-up address.
#include <mutex>

#include "mori_internal.h"

namespace mori {
namespace {

constexpr uint64_t kScratchBytes = evict_workspace_bytes(MORI_EVICT_NOALLOC_MAX_BLOCKS);
static_assert(kScratchBytes % 256 == 0, "workspace pieces are 256-B aligned");

// The workspace is largest at the maximum: the 4-keys-per-thread tiles are used up
// to 2^19 blocks, and every piece grows with N at a fixed tile size.
static_assert(MORI_EVICT_NOALLOC_MAX_BLOCKS <= EVICT_SMALL_SORT, "one tile size up to the maximum");

static __device__ __align__(256) uint8_t scratch[kScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_mutex;
void* g_scratch[kMaxDevices] = {};

// This device's copy of `scratch` (the current device), looked up on the
// first call on it.
hipError_t device_scratch(int dev, void** out) {
  std::lock_guard<std::mutex> lock(g_mutex);
  if (!g_scratch[dev]) {
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (!p || (reinterpret_cast<uintptr_t>(p) & 255u)) return hipErrorInvalidSymbol;
    g_scratch[dev] = p;
  }
  *out = g_scratch[dev];
  return hipSuccess;
}

}  // namespace
}  // namespace mori

extern "C" int mori_evict_order_noalloc(const mori_blocks* b, uint32_t tier, uint64_t need_bytes, uint32_t* order,
                                        uint64_t* prefix, uint32_t* result, void* stream) {
  using namespace mori;
  if (!b || !result) return MORI_EINVAL;
  if (tier != MORI_TIER_GPU && tier != MORI_TIER_CPU) return MORI_EINVAL;
  if (b->num_blocks && (!b->type || !b->last_access || !order)) return MORI_EINVAL;
  if (b->num_blocks > MORI_EVICT_NOALLOC_MAX_BLOCKS) return MORI_ENOSPC;
  if (evict_workspace_bytes(b->num_blocks) > kScratchBytes) return MORI_ENOSPC;  // not reached: see above
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) {
    (void)hipGetLastError();
    return MORI_EHIP;
  }
  if (dev < 0 || dev >= kMaxDevices) return MORI_EINVAL;
  void* ws = nullptr;
  if (device_scratch(dev, &ws) != hipSuccess) {
    (void)hipGetLastError();
    return MORI_EHIP;
  }
  const hipError_t e = launch_evict(b->num_blocks, b->type, b->last_access, b->size, b->unit_bytes, tier, need_bytes,
                                    ws, order, prefix, result, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) {
    (void)hipGetLastError();
    return MORI_EHIP;
  }
  return MORI_OK;
}
