// Internal declarations of libmori shared by the kernel files and the C ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/mori.h"

namespace mori {

// Page-state bits of the page-allocation pass.
constexpr uint32_t PS_FREE = 1u;   // marked free in the caller's free map before the step
constexpr uint32_t PS_OWNED = 2u;  // owned by a GPU-resident program
constexpr uint32_t PS_REL = 4u;    // owned by a program leaving the GPU this step
constexpr uint32_t PS_LATER = 8u;  // ... and free only after the swap-out stream has passed: the
                                   // swap-out reads it, or its dropped program may still be running

constexpr int PAGE_TILE = 512;     // pages per workgroup in the page-allocation kernels (2 per thread;
                                   // measured: 0.5-1 us faster per plan than 1024, 2048 slower)
constexpr int PAGE_WG = 256;       // threads per page-allocation workgroup (16 pages each)

// Plan summary as kept on the device (the head of the plan blob, mirrored on the host).
struct DevSummary {
  uint32_t num_programs, m_gpu, m_cpu, m_ssd;
  uint32_t n_out, n_in, n_drop_gpu, n_drop_cpu, n_admit_gpu, n_admit_cpu;
  uint32_t error;
  uint64_t pages_out, pages_in, pages_admit;
  uint64_t pages_free_before, pages_released, pages_recycled, pages_free_after;
  uint64_t bytes_out, bytes_in, gpu_bytes_after, cpu_bytes_after, ssd_bytes_after;
  uint64_t need;  // pages_in + pages_admit
  uint64_t pages_dropped;  // released pages nothing reads any more: slots below free-before + this need no wait
};

// A registered memory range usable by the swap kernels.
struct DevRange {
  uint64_t host_base;  // address as the caller names it
  uint64_t bytes;
  uint64_t dev_base;   // the same memory as the GPU addresses it
  uint64_t is_device;  // 1: HBM, 0: pinned host memory
};

// Everything the plan kernels read and write.
struct PlanArgs {
  // caller-owned
  const float* window;
  const float* idleness;
  const uint8_t* status;
  const uint32_t* tbl_off;
  uint32_t* tbl;
  uint8_t* tier;
  uint8_t* free_map;
  uint32_t tbl_len, P, k, flags, NB, ntiles;
  uint64_t block_bytes, gpu_bytes, cpu_bytes, ssd_bytes;
  // context scratch: plan blob (mirrored to the host)
  DevSummary* sum;
  uint32_t* order;
  uint64_t* prefix;
  uint8_t* tier_old;
  uint8_t* tier_new;
  uint8_t* cat;
  uint32_t* out_prog;
  uint32_t* in_prog;
  uint32_t* out_pg_base;  // [n_out + 1] first out-page index of each out program
  uint32_t* in_pg_base;   // [n_in + 1] first slot of each in program
  // context scratch: device only
  uint32_t* base;         // per program: out-page base (OUT) or slot base (IN, ADMIT_GPU)
  uint32_t* pstate;       // [NB]
  uint32_t* out_src;      // [pages_out] old page of each out page index
  uint32_t* in_dst;       // [need] page of each slot
  uint64_t* tile_cnt;     // [2 ntiles]: packed (free-before, dropped << 32), then free-later counts
  uint64_t* tile_base;    // [2 ntiles] exclusive prefixes of both halves of tile_cnt
  uint32_t* swap_err;     // [2] swap-out, swap-in address errors; cleared by every plan
  // The pinned host mirror of the plan blob, as the device addresses it: the
  // kernels that finish a part of the plan store it there too, so no copy of
  // the blob follows the plan.  Mirror address = blob address + host_delta.
  int64_t host_delta;
};

template <typename T>
__device__ inline T* host_mirror(const PlanArgs& a, T* blob_ptr) {
  return reinterpret_cast<T*>(reinterpret_cast<char*>(blob_ptr) + a.host_delta);
}

// Everything a swap kernel reads.
struct SwapArgs {
  uint8_t* pool;
  uint64_t NB, run;
  uint32_t LC;              // layers * planes
  const DevSummary* sum;
  const uint32_t* prog;     // out_prog or in_prog
  const uint32_t* pg_base;  // out_pg_base or in_pg_base
  const uint32_t* pages;    // out_src (by out-page index) or in_dst (by slot)
  const uint64_t* addr;     // device address of each program's host buffer
  const uint32_t* swap_err; // [2] address errors found by the swap-out's and the swap-in's translation
  uint8_t* staging;         // non-null: chunk staging buffer (copy-engine mode)
  uint64_t u_begin, u_end;  // staging mode: unit range of the chunk
  uint32_t part;            // swap-in: 0 all slots, 1 slots < free-before, 2 slots >= free-before
  uint32_t host_link;       // 1: the other side is pinned host memory (kernel-direct mode over the host link)
};

struct TranslateArgs {
  const DevSummary* sum;
  const uint32_t* prog;     // out_prog or in_prog (count n_out / n_in)
  int dir_in;               // 0 out, 1 in
  const uint32_t* tbl_off;
  uint64_t block_bytes;
  const uint64_t* addr_in;  // [P] caller addresses (copied to the device)
  uint64_t* addr_out;       // [P] translated device addresses
  const DevRange* ranges;
  uint32_t nranges;
  uint32_t* swap_err;       // [2]: this direction's word is swap_err[dir_in]
};

// Typed eviction order: workgroup size, keys per thread (measured on MI355X:
// 4 is fastest up to ~2^19 blocks, more workgroups for a latency-bound sort;
// 8 above, fewer tiles to scan per digit), keys-kernel workgroups at most.
constexpr int EVICT_WG = 256;
constexpr uint32_t EVICT_SMALL_SORT = 1u << 19;
constexpr uint32_t EVICT_KEY_WG_MAX = 128;
constexpr int evict_keys_per_thread(uint32_t N) { return N <= EVICT_SMALL_SORT ? 4 : 8; }

// Device workspace of the eviction order for N blocks, in the order
// launch_evict lays it out (each piece 256-B aligned): two key and two value
// buffers, the tile histogram, digit totals, two look-back status arrays,
// per-workgroup digit counts, their totals, tile counters, tile sums, a
// prefix buffer and a few words of results.
constexpr uint64_t evict_workspace_bytes(uint32_t N) {
  const uint64_t tile = (uint64_t)EVICT_WG * evict_keys_per_thread(N);
  const uint64_t ntiles = ((uint64_t)N + tile - 1) / tile;
  auto up = [](uint64_t b) { return (b + 255) & ~255ull; };
  return 2 * up(8ull * N) + 2 * up(4ull * N) + up(4ull * 256 * ntiles) + up(4 * 256) + 2 * up(8ull * 256 * ntiles) +
         up(4ull * EVICT_KEY_WG_MAX * 8 * 256) + up(4 * 8 * 256) + up(4 * 8) + up(8ull * ntiles) + up(8ull * N) +
         up(8 * 4);
}

// launchers (return the launch error)
hipError_t launch_rank(const PlanArgs& a, hipStream_t s);
hipError_t launch_pages(const PlanArgs& a, hipStream_t s);
hipError_t launch_translate(const TranslateArgs& a, hipStream_t s);
hipError_t launch_swap_out(const SwapArgs& a, uint32_t grid, hipStream_t s);
hipError_t launch_swap_in(const SwapArgs& a, uint32_t grid, hipStream_t s);
hipError_t launch_evict(uint32_t N, const uint8_t* type, const uint64_t* last_access, const uint32_t* size,
                        uint64_t unit_bytes, uint32_t tier, uint64_t need, void* workspace, uint32_t* order,
                        uint64_t* prefix, uint32_t* result, hipStream_t s);

}  // namespace mori
