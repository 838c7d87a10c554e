// Typed eviction order of one memory tier (Sec. 4.3.2, typed offloading).
//
// Each KV block carries its program's type label (busy = GPU queue, idle =
// CPU queue, inactive = Waiting) and its last access time.  A tier evicts by
// type first, in tier-reversed order (GPU: inactive, idle, busy; CPU:
// inactive, busy, idle), least recently used first within a type, equal
// (type, time) lowest block id first.  That is one ascending sort of the
// 64-bit key (type position << 62 | last access) with the block id riding
// along, done here as a device-wide stable LSD radix sort:
//
//   keys     build keys, validate, OR/AND of all keys (digits on which every
//            key agrees need no pass);
//   per pass (8-bit digit, 8 passes)
//     hist   per 4096-key tile: 256-bin histogram  -> hist[digit][tile]
//     scan   one workgroup: exclusive scan of hist in (digit, tile) order
//     scatter per tile: stable rank of every key among the tile's keys of its
//            digit (wave64 ballots over the 8 digit bits, slices of 256 keys
//            in original order) + the scanned base -> position
//            (a pass over a constant digit copies instead);
//   prefix   inclusive u64 scan of block bytes in eviction order (tile scans,
//            one-workgroup scan of tile totals, fix-up) and the number of
//            evictions that frees the requested bytes.
//
// Everything is latency-bound at 10^5-10^6 blocks (tens of microseconds);
// the workspace is the caller's, so nothing is allocated here.
#include "mori_internal.h"

namespace mori {
namespace {

constexpr int ET = 256;                 // threads per tile workgroup
constexpr int EIPT = 16;                // keys per thread
constexpr int ETILE = ET * EIPT;        // 4096 keys per tile
constexpr int ENW = ET / 64;            // waves per tile workgroup
constexpr uint64_t TIME_LIMIT = 1ull << 62;

struct EvictArgs {
  uint32_t N, ntiles, tier;
  const uint8_t* type;
  const uint64_t* last_access;
  const uint32_t* size;
  uint64_t unit_bytes, need;
  uint64_t* keys[2];
  uint32_t* vals[2];
  uint32_t* hist;       // [256][ntiles]
  uint64_t* tile_sum;   // [ntiles]
  uint64_t* misc;       // [0] OR of keys, [1] AND of keys, [2] error bits, [3] evictions short of need
  uint32_t* order;      // out [N]
  uint64_t* prefix;     // out [N] (or workspace)
  uint32_t* result;     // out [2]: count, error bits
};

__global__ void evict_init_kernel(EvictArgs a) {
  a.misc[0] = 0;
  a.misc[1] = ~0ull;
  a.misc[2] = 0;
  a.misc[3] = 0;
}

__global__ __launch_bounds__(ET) void evict_keys_kernel(EvictArgs a) {
  // position of each type label in the tier's eviction order (busy, idle, inactive)
  const uint32_t gpu_pos[3] = {2, 1, 0}, cpu_pos[3] = {1, 2, 0};
  const uint32_t* pos = a.tier == MORI_TIER_GPU ? gpu_pos : cpu_pos;
  uint64_t o = 0, n = ~0ull, err = 0;
  for (uint32_t i = blockIdx.x * ET + threadIdx.x; i < a.N; i += gridDim.x * ET) {
    const uint8_t t = a.type[i];
    const uint64_t la = a.last_access[i];
    if (t > MORI_TYPE_INACTIVE || la >= TIME_LIMIT) {
      err |= MORI_DEV_BAD_BLOCK;
      continue;
    }
    const uint64_t key = ((uint64_t)pos[t] << 62) | la;
    a.keys[0][i] = key;
    a.vals[0][i] = i;
    o |= key;
    n &= key;
  }
  // wave-level reduction before the global atomics
  for (int off = 32; off > 0; off >>= 1) {
    o |= __shfl_xor(o, off, 64);
    n &= __shfl_xor(n, off, 64);
    err |= __shfl_xor(err, off, 64);
  }
  if ((threadIdx.x & 63) == 0) {
    atomicOr((unsigned long long*)&a.misc[0], (unsigned long long)o);
    atomicAnd((unsigned long long*)&a.misc[1], (unsigned long long)n);
    if (err) atomicOr((unsigned long long*)&a.misc[2], (unsigned long long)err);
  }
}

__device__ inline bool digit_varies(const EvictArgs& a, int shift) {
  return (((a.misc[0] ^ a.misc[1]) >> shift) & 255u) != 0;
}

__global__ __launch_bounds__(ET) void evict_hist_kernel(EvictArgs a, int src, int shift) {
  __shared__ uint32_t s_h[256];
  if (a.misc[2] || !digit_varies(a, shift)) return;
  s_h[threadIdx.x] = 0;
  __syncthreads();
  const uint64_t* k = a.keys[src];
  const uint64_t base = (uint64_t)blockIdx.x * ETILE;
#pragma unroll 4
  for (int it = 0; it < EIPT; ++it) {
    const uint64_t i = base + it * ET + threadIdx.x;
    if (i < a.N) atomicAdd(&s_h[(k[i] >> shift) & 255u], 1u);
  }
  __syncthreads();
  a.hist[(uint64_t)threadIdx.x * a.ntiles + blockIdx.x] = s_h[threadIdx.x];
}

// Exclusive scan of u32 counts in place (1024 threads); total fits in u32 (N < 2^32).
__global__ __launch_bounds__(1024) void evict_scan_kernel(EvictArgs a, int shift) {
  __shared__ uint32_t s_w[1024 / 64 + 1];
  if (a.misc[2] || !digit_varies(a, shift)) return;
  const uint64_t E = 256ull * a.ntiles;
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
  uint32_t carry = 0;
  for (uint64_t e0 = 0; e0 < E; e0 += 1024) {
    const uint64_t e = e0 + threadIdx.x;
    const uint32_t v = e < E ? a.hist[e] : 0u;
    uint32_t x = v;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
      const uint32_t y = __shfl_up(x, off, 64);
      if (lane >= off) x += y;
    }
    if (lane == 63) s_w[wid] = x;
    __syncthreads();
    if (wid == 0) {
      const uint32_t w = lane < 16 ? s_w[lane] : 0u;
      uint32_t wi = w;
#pragma unroll
      for (int off = 1; off < 16; off <<= 1) {
        const uint32_t y = __shfl_up(wi, off, 64);
        if (lane >= off) wi += y;
      }
      if (lane < 16) s_w[lane] = wi - w;
      if (lane == 15) s_w[16] = wi;
    }
    __syncthreads();
    if (e < E) a.hist[e] = carry + s_w[wid] + x - v;
    carry += s_w[16];
    __syncthreads();
  }
}

__global__ __launch_bounds__(ET) void evict_scatter_kernel(EvictArgs a, int src, int shift) {
  __shared__ uint32_t s_off[256];     // this tile's global base per digit
  __shared__ uint32_t s_run[256];     // keys of each digit already placed by earlier slices
  __shared__ uint32_t s_wc[ENW][256]; // per-slice, per-wave counts -> bases
  if (a.misc[2]) return;
  const uint64_t* ks = a.keys[src];
  const uint32_t* vs = a.vals[src];
  uint64_t* kd = a.keys[src ^ 1];
  uint32_t* vd = a.vals[src ^ 1];
  const uint64_t base = (uint64_t)blockIdx.x * ETILE;
  if (!digit_varies(a, shift)) {  // every key has the same digit: the pass keeps the order
    for (int it = 0; it < EIPT; ++it) {
      const uint64_t i = base + it * ET + threadIdx.x;
      if (i < a.N) {
        kd[i] = ks[i];
        vd[i] = vs[i];
      }
    }
    return;
  }
  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  s_off[tid] = a.hist[(uint64_t)tid * a.ntiles + blockIdx.x];
  s_run[tid] = 0;
#pragma unroll
  for (int w = 0; w < ENW; ++w) s_wc[w][tid] = 0;
  __syncthreads();
  const uint64_t lanemask_lt = (1ull << lane) - 1ull;
  for (int it = 0; it < EIPT; ++it) {
    const uint64_t i = base + it * ET + tid;
    const bool valid = i < a.N;
    const uint64_t key = valid ? ks[i] : 0ull;
    const uint32_t val = valid ? vs[i] : 0u;
    const uint32_t d = (uint32_t)(key >> shift) & 255u;
    uint64_t same = __ballot(valid);
#pragma unroll
    for (int b = 0; b < 8; ++b) {
      const uint64_t bal = __ballot((d >> b) & 1u);
      same &= ((d >> b) & 1u) ? bal : ~bal;
    }
    const uint32_t r = __popcll(same & lanemask_lt);
    if (valid && r == 0) s_wc[wid][d] = __popcll(same);
    __syncthreads();
    {  // bases of this slice: earlier slices, then earlier waves of this slice
      uint32_t run = s_run[tid];
#pragma unroll
      for (int w = 0; w < ENW; ++w) {
        const uint32_t c = s_wc[w][tid];
        s_wc[w][tid] = run;
        run += c;
      }
      s_run[tid] = run;
    }
    __syncthreads();
    if (valid) {
      const uint32_t pos = s_off[d] + s_wc[wid][d] + r;
      kd[pos] = key;
      vd[pos] = val;
    }
    __syncthreads();
#pragma unroll
    for (int w = 0; w < ENW; ++w) s_wc[w][tid] = 0;
    __syncthreads();
  }
}

// Inclusive scan of freed bytes within each tile; tile totals to tile_sum.
__global__ __launch_bounds__(ET) void evict_prefix_tiles_kernel(EvictArgs a, int src) {
  __shared__ uint64_t s_w[ENW + 1];
  if (a.misc[2]) return;
  const uint32_t* order = a.vals[src];
  const uint64_t base = (uint64_t)blockIdx.x * ETILE + (uint64_t)threadIdx.x * EIPT;  // blocked: 16 consecutive
  uint64_t v[EIPT];
  uint64_t s = 0;
#pragma unroll
  for (int j = 0; j < EIPT; ++j) {
    const uint64_t i = base + j;
    uint64_t bytes = 0;
    if (i < a.N) {
      const uint32_t b = order[i];
      a.order[i] = b;
      bytes = (uint64_t)(a.size ? a.size[b] : 1u) * a.unit_bytes;
    }
    s += bytes;
    v[j] = s;
  }
  // exclusive scan of the per-thread totals
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
  uint64_t x = s;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const uint64_t y = __shfl_up(x, off, 64);
    if (lane >= off) x += y;
  }
  if (lane == 63) s_w[wid] = x;
  __syncthreads();
  if (threadIdx.x == 0) {
    uint64_t run = 0;
    for (int w = 0; w < ENW; ++w) {
      const uint64_t c = s_w[w];
      s_w[w] = run;
      run += c;
    }
    s_w[ENW] = run;
  }
  __syncthreads();
  const uint64_t before = s_w[wid] + x - s;
#pragma unroll
  for (int j = 0; j < EIPT; ++j)
    if (base + j < a.N) a.prefix[base + j] = before + v[j];
  if (threadIdx.x == 0) a.tile_sum[blockIdx.x] = s_w[ENW];
}

__global__ __launch_bounds__(1024) void evict_prefix_top_kernel(EvictArgs a) {
  __shared__ uint64_t s_w[1024 / 64 + 1];
  if (a.misc[2]) return;
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
  uint64_t carry = 0;
  for (uint32_t t0 = 0; t0 < a.ntiles; t0 += 1024) {
    const uint32_t t = t0 + threadIdx.x;
    const uint64_t v = t < a.ntiles ? a.tile_sum[t] : 0ull;
    uint64_t x = v;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
      const uint64_t y = __shfl_up(x, off, 64);
      if (lane >= off) x += y;
    }
    if (lane == 63) s_w[wid] = x;
    __syncthreads();
    if (wid == 0) {
      const uint64_t w = lane < 16 ? s_w[lane] : 0ull;
      uint64_t wi = w;
#pragma unroll
      for (int off = 1; off < 16; off <<= 1) {
        const uint64_t y = __shfl_up(wi, off, 64);
        if (lane >= off) wi += y;
      }
      if (lane < 16) s_w[lane] = wi - w;
      if (lane == 15) s_w[16] = wi;
    }
    __syncthreads();
    if (t < a.ntiles) a.tile_sum[t] = carry + s_w[wid] + x - v;  // exclusive base of tile t
    carry += s_w[16];
    __syncthreads();
  }
}

__global__ __launch_bounds__(ET) void evict_prefix_fix_kernel(EvictArgs a) {
  if (a.misc[2]) return;
  const uint64_t add = a.tile_sum[blockIdx.x];
  const uint64_t base = (uint64_t)blockIdx.x * ETILE;
  uint32_t short_of_need = 0;
  for (int it = 0; it < EIPT; ++it) {
    const uint64_t i = base + it * ET + threadIdx.x;
    if (i < a.N) {
      const uint64_t p = a.prefix[i] + add;
      a.prefix[i] = p;
      short_of_need += p < a.need;
    }
  }
  for (int off = 32; off > 0; off >>= 1) short_of_need += __shfl_xor(short_of_need, off, 64);
  if ((threadIdx.x & 63) == 0 && short_of_need)
    atomicAdd((unsigned long long*)&a.misc[3], (unsigned long long)short_of_need);
}

__global__ void evict_result_kernel(EvictArgs a) {
  const uint64_t err = a.misc[2];
  uint64_t count = 0;
  if (!err && a.need > 0) {
    count = a.misc[3] + 1;  // freed bytes are non-decreasing along the order
    if (count > a.N) count = a.N;
  }
  a.result[0] = (uint32_t)count;
  a.result[1] = (uint32_t)err;
}

}  // namespace

uint64_t evict_workspace_bytes(uint32_t N) {
  const uint64_t ntiles = ((uint64_t)N + ETILE - 1) / ETILE;
  auto up = [](uint64_t b) { return (b + 255) & ~255ull; };
  return 2 * up(8ull * N) + 2 * up(4ull * N) + up(4ull * 256 * ntiles) + up(8ull * ntiles) + up(8ull * N) +
         up(8 * 4);
}

hipError_t launch_evict(uint32_t N, const uint8_t* type, const uint64_t* last_access, const uint32_t* size,
                        uint64_t unit_bytes, uint32_t tier, uint64_t need, void* workspace, uint32_t* order,
                        uint64_t* prefix, uint32_t* result, hipStream_t s) {
  EvictArgs a{};
  a.N = N;
  a.ntiles = (uint32_t)(((uint64_t)N + ETILE - 1) / ETILE);
  a.tier = tier;
  a.type = type;
  a.last_access = last_access;
  a.size = size;
  a.unit_bytes = unit_bytes;
  a.need = need;
  auto up = [](uint64_t b) { return (b + 255) & ~255ull; };
  uint8_t* w = static_cast<uint8_t*>(workspace);
  a.keys[0] = reinterpret_cast<uint64_t*>(w);
  w += up(8ull * N);
  a.keys[1] = reinterpret_cast<uint64_t*>(w);
  w += up(8ull * N);
  a.vals[0] = reinterpret_cast<uint32_t*>(w);
  w += up(4ull * N);
  a.vals[1] = reinterpret_cast<uint32_t*>(w);
  w += up(4ull * N);
  a.hist = reinterpret_cast<uint32_t*>(w);
  w += up(4ull * 256 * a.ntiles);
  a.tile_sum = reinterpret_cast<uint64_t*>(w);
  w += up(8ull * a.ntiles);
  uint64_t* prefix_tmp = reinterpret_cast<uint64_t*>(w);
  w += up(8ull * N);
  a.misc = reinterpret_cast<uint64_t*>(w);
  a.order = order;
  a.prefix = prefix ? prefix : prefix_tmp;
  a.result = result;
  const uint32_t tiles = a.ntiles ? a.ntiles : 1;
  hipLaunchKernelGGL(evict_init_kernel, dim3(1), dim3(1), 0, s, a);
  hipLaunchKernelGGL(evict_keys_kernel, dim3(tiles < 2048 ? tiles * 4 : 8192), dim3(ET), 0, s, a);
  int src = 0;
  for (int shift = 0; shift < 64; shift += 8) {
    if (a.ntiles) {
      hipLaunchKernelGGL(evict_hist_kernel, dim3(a.ntiles), dim3(ET), 0, s, a, src, shift);
      hipLaunchKernelGGL(evict_scan_kernel, dim3(1), dim3(1024), 0, s, a, shift);
      hipLaunchKernelGGL(evict_scatter_kernel, dim3(a.ntiles), dim3(ET), 0, s, a, src, shift);
    }
    src ^= 1;
  }
  if (a.ntiles) {
    hipLaunchKernelGGL(evict_prefix_tiles_kernel, dim3(a.ntiles), dim3(ET), 0, s, a, src);
    hipLaunchKernelGGL(evict_prefix_top_kernel, dim3(1), dim3(1024), 0, s, a);
    hipLaunchKernelGGL(evict_prefix_fix_kernel, dim3(a.ntiles), dim3(ET), 0, s, a);
  }
  hipLaunchKernelGGL(evict_result_kernel, dim3(1), dim3(1), 0, s, a);
  return hipGetLastError();
}

}  // namespace mori
