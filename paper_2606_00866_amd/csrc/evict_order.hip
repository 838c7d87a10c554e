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
//   keys     build keys, validate, OR/AND of all keys; for the one-kernel
//            passes also the digit counts of all eight passes at once (they
//            do not depend on the order), one set per workgroup, equal keys
//            (the blocks of a program share their time) counted once per run;
//   totals   those counts summed over the keys workgroups;
//   per pass (8-bit digit, 8 passes; a digit on which every key agrees needs
//   no pass, and each kernel works out from the OR/AND which of the two
//   key/value buffers holds the current order, so such a pass is empty
//   launches and no memory traffic), one workgroup per tile, in one of two
//   forms by tile count:
//     one kernel (up to ONESWEEP_TILES tiles):
//     - the tile index comes from a counter in the order workgroups start, so
//       every lower tile belongs to a workgroup that is already running;
//     - the stable rank of every key among the tile's keys of its digit:
//       wave64 ballots over the 8 digit bits rank it within its wave's 64
//       keys of a slice, one scan per digit over (slice, wave) in LDS orders
//       the groups as the keys were ordered;
//     - the tile's count of each digit is published, then the keys of that
//       digit in all lower tiles are summed by looking back over the
//       published counts, four tiles per round, until a tile that already
//       holds its inclusive sum (a decoupled look-back; the wait is bounded
//       and reports a stall);
//     - position = digit base (a 256-entry scan of the digit totals) + keys
//       of the digit in lower tiles + the rank in the tile;
//     three kernels (more tiles):
//     - hist: per tile, a 256-bin histogram -> hist[digit][tile];
//     - dscan: one workgroup per digit, an exclusive scan of that digit's
//       counts over the tiles and the digit's total;
//     - scatter: the same ranking and position, with the lower tiles' count
//       read from the scanned histogram;
//   prefix   inclusive u64 scan of block bytes in eviction order (tile scans,
//            then a fix-up whose workgroups each sum the tile totals below
//            their tile, or above FIX_SCAN_TILES a one-workgroup scan of the
//            tile totals first) and the number of evictions that frees the
//            requested bytes.
//
// Everything is latency-bound at 10^5-10^6 blocks (tens of microseconds);
// the workspace is the caller's, so nothing is allocated here.
#include "mori_internal.h"
#include "wave.h"

namespace mori {
namespace {

constexpr int ET = EVICT_WG;            // threads per tile workgroup
constexpr int ENW = ET / 64;            // waves per tile workgroup
// Keys per thread (tile = 256 x that), measured with the bench's block metadata.
inline int keys_per_thread(uint32_t N) { return evict_keys_per_thread(N); }
constexpr uint64_t TIME_LIMIT = 1ull << 62;
constexpr uint32_t KEY_WG_MAX = EVICT_KEY_WG_MAX;  // workgroups of the keys kernel at most (one digit-count set each)
// Keys per thread whose loads the keys kernel issues together: 4 for the
// look-back passes, 8 above (measured: 8 and 16 are 3 and 11 us slower at
// 69 938 blocks, 8 is 2.5 us faster at 2^20).
constexpr int KEYS_PER_ROUND_SMALL = 4, KEYS_PER_ROUND_LARGE = 8;
constexpr uint32_t TOT_SPLIT = 8;        // totals: workgroups per pass, each summing a share of the sets
// Tile counts up to this use one look-back kernel per pass, more use three
// kernels (histogram, per-digit scan, scatter): each look-back round is a
// device-coherent load, so the look-back chains grow with the tile count.
constexpr uint32_t ONESWEEP_TILES = 128;
// Tile counts up to this finish the prefix with one kernel (every workgroup
// reads the tile totals: 8 B each) instead of a tile scan, a fix-up and a
// result kernel.
constexpr uint32_t FIX_SCAN_TILES = 1024;
constexpr uint64_t ST_AGG = 1ull << 32;  // status flags: the tile's own count ...
constexpr uint64_t ST_INCL = 2ull << 32; // ... or its inclusive count over tiles 0..t
constexpr uint32_t SPIN_LIMIT = 1u << 22;  // polls of one status word before reporting a stall

struct EvictArgs {
  uint32_t N, ntiles, tier;
  const uint8_t* type;
  const uint64_t* last_access;
  const uint32_t* size;
  uint64_t unit_bytes, need;
  uint64_t* keys[2];
  uint32_t* vals[2];
  uint32_t* hist;       // [256][ntiles] (three-kernel passes)
  uint32_t* dtot;       // [256] keys per digit (three-kernel passes)
  uint32_t onesweep;    // passes are single look-back kernels (few tiles)
  uint64_t* status[2];  // [ntiles][256] per pass: (flag << 32) | count; passes alternate the two
  uint32_t* part;       // [key_wg][8][256] digit counts of each keys workgroup, all passes
  uint32_t* gtot;       // [8][256] keys per digit, all passes
  uint32_t key_wg;      // workgroups of the keys kernel
  uint32_t* tile_ctr;   // [8] tiles taken in each pass
  uint64_t* tile_sum;   // [ntiles]
  uint64_t* misc;       // [0] OR of keys, [1] AND of keys, [2] error bits, [3] evictions short of need
  uint32_t* order;      // out [N]
  uint64_t* prefix;     // out [N] (or workspace)
  uint32_t* result;     // out [2]: count, error bits
};

__global__ __launch_bounds__(ET) void evict_init_kernel(EvictArgs a) {
  // status of the first pass that runs, and the tile counters
  for (uint64_t i = (uint64_t)blockIdx.x * ET + threadIdx.x; i < (uint64_t)a.ntiles * 256; i += (uint64_t)gridDim.x * ET)
    a.status[0][i] = 0;
  for (uint32_t i = blockIdx.x * ET + threadIdx.x; i < 8 * 256; i += gridDim.x * ET) a.gtot[i] = 0;
  if (blockIdx.x == 0) {
    if (threadIdx.x < 8) a.tile_ctr[threadIdx.x] = 0;
    if (threadIdx.x == 0) {
      a.misc[0] = 0;
      a.misc[1] = ~0ull;
      a.misc[2] = 0;
      a.misc[3] = 0;
    }
  }
}

template <int KEYS_PER_ROUND>
__global__ __launch_bounds__(ET) void evict_keys_kernel(EvictArgs a) {
  // position of each type label in the tier's eviction order (busy, idle, inactive)
  const uint32_t gpu_pos[3] = {2, 1, 0}, cpu_pos[3] = {1, 2, 0};
  const uint32_t* pos = a.tier == MORI_TIER_GPU ? gpu_pos : cpu_pos;
  __shared__ uint32_t s_c[8][256];  // this workgroup's keys per (pass, digit)
#pragma unroll
  for (int k = 0; k < 8; ++k) s_c[k][threadIdx.x] = 0;
  __syncthreads();
  uint64_t o = 0, n = ~0ull, err = 0;
  const int lane = threadIdx.x & 63;
  // rounds of KEYS_PER_ROUND keys per thread, all their loads issued first;
  // uniform trip count: the cross-lane steps below need every lane of the wave
  for (uint64_t i0 = (uint64_t)blockIdx.x * ET * KEYS_PER_ROUND; i0 < a.N;
       i0 += (uint64_t)gridDim.x * ET * KEYS_PER_ROUND) {
    uint8_t typ[KEYS_PER_ROUND];
    uint64_t la[KEYS_PER_ROUND];
#pragma unroll
    for (int u = 0; u < KEYS_PER_ROUND; ++u) {
      const uint64_t i = i0 + (uint64_t)u * ET + threadIdx.x;
      typ[u] = i < a.N ? a.type[i] : 0;
      la[u] = i < a.N ? a.last_access[i] : 0;
    }
#pragma unroll
    for (int u = 0; u < KEYS_PER_ROUND; ++u) {
      const uint64_t i = i0 + (uint64_t)u * ET + threadIdx.x;
      bool valid = i < a.N;
      uint64_t key = 0;
      if (valid) {
        if (typ[u] > MORI_TYPE_INACTIVE || la[u] >= TIME_LIMIT) {
          err |= MORI_DEV_BAD_BLOCK;
          valid = false;
        } else {
          key = ((uint64_t)pos[typ[u]] << 62) | la[u];
          a.keys[0][i] = key;
          a.vals[0][i] = (uint32_t)i;
          o |= key;
          n &= key;
        }
      }
      if (!a.onesweep) continue;  // uniform: the three-kernel passes count per tile
      // runs of equal keys within the wave (the blocks of a program share their
      // time): the first lane of a run adds the run's length for each digit
      const uint64_t prev = __shfl_up(key, 1, 64);
      const bool prev_valid = __shfl_up(valid ? 1 : 0, 1, 64) != 0;
      const bool head = valid && (lane == 0 || !prev_valid || prev != key);
      const uint64_t heads = __ballot(head);
      const uint64_t vmask = __ballot(valid);
      if (!heads) continue;  // uniform: no valid key in this wave
      const uint64_t ends = heads | ~vmask;  // a run ends at the next head or invalid lane
      uint32_t len = 0;
      if (head) {
        const uint64_t later = lane == 63 ? 0ull : ends & ~((2ull << lane) - 1ull);
        len = (later ? (uint32_t)__builtin_ctzll(later) : 64u) - (uint32_t)lane;
      }
      // a digit that every run of the wave shares (the high time digits and
      // the type, mostly) takes one increment of all the wave's valid keys
      const int first = __builtin_ctzll(heads);
#pragma unroll
      for (int k = 0; k < 8; ++k) {
        const uint32_t d = (uint32_t)(key >> (8 * k)) & 255u;
        const uint32_t d0 = (uint32_t)__builtin_amdgcn_readlane((int)d, first);
        if (__ballot(head && d != d0) == 0) {
          if (lane == first) atomicAdd(&s_c[k][d0], (uint32_t)__popcll(vmask));
        } else if (head) {
          atomicAdd(&s_c[k][d], len);
        }
      }
    }
  }
  __syncthreads();
  if (a.onesweep)
#pragma unroll
    for (int k = 0; k < 8; ++k) a.part[((uint64_t)blockIdx.x * 8 + k) * 256 + threadIdx.x] = s_c[k][threadIdx.x];
  // wave, then workgroup reduction: one set of global atomics per workgroup
  __shared__ uint64_t s_red[3][ENW];
  o = wave::all_or<uint64_t>(o);
  n = wave::all_and<uint64_t>(n);
  err = wave::all_or<uint64_t>(err);
  const int wid = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) {
    s_red[0][wid] = o;
    s_red[1][wid] = n;
    s_red[2][wid] = err;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    for (int w = 1; w < ENW; ++w) {
      o |= s_red[0][w];
      n &= s_red[1][w];
      err |= s_red[2][w];
    }
    atomicOr((unsigned long long*)&a.misc[0], (unsigned long long)o);
    atomicAnd((unsigned long long*)&a.misc[1], (unsigned long long)n);
    if (err) atomicOr((unsigned long long*)&a.misc[2], (unsigned long long)err);
  }
}

__device__ inline uint64_t varying_bits(const EvictArgs& a) { return a.misc[0] ^ a.misc[1]; }

__device__ inline bool digit_varies(const EvictArgs& a, int shift) {
  return ((varying_bits(a) >> shift) & 255u) != 0;
}

// Which buffer holds the order before the pass at `shift`: passes over
// constant digits are skipped, so it is the parity of the varying digits below.
__device__ inline int source_buffer(const EvictArgs& a, int shift) {
  const uint64_t v = varying_bits(a);
  int n = 0;
  for (int s = 0; s < shift; s += 8) n += ((v >> s) & 255u) != 0;
  return n & 1;
}

template <int EIPT>
__global__ __launch_bounds__(ET) void evict_hist_kernel(EvictArgs a, int shift) {
  __shared__ uint32_t s_h[256];
  if (a.misc[2] || !digit_varies(a, shift)) return;
  s_h[threadIdx.x] = 0;
  __syncthreads();
  const uint64_t* k = a.keys[source_buffer(a, shift)];
  const uint64_t base = (uint64_t)blockIdx.x * (ET * EIPT);
  const uint64_t lanemask_lt = (1ull << (threadIdx.x & 63)) - 1ull;
#pragma unroll
  for (int it = 0; it < EIPT; ++it) {
    // keys of a program share their time, so digits repeat within a wave: one
    // LDS increment per distinct digit (its first lane adds the group's size)
    const uint64_t i = base + it * ET + threadIdx.x;
    const bool valid = i < a.N;
    const uint32_t d = valid ? (uint32_t)(k[i] >> shift) & 255u : 0u;
    const uint64_t same = __ballot(valid) & ~wave::digit_differs<8>(d);
    if (valid && (same & lanemask_lt) == 0) atomicAdd(&s_h[d], (uint32_t)__popcll(same));
  }
  __syncthreads();
  a.hist[(uint64_t)threadIdx.x * a.ntiles + blockIdx.x] = s_h[threadIdx.x];
}

// Block-wide exclusive scan of one u32 per thread (256 threads); *total gets the sum.
__device__ inline uint32_t scan256(uint32_t v, uint32_t* s_w, uint32_t* total) {
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
  const uint32_t x = wave::incl_add(v);
  if (lane == 63) s_w[wid] = x;
  __syncthreads();
  uint32_t before = 0, all = 0;
#pragma unroll
  for (int w = 0; w < ENW; ++w) {
    before += w < wid ? s_w[w] : 0u;
    all += s_w[w];
  }
  __syncthreads();
  *total = all;
  return before + x - v;
}

// The tile's keys to their global positions, staged through LDS in the
// tile's digit order so that each wave's stores cover a few contiguous runs
// (one per digit it meets) instead of one scattered 8-byte store per lane.
// s_tstart[d]: first tile-local slot of digit d; s_off[d]: its global slot;
// s_cnt: the (slice, wave, digit) offsets within each digit; n: valid keys.
// Every thread calls it; it begins and ends with a barrier.
template <int EIPT>
__device__ void store_tile(const uint64_t (&key)[EIPT], const uint32_t (&val)[EIPT], const uint32_t (&dig)[EIPT],
                           const uint32_t (&rnk)[EIPT], const uint16_t (*s_cnt)[ENW][256], const uint32_t* s_tstart,
                           const uint32_t* s_off, uint64_t* s_k, uint32_t* s_v, uint32_t n, int shift, uint64_t* kd,
                           uint32_t* vd) {
  const int tid = threadIdx.x, wid = tid >> 6;
  __syncthreads();
#pragma unroll
  for (int it = 0; it < EIPT; ++it) {
    const uint32_t d = dig[it];
    if (d < 256u) {
      const uint32_t local = s_tstart[d] + s_cnt[it][wid][d] + rnk[it];
      s_k[local] = key[it];
      s_v[local] = val[it];
    }
  }
  __syncthreads();
#pragma unroll
  for (int j = 0; j < EIPT; ++j) {
    const uint32_t local = j * ET + tid;
    if (local < n) {
      const uint64_t k = s_k[local];
      const uint32_t d = (uint32_t)(k >> shift) & 255u;
      const uint32_t pos = s_off[d] + (local - s_tstart[d]);
      kd[pos] = k;
      vd[pos] = s_v[local];
    }
  }
}

// One workgroup per digit: exclusive scan of hist[digit][0..ntiles) in place
// and the digit's total.
__global__ __launch_bounds__(ET) void evict_dscan_kernel(EvictArgs a, int shift) {
  __shared__ uint32_t s_w[ENW];
  if (a.misc[2] || !digit_varies(a, shift)) return;
  uint32_t* h = a.hist + (uint64_t)blockIdx.x * a.ntiles;
  uint32_t carry = 0;
  for (uint32_t t0 = 0; t0 < a.ntiles; t0 += ET) {
    const uint32_t t = t0 + threadIdx.x;
    const uint32_t v = t < a.ntiles ? h[t] : 0u;
    uint32_t tot;
    const uint32_t ex = scan256(v, s_w, &tot);
    if (t < a.ntiles) h[t] = carry + ex;
    carry += tot;
  }
  if (threadIdx.x == 0) a.dtot[blockIdx.x] = carry;
}

template <int EIPT>
__global__ __launch_bounds__(ET) void evict_scatter_kernel(EvictArgs a, int shift) {
  // s_cnt[slice][wave][digit]: keys of that digit in that wave's 64 keys of the
  // slice, then (after the per-digit scan) their offset within the tile
  __shared__ uint16_t s_cnt[EIPT][ENW][256];
  __shared__ uint32_t s_off[256];     // this tile's global base per digit
  __shared__ uint32_t s_tstart[256];  // ... and its first slot within the tile
  __shared__ uint64_t s_k[ET * EIPT];
  __shared__ uint32_t s_v[ET * EIPT];
  __shared__ uint32_t s_w[ENW];
  if (a.misc[2] || !digit_varies(a, shift)) return;
  const int src = source_buffer(a, shift);
  const uint64_t* ks = a.keys[src];
  const uint32_t* vs = a.vals[src];
  uint64_t* kd = a.keys[src ^ 1];
  uint32_t* vd = a.vals[src ^ 1];
  const uint64_t base = (uint64_t)blockIdx.x * (ET * EIPT);
  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  uint32_t tot;
  const uint32_t before = a.hist[(uint64_t)tid * a.ntiles + blockIdx.x];  // scanned by evict_dscan_kernel
  const uint32_t total_d = a.dtot[tid];
  const uint32_t digit_base = scan256(total_d, s_w, &tot);
  s_off[tid] = digit_base + before;
#pragma unroll
  for (int it = 0; it < EIPT; ++it)
#pragma unroll
    for (int w = 0; w < ENW; ++w) s_cnt[it][w][tid] = 0;
  __syncthreads();
  // rank of every key among the keys of its digit in its wave's slice (ballots)
  const uint64_t lanemask_lt = (1ull << lane) - 1ull;
  uint64_t key[EIPT];
  uint32_t val[EIPT], dig[EIPT], rnk[EIPT];
#pragma unroll
  for (int it = 0; it < EIPT; ++it) {
    const uint64_t i = base + it * ET + tid;
    const bool valid = i < a.N;
    key[it] = valid ? ks[i] : 0ull;
    val[it] = valid ? vs[i] : 0u;
    const uint32_t d = (uint32_t)(key[it] >> shift) & 255u;
    const uint64_t same = __ballot(valid) & ~wave::digit_differs<8>(d);
    const uint32_t r = __popcll(same & lanemask_lt);
    if (valid && r == 0) s_cnt[it][wid][d] = (uint16_t)__popcll(same);
    dig[it] = valid ? d : 256u;
    rnk[it] = r;
  }
  __syncthreads();
  uint32_t run = 0;  // per digit (one per thread): offsets in (slice, wave) order, i.e. original key order
#pragma unroll
  for (int it = 0; it < EIPT; ++it)
#pragma unroll
    for (int w = 0; w < ENW; ++w) {
      const uint32_t c = s_cnt[it][w][tid];
      s_cnt[it][w][tid] = (uint16_t)run;
      run += c;
    }
  uint32_t n;
  s_tstart[tid] = scan256(run, s_w, &n);
  store_tile<EIPT>(key, val, dig, rnk, s_cnt, s_tstart, s_off, s_k, s_v, n, shift, kd, vd);
}

// Keys per digit of every pass: workgroup (pass, share) sums a share of the
// keys workgroups' counts, one digit per thread.
__global__ __launch_bounds__(ET) void evict_totals_kernel(EvictArgs a) {
  const uint32_t k = blockIdx.x / TOT_SPLIT, j = blockIdx.x % TOT_SPLIT;
  uint32_t sum = 0;
  for (uint32_t g = j; g < a.key_wg; g += TOT_SPLIT) sum += a.part[((uint64_t)g * 8 + k) * 256 + threadIdx.x];
  if (sum) atomicAdd(&a.gtot[k * 256 + threadIdx.x], sum);
}

__device__ inline void status_store(uint64_t* p, uint64_t v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ inline uint64_t status_load(const uint64_t* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// One pass of the sort (the digit at `shift`), one workgroup per tile.
template <int EIPT>
__global__ __launch_bounds__(ET) void evict_pass_kernel(EvictArgs a, int shift) {
  // s_cnt[slice][wave][digit]: keys of that digit in that wave's 64 keys of the
  // slice, then (after the per-digit scan) their offset within the tile
  __shared__ uint16_t s_cnt[EIPT][ENW][256];
  __shared__ uint32_t s_off[256];  // this tile's global base per digit
  __shared__ uint32_t s_w[ENW];
  __shared__ uint32_t s_tile;
  if (a.misc[2] || !digit_varies(a, shift)) return;
  const int src = source_buffer(a, shift);  // the parity of this pass among those that run
  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  if (tid == 0) s_tile = atomicAdd(&a.tile_ctr[shift >> 3], 1u);
#pragma unroll
  for (int it = 0; it < EIPT; ++it)
#pragma unroll
    for (int w = 0; w < ENW; ++w) s_cnt[it][w][tid] = 0;
  const uint32_t total_d = a.gtot[(shift >> 3) * 256 + tid];  // keys of this digit in all tiles
  __syncthreads();
  const uint32_t tile = s_tile;
  // the next pass that runs uses the other status array; the previous one that
  // used it has finished
  a.status[src ^ 1][(uint64_t)tile * 256 + tid] = 0;
  const uint64_t* ks = a.keys[src];
  const uint32_t* vs = a.vals[src];
  uint64_t* kd = a.keys[src ^ 1];
  uint32_t* vd = a.vals[src ^ 1];
  const uint64_t base = (uint64_t)tile * (ET * EIPT);
  // rank of every key among the keys of its digit in its wave's slice (ballots)
  const uint64_t lanemask_lt = (1ull << lane) - 1ull;
  uint64_t key[EIPT];
  uint32_t val[EIPT], dig[EIPT], rnk[EIPT];
#pragma unroll
  for (int it = 0; it < EIPT; ++it) {
    const uint64_t i = base + it * ET + tid;
    const bool valid = i < a.N;
    key[it] = valid ? ks[i] : 0ull;
    val[it] = valid ? vs[i] : 0u;
    const uint32_t d = (uint32_t)(key[it] >> shift) & 255u;
    const uint64_t same = __ballot(valid) & ~wave::digit_differs<8>(d);
    const uint32_t r = __popcll(same & lanemask_lt);
    if (valid && r == 0) s_cnt[it][wid][d] = (uint16_t)__popcll(same);
    dig[it] = valid ? d : 256u;
    rnk[it] = r;
  }
  __syncthreads();
  // per digit (one per thread): offsets in (slice, wave) order, i.e. original
  // key order, and the tile's count of the digit
  uint32_t run = 0;
#pragma unroll
  for (int it = 0; it < EIPT; ++it)
#pragma unroll
    for (int w = 0; w < ENW; ++w) {
      const uint32_t c = s_cnt[it][w][tid];
      s_cnt[it][w][tid] = (uint16_t)run;
      run += c;
    }
  // publish, then look back over the lower tiles
  uint64_t* st = a.status[src];
  uint64_t* mine = st + (uint64_t)tile * 256 + tid;
  uint32_t before = 0;
  if (tile == 0) {
    status_store(mine, ST_INCL | run);
  } else {
    status_store(mine, ST_AGG | run);
    // rounds of four tiles below the next unaccounted one, loaded at once and
    // taken in order: counts add up until a tile holding its inclusive sum; a
    // tile that has not published yet ends the round and is polled again
    constexpr int LB = 4;  // measured: 2 and 4 alike, 8 1-2 us slower, 16 15-20 us slower
    uint32_t next = tile;  // tiles next..tile-1 are accounted for
    uint32_t spins = 0;
    bool done = false;
    while (!done) {
      uint64_t w[LB];
#pragma unroll
      for (int j = 0; j < LB; ++j)
        w[j] = next > (uint32_t)j ? status_load(st + (uint64_t)(next - 1 - j) * 256 + tid) : ST_INCL;
      int used = 0;
#pragma unroll
      for (int j = 0; j < LB; ++j) {
        if (used < j) break;  // an earlier entry of this round was not ready
        const uint64_t flag = w[j] >> 32;
        if (flag == 0) break;
        before += (uint32_t)w[j];
        used = j + 1;
        if (flag == (ST_INCL >> 32)) {
          done = true;
          break;
        }
      }
      next -= (uint32_t)used;
      if (!done && used < LB) {  // the tile below `next` has not published yet
        if (++spins > SPIN_LIMIT) {
          atomicOr((unsigned long long*)&a.misc[2], (unsigned long long)MORI_DEV_STALL);
          break;
        }
        __builtin_amdgcn_s_sleep(1);
      }
    }
    status_store(mine, ST_INCL | (uint64_t)(before + run));
  }
  // stores straight from registers: at up to 128 tiles, staging them through
  // LDS in digit order (as the three-kernel scatter does) measured slower
  uint32_t tot;
  const uint32_t digit_base = scan256(total_d, s_w, &tot);
  s_off[tid] = digit_base + before;
  __syncthreads();
#pragma unroll
  for (int it = 0; it < EIPT; ++it) {
    const uint32_t d = dig[it];
    if (d < 256u) {
      const uint32_t pos = s_off[d] + s_cnt[it][wid][d] + rnk[it];
      kd[pos] = key[it];
      vd[pos] = val[it];
    }
  }
}

// Inclusive scan of freed bytes within each tile; tile totals to tile_sum.
// Global memory is read and written in striped (coalesced) order and the
// blocked per-thread scan runs on an LDS copy of the tile.
template <int EIPT>
__global__ __launch_bounds__(ET) void evict_prefix_tiles_kernel(EvictArgs a) {
  __shared__ uint64_t s_b[ET * EIPT];
  __shared__ uint64_t s_w[ENW + 1];
  if (a.misc[2]) return;
  const uint32_t* order = a.vals[source_buffer(a, 64)];
  const uint64_t base = (uint64_t)blockIdx.x * (ET * EIPT);
  const int tid = threadIdx.x;
#pragma unroll
  for (int it = 0; it < EIPT; ++it) {
    const uint64_t i = base + it * ET + tid;
    uint64_t bytes = 0;
    if (i < a.N) {
      const uint32_t b = order[i];
      a.order[i] = b;
      bytes = (uint64_t)(a.size ? a.size[b] : 1u) * a.unit_bytes;
    }
    s_b[it * ET + tid] = bytes;
  }
  __syncthreads();
  uint64_t v[EIPT];
  uint64_t sum = 0;
#pragma unroll
  for (int j = 0; j < EIPT; ++j) {  // blocked: keys tid * EIPT .. + EIPT - 1 of the tile
    sum += s_b[tid * EIPT + j];
    v[j] = sum;
  }
  // exclusive scan of the per-thread totals
  const int lane = tid & 63, wid = tid >> 6;
  const uint64_t x = wave::incl_add(sum);
  if (lane == 63) s_w[wid] = x;
  __syncthreads();
  if (tid == 0) {
    uint64_t run = 0;
    for (int w = 0; w < ENW; ++w) {
      const uint64_t c = s_w[w];
      s_w[w] = run;
      run += c;
    }
    s_w[ENW] = run;
  }
  __syncthreads();
  const uint64_t before = s_w[wid] + x - sum;
#pragma unroll
  for (int j = 0; j < EIPT; ++j) s_b[tid * EIPT + j] = before + v[j];
  __syncthreads();
#pragma unroll
  for (int it = 0; it < EIPT; ++it) {
    const uint64_t i = base + it * ET + tid;
    if (i < a.N) a.prefix[i] = s_b[it * ET + tid];
  }
  if (tid == 0) a.tile_sum[blockIdx.x] = s_w[ENW];
}

__global__ __launch_bounds__(1024) void evict_prefix_top_kernel(EvictArgs a) {
  __shared__ uint64_t s_w[1024 / 64 + 1];
  if (a.misc[2]) return;
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
  uint64_t carry = 0;
  for (uint32_t t0 = 0; t0 < a.ntiles; t0 += 1024) {
    const uint32_t t = t0 + threadIdx.x;
    const uint64_t v = t < a.ntiles ? a.tile_sum[t] : 0ull;
    const uint64_t x = wave::incl_add(v);
    if (lane == 63) s_w[wid] = x;
    __syncthreads();
    if (wid == 0) {
      const uint64_t w = lane < 16 ? s_w[lane] : 0ull;
      const uint64_t wi = wave::incl_add(w);
      if (lane < 16) s_w[lane] = wi - w;
      if (lane == 15) s_w[16] = wi;
    }
    __syncthreads();
    if (t < a.ntiles) a.tile_sum[t] = carry + s_w[wid] + x - v;  // exclusive base of tile t
    carry += s_w[16];
    __syncthreads();
  }
}

template <int EIPT>
__global__ __launch_bounds__(ET) void evict_prefix_fix_kernel(EvictArgs a) {
  if (a.misc[2]) return;
  const uint64_t add = a.tile_sum[blockIdx.x];
  const uint64_t base = (uint64_t)blockIdx.x * (ET * EIPT);
  uint32_t short_of_need = 0;
  for (int it = 0; it < EIPT; ++it) {
    const uint64_t i = base + it * ET + threadIdx.x;
    if (i < a.N) {
      const uint64_t p = a.prefix[i] + add;
      a.prefix[i] = p;
      short_of_need += p < a.need;
    }
  }
  __shared__ uint32_t s_short[ENW];
  short_of_need = wave::sum(short_of_need);
  if ((threadIdx.x & 63) == 0) s_short[threadIdx.x >> 6] = short_of_need;
  __syncthreads();
  if (threadIdx.x == 0) {
    uint32_t t = 0;
    for (int w = 0; w < ENW; ++w) t += s_short[w];
    if (t) atomicAdd((unsigned long long*)&a.misc[3], (unsigned long long)t);
  }
}

// Up to FIX_SCAN_TILES tiles: the fix-up workgroups scan the tile totals
// themselves (each sums the totals below its tile) and the result comes from
// the one workgroup whose tile holds the first prefix >= need (the prefix never
// decreases, so that tile is unique; without one, the last tile's workgroup
// reports every block), so neither the one-workgroup tile scan nor the result
// kernel runs.
template <int EIPT>
__global__ __launch_bounds__(ET) void evict_prefix_fix_scan_kernel(EvictArgs a) {
  __shared__ uint64_t s_red[ENW][2];
  if (a.misc[2]) {
    if (blockIdx.x == 0 && threadIdx.x == 0) {
      a.result[0] = 0;
      a.result[1] = (uint32_t)a.misc[2];
    }
    return;
  }
  uint64_t below = 0, all = 0;  // totals of the tiles below this one, and of every tile
  for (uint32_t t = threadIdx.x; t < a.ntiles; t += ET) {
    const uint64_t v = a.tile_sum[t];
    if (t < blockIdx.x) below += v;
    all += v;
  }
  below = wave::sum(below);
  all = wave::sum(all);
  if ((threadIdx.x & 63) == 0) {
    s_red[threadIdx.x >> 6][0] = below;
    s_red[threadIdx.x >> 6][1] = all;
  }
  __syncthreads();
  below = all = 0;
#pragma unroll
  for (int w = 0; w < ENW; ++w) {
    below += s_red[w][0];
    all += s_red[w][1];
  }
  const uint64_t base = (uint64_t)blockIdx.x * (ET * EIPT);
  uint32_t short_of_need = 0;
  for (int it = 0; it < EIPT; ++it) {
    const uint64_t i = base + it * ET + threadIdx.x;
    if (i < a.N) {
      const uint64_t p = a.prefix[i] + below;
      a.prefix[i] = p;
      short_of_need += p < a.need;
    }
  }
  __syncthreads();  // s_red is reused
  short_of_need = wave::sum(short_of_need);
  if ((threadIdx.x & 63) == 0) s_red[threadIdx.x >> 6][0] = short_of_need;
  __syncthreads();
  if (threadIdx.x == 0) {
    uint64_t c = 0;
    for (int w = 0; w < ENW; ++w) c += s_red[w][0];
    const uint64_t len = a.N - base < (uint64_t)(ET * EIPT) ? a.N - base : (uint64_t)(ET * EIPT);
    const bool last = blockIdx.x == a.ntiles - 1;
    if (blockIdx.x == 0) a.result[1] = 0;
    if (a.need == 0) {
      if (blockIdx.x == 0) a.result[0] = 0;
    } else if (below < a.need && c < len) {  // the first prefix >= need is in this tile
      a.result[0] = (uint32_t)(base + c + 1);
    } else if (last && all < a.need) {  // no prefix reaches need: every block
      a.result[0] = a.N;
    }
  }
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

template <int EIPT>
void launch_tiles(const EvictArgs& a, hipStream_t s) {
  for (int shift = 0; shift < 64; shift += 8) {
    if (a.onesweep) {
      hipLaunchKernelGGL(evict_pass_kernel<EIPT>, dim3(a.ntiles), dim3(ET), 0, s, a, shift);
    } else {
      hipLaunchKernelGGL(evict_hist_kernel<EIPT>, dim3(a.ntiles), dim3(ET), 0, s, a, shift);
      hipLaunchKernelGGL(evict_dscan_kernel, dim3(256), dim3(ET), 0, s, a, shift);
      hipLaunchKernelGGL(evict_scatter_kernel<EIPT>, dim3(a.ntiles), dim3(ET), 0, s, a, shift);
    }
  }
  hipLaunchKernelGGL(evict_prefix_tiles_kernel<EIPT>, dim3(a.ntiles), dim3(ET), 0, s, a);
  if (a.ntiles <= FIX_SCAN_TILES) {
    hipLaunchKernelGGL(evict_prefix_fix_scan_kernel<EIPT>, dim3(a.ntiles), dim3(ET), 0, s, a);
  } else {
    hipLaunchKernelGGL(evict_prefix_top_kernel, dim3(1), dim3(1024), 0, s, a);
    hipLaunchKernelGGL(evict_prefix_fix_kernel<EIPT>, dim3(a.ntiles), dim3(ET), 0, s, a);
    hipLaunchKernelGGL(evict_result_kernel, dim3(1), dim3(1), 0, s, a);
  }
}

}  // namespace

hipError_t launch_evict(uint32_t N, const uint8_t* type, const uint64_t* last_access, const uint32_t* size,
                        uint64_t unit_bytes, uint32_t tier, uint64_t need, void* workspace, uint32_t* order,
                        uint64_t* prefix, uint32_t* result, hipStream_t s) {
  EvictArgs a{};
  a.N = N;
  const int kpt = keys_per_thread(N);
  const uint64_t tile = (uint64_t)ET * kpt;
  a.ntiles = (uint32_t)(((uint64_t)N + tile - 1) / tile);
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
  a.dtot = reinterpret_cast<uint32_t*>(w);
  w += up(4 * 256);
  a.onesweep = a.ntiles <= ONESWEEP_TILES;
  for (int b = 0; b < 2; ++b) {
    a.status[b] = reinterpret_cast<uint64_t*>(w);
    w += up(8ull * 256 * a.ntiles);
  }
  a.part = reinterpret_cast<uint32_t*>(w);
  w += up(4ull * KEY_WG_MAX * 8 * 256);
  a.gtot = reinterpret_cast<uint32_t*>(w);
  w += up(4 * 8 * 256);
  a.tile_ctr = reinterpret_cast<uint32_t*>(w);
  w += up(4 * 8);
  a.tile_sum = reinterpret_cast<uint64_t*>(w);
  w += up(8ull * a.ntiles);
  uint64_t* prefix_tmp = reinterpret_cast<uint64_t*>(w);
  w += up(8ull * N);
  a.misc = reinterpret_cast<uint64_t*>(w);
  a.order = order;
  a.prefix = prefix ? prefix : prefix_tmp;
  a.result = result;
  const uint32_t tiles = a.ntiles ? a.ntiles : 1;
  hipLaunchKernelGGL(evict_init_kernel, dim3(tiles < 256 ? tiles : 256), dim3(ET), 0, s, a);
  a.key_wg = tiles < KEY_WG_MAX ? tiles : KEY_WG_MAX;
  if (a.onesweep) hipLaunchKernelGGL(evict_keys_kernel<KEYS_PER_ROUND_SMALL>, dim3(a.key_wg), dim3(ET), 0, s, a);
  else hipLaunchKernelGGL(evict_keys_kernel<KEYS_PER_ROUND_LARGE>, dim3(a.key_wg), dim3(ET), 0, s, a);
  if (a.onesweep) hipLaunchKernelGGL(evict_totals_kernel, dim3(8 * TOT_SPLIT), dim3(ET), 0, s, a);
  if (a.ntiles) {
    if (kpt == 4) launch_tiles<4>(a, s);
    else launch_tiles<8>(a, s);
  } else {
    hipLaunchKernelGGL(evict_result_kernel, dim3(1), dim3(1), 0, s, a);
  }
  return hipGetLastError();
}

}  // namespace mori
