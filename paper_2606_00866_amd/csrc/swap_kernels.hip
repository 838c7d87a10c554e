// Byte movement of one rebalance.
//
// A "unit" is one run: the block_tokens * row_bytes contiguous bytes of one
// (plane, page).  Units are numbered program-major in rank order,
//     unit = pg_base[a] * LC + q * nblk + i
// for the a-th moving program, plane q, logical block i, so consecutive units
// land on consecutive bytes of that program's host buffer ([plane][block]
// layout) or of the staging buffer, while the pool side is scattered over the
// program's pages.  Each workgroup copies whole units with 16-byte
// non-temporal loads and stores (every byte is touched once, so nothing is
// worth caching); the index arithmetic is wavefront-uniform.  A grid of
// workgroups walks the units with a grid stride.  A run is copied in rounds by
// a group of whole wavefronts (the whole workgroup for long runs between HBM
// buffers, half of it over the host link, smaller groups for short runs):
// each thread issues all its loads of a round, then its stores, then waits
// for the stores before the next round.
//
//   swap_out : pool page  -> host buffer (direct) or staging (copy engine)
//   swap_in  : host buffer (direct) or staging -> newly allocated pool page
//
// Swap-in is launched in two parts in direct mode: slots taken from pages
// that were free before the step or released by idle programs dropped to
// Waiting, which nothing uses any more, and slots taken from pages that are
// free only once the swap-out stream has passed (pages the swap-out reads,
// and pages of dropped programs whose inference step the caller orders
// before the swap-out), which must wait for the swap-out (the host orders the
// second part after the swap-out's completion event).  Page allocation hands
// out the first kind first, so the split is one slot index.
#include "mori_internal.h"

namespace mori {
namespace {

typedef unsigned int v4u __attribute__((ext_vector_type(4)));
// Pool, staging and host-mapped buffers are all reached by global (not flat)
// loads and stores, addressed as a uniform base plus a 32-bit byte offset.
typedef __attribute__((address_space(1))) v4u gv4u;
typedef __attribute__((address_space(1))) const uint8_t gcbyte;
typedef __attribute__((address_space(1))) uint8_t gbyte;

// The plan's tables (program lists, first slots, page lists, host addresses,
// the summary) are not written while a swap kernel runs, so they are read
// through the constant address space: wavefront-uniform reads of them become
// scalar loads, which wait on their own counter instead of behind the copy's
// outstanding vector loads and stores.
typedef __attribute__((address_space(4))) const uint32_t cu32;
typedef __attribute__((address_space(4))) const uint64_t cu64;
__device__ inline uint32_t ldc(const uint32_t* p, uint64_t i) { return ((cu32*)p)[i]; }
__device__ inline uint64_t ldc(const uint64_t* p, uint64_t i) { return ((cu64*)p)[i]; }
__device__ inline const __attribute__((address_space(4))) DevSummary* sumc(const SwapArgs& s) {
  return (const __attribute__((address_space(4))) DevSummary*)s.sum;
}

// Wavefront-uniform values moved to scalar registers.
__device__ inline uint32_t uniform32(uint32_t x) { return (uint32_t)__builtin_amdgcn_readfirstlane((int)x); }
__device__ inline uint64_t uniform64(uint64_t x) {
  return ((uint64_t)uniform32((uint32_t)(x >> 32)) << 32) | uniform32((uint32_t)x);
}

// Workgroups of 1024 threads, two per compute unit (64 registers at most).
constexpr uint32_t NT = 1024;
constexpr uint32_t LONG_VEC = 4;                 // vectors per thread per round for runs of 32 KiB and more
constexpr uint32_t MAX_RUNS_PER_PASS = NT / 64;  // groups stay whole wavefronts

// Largest a in [0, n) with base[a] <= x.
__device__ inline uint32_t find_slice(const uint32_t* base, uint32_t n, uint64_t x) {
  uint32_t lo = 0, hi = n;
  while (hi - lo > 1) {
    const uint32_t mid = (lo + hi) >> 1;
    if (ldc(base, mid) <= x) lo = mid;
    else hi = mid;
  }
  return lo;
}

__device__ inline v4u ld16(gcbyte* base, uint32_t i) {
  return __builtin_nontemporal_load((const gv4u*)(base + (i << 4)));
}
__device__ inline void st16(gbyte* base, uint32_t i, v4u v) { __builtin_nontemporal_store(v, (gv4u*)(base + (i << 4))); }

// Copies n16 vectors with a group of G threads; t is the thread's index in it.
// Each thread loads U vectors (all in flight at once), stores them, and waits
// until its stores have completed before the next round (the next run's
// loads included); a run longer than G * U vectors takes several rounds.
// Measured in the full-size pipelined rebalance on gfx950: the wait after the
// stores makes the gather 3-5% faster on 72 KiB and 16 KiB runs than letting
// the next round's loads overtake them.  Neither loads nor stores branch: an
// index past the run is clamped to the run's last vector, so a thread past the
// end reads that vector and writes the same bytes back to it (one address for
// the whole wavefront); masking those stores instead measured 1-3% slower on
// 32 and 72 KiB runs.
template <uint32_t G, uint32_t U>
__device__ inline void copy_run(const uint8_t* src_run, uint8_t* dst_run, uint32_t n16, uint32_t t) {
  gcbyte* src = (gcbyte*)uniform64((uint64_t)src_run);
  gbyte* dst = (gbyte*)uniform64((uint64_t)dst_run);
  const uint32_t last = n16 - 1;
  for (uint32_t c0 = 0; c0 < n16; c0 += G * U) {
    v4u v[U];
#pragma unroll
    for (uint32_t k = 0; k < U; ++k) v[k] = ld16(src, min(c0 + k * G + t, last));
#pragma unroll
    for (uint32_t k = 0; k < U; ++k) st16(dst, min(c0 + k * G + t, last), v[k]);
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  }
}

// Unit range of this launch; returns false when there is nothing to do.
template <bool kOut>
__device__ inline bool unit_range(const SwapArgs& s, uint32_t n, uint64_t* lo, uint64_t* hi) {
  const uint64_t LC = s.LC;
  const uint64_t total = (uint64_t)ldc(s.pg_base, n) * LC;
  const uint64_t nf = sumc(s)->pages_free_before + sumc(s)->pages_dropped;  // slots needing no wait
  *lo = 0;
  *hi = total;
  if (s.staging) {
    *lo = s.u_begin;
    *hi = s.u_end < total ? s.u_end : total;
  } else if (!kOut && s.part == 1) {
    uint32_t a = 0, b = n;  // number of moving programs whose first slot is below nf
    while (a < b) {
      const uint32_t mid = (a + b) >> 1;
      if (ldc(s.pg_base, mid) < nf) a = mid + 1;
      else b = mid;
    }
    *hi = (uint64_t)ldc(s.pg_base, a) * LC;
  } else if (!kOut && s.part == 2) {
    if (ldc(s.pg_base, n) <= nf) return false;  // no slot reaches a page that is free only later
    *lo = (uint64_t)ldc(s.pg_base, find_slice(s.pg_base, n, nf)) * LC;
  }
  return *lo < *hi;
}

// Decode state of one wavefront group: the moving program of the current unit.
// A group's units only increase, so the program index only moves forward.
struct Cursor {
  uint32_t a;        // program (index into the direction's list)
  uint64_t first;    // its first page index / slot
  uint64_t nb;       // its blocks
  uint64_t u_first;  // its first unit
  uint8_t* side;     // its host buffer (direct mode)
};

__device__ inline void cursor_set(const SwapArgs& s, Cursor& c, uint32_t a) {
  c.a = a;
  c.first = ldc(s.pg_base, a);
  c.nb = (uint64_t)ldc(s.pg_base, a + 1) - c.first;
  c.u_first = c.first * s.LC;
  c.side = s.staging ? nullptr : reinterpret_cast<uint8_t*>(ldc(s.addr, ldc(s.prog, a)));
}

// Source and destination of unit u (u >= the cursor's unit); false when the
// unit belongs to the other part of a two-part swap-in.
template <bool kOut>
__device__ inline bool unit_ends(const SwapArgs& s, Cursor& c, uint64_t u, uint64_t u_lo, uint64_t nf,
                                 const uint8_t** src, uint8_t** dst) {
  // u < the direction's total units, so the cursor stops at its last program
  while (u >= c.u_first + c.nb * s.LC) cursor_set(s, c, c.a + 1);
  const uint64_t rem = u - c.u_first;
  uint64_t q, i;
  if ((rem >> 32) == 0 && (c.nb >> 32) == 0) {  // the usual case: a 32-bit division
    q = (uint32_t)rem / (uint32_t)c.nb;
    i = (uint32_t)rem - (uint32_t)q * (uint32_t)c.nb;
  } else {
    q = rem / c.nb;
    i = rem - q * c.nb;
  }
  const uint64_t slot = c.first + i;
  if (!kOut && s.part != 0 && (s.part == 1) != (slot < nf)) return false;
  uint8_t* pool_run = s.pool + (q * s.NB + ldc(s.pages, slot)) * s.run;
  uint8_t* side = s.staging ? s.staging + (u - u_lo) * s.run : c.side + rem * s.run;
  *src = kOut ? pool_run : side;
  *dst = kOut ? side : pool_run;
  return true;
}

// PER runs per pass, U vectors per thread (copy_shape below, chosen on the
// host from the run size and the kind of memory on the other side).
template <bool kOut, uint32_t PER, uint32_t U>
__global__ __launch_bounds__(NT) __attribute__((amdgpu_waves_per_eu(8))) void swap_kernel(SwapArgs s) {
  // A swap-out stops on its own address errors only: the swap-in translates
  // concurrently on the other stream.  A swap-in also stops on the swap-out's
  // (ordered before it by the time it writes a page the swap-out reads): it
  // must not overwrite pages whose KV a failed swap-out did not save.
  if (sumc(s)->error || s.swap_err[0] || (!kOut && s.swap_err[1])) return;
  const uint32_t n = kOut ? sumc(s)->n_out : sumc(s)->n_in;
  uint64_t lo, hi;
  if (n == 0 || !unit_range<kOut>(s, n, &lo, &hi)) return;
  const uint32_t n16 = (uint32_t)(s.run / 16);
  constexpr uint32_t G = NT / PER;  // threads per run, whole wavefronts
  // groups are whole wavefronts, so the group index is wavefront-uniform
  const uint32_t grp = uniform32(threadIdx.x / G), t = threadIdx.x % G;
  const uint64_t stride = (uint64_t)gridDim.x * PER;
  uint64_t u = lo + (uint64_t)blockIdx.x * PER + grp;
  if (u >= hi) return;  // the group's whole wavefronts leave together
  const uint64_t nf = sumc(s)->pages_free_before + sumc(s)->pages_dropped;
  Cursor c;
  cursor_set(s, c, find_slice(s.pg_base, n, u / s.LC));
  const uint8_t* src;
  uint8_t* dst;
  bool ok = unit_ends<kOut>(s, c, u, lo, nf, &src, &dst);
  for (;;) {
    // decode the next unit first: its loads overlap this unit's copy
    const uint64_t un = u + stride;
    const uint8_t* nsrc = nullptr;
    uint8_t* ndst = nullptr;
    const bool more = un < hi;
    const bool nok = more && unit_ends<kOut>(s, c, un, lo, nf, &nsrc, &ndst);
    if (ok) copy_run<G, U>(src, dst, n16, t);
    if (!more) break;
    u = un;
    src = nsrc;
    dst = ndst;
    ok = nok;
  }
}

struct CopyShape {
  uint32_t per, vec;
};

// Between HBM buffers, runs of 2048 vectors (32 KiB) and more: one per
// workgroup, LONG_VEC vectors per thread per round (a 72 KiB run takes a
// round of 64 KiB and one of 8 KiB; a 32 KiB run one round, half of it
// clamped); from 1024 vectors: one per workgroup, one vector per thread per
// round.  Over the host link (kernel-direct mode), runs of 1024 vectors and
// more: two per workgroup, one vector per thread per round.  Shorter runs: as
// many per workgroup (a power of two, at most one per wavefront) as give each
// thread one vector.  Measured in the full-size pipelined rebalance: between
// HBM buffers four vectors per thread beat one to three, five and eight on
// runs of 32 and 72 KiB (one is best on 16 KiB runs); over the host link four
// or two vectors per thread lose 12% or 7% against one (fewer accesses in
// flight suit the link's two directions), and two runs per workgroup gain 1%.
CopyShape copy_shape(uint64_t run, bool host_link) {
  const uint64_t n16 = run / 16;
  if (host_link && n16 >= NT) return {2, 1};
  if (n16 >= 2 * NT) return {1, LONG_VEC};
  uint32_t per = 1;
  while (per < MAX_RUNS_PER_PASS && 2ull * per * n16 <= (uint64_t)NT) per *= 2;
  return {per, 1};
}

template <bool kOut, uint32_t PER, uint32_t U>
void launch_shape(const SwapArgs& a, uint32_t grid, hipStream_t s) {
  hipLaunchKernelGGL((swap_kernel<kOut, PER, U>), dim3(grid), dim3(NT), 0, s, a);
}

template <bool kOut>
hipError_t launch_swap(const SwapArgs& a, uint32_t grid, hipStream_t s) {
  const CopyShape sh = copy_shape(a.run, a.host_link != 0);
  switch (sh.per) {
    case 1:
      if (sh.vec == LONG_VEC) launch_shape<kOut, 1, LONG_VEC>(a, grid, s);
      else launch_shape<kOut, 1, 1>(a, grid, s);
      break;
    case 2: launch_shape<kOut, 2, 1>(a, grid, s); break;
    case 4: launch_shape<kOut, 4, 1>(a, grid, s); break;
    case 8: launch_shape<kOut, 8, 1>(a, grid, s); break;
    default: launch_shape<kOut, 16, 1>(a, grid, s); break;
  }
  return hipGetLastError();
}

}  // namespace

hipError_t launch_swap_out(const SwapArgs& a, uint32_t grid, hipStream_t s) { return launch_swap<true>(a, grid, s); }

hipError_t launch_swap_in(const SwapArgs& a, uint32_t grid, hipStream_t s) { return launch_swap<false>(a, grid, s); }

}  // namespace mori
