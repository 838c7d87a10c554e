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
// worth caching); the index arithmetic is wavefront-uniform.  A persistent grid
// walks the units with a grid stride.  Runs shorter than a workgroup's pass
// (1024 threads x two vectors = 32 KiB) are copied several at a time: the
// workgroup splits into wave-aligned groups of threads, one run each, so every
// thread still has two vectors in flight.
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

// Shape measured on gfx950 in the full-size rebalance (32 KiB and 72 KiB
// runs): 1024-thread workgroups moving one run at a time with two 16-byte
// vectors per thread in flight (one 32 KiB run per pass), grid-stride over
// runs.  Against 256 x 8 this is 5% faster for the gather and 8% for the
// scatter; 512 x 4 lies between, 1024 x 1 and 1024 x 3 match 1024 x 2.  Big
// workgroups pay off only because the decode is cheap and overlapped: each
// workgroup walks its programs forward with a cursor instead of searching
// the program list per run, and decodes the next run before copying the
// current one, so the dependent page-table load is in flight meanwhile.
constexpr int NT = 1024;
constexpr int UNR = 2;

// Largest a in [0, n) with base[a] <= x.
__device__ inline uint32_t find_slice(const uint32_t* base, uint32_t n, uint64_t x) {
  uint32_t lo = 0, hi = n;
  while (hi - lo > 1) {
    const uint32_t mid = (lo + hi) >> 1;
    if (base[mid] <= x) lo = mid;
    else hi = mid;
  }
  return lo;
}

constexpr uint32_t MAX_RUNS_PER_PASS = NT / 64;  // groups stay whole wavefronts

// Copies n16 vectors with a group of G threads; t is the thread's index in it.
template <uint32_t G>
__device__ inline void copy_run(const v4u* __restrict__ src, v4u* __restrict__ dst, uint32_t n16, uint32_t t) {
  for (uint32_t t0 = 0; t0 < n16; t0 += G * UNR) {
    v4u v[UNR];
#pragma unroll
    for (int k = 0; k < UNR; ++k) {
      const uint32_t i = t0 + k * G + t;
      if (i < n16) v[k] = __builtin_nontemporal_load(src + i);
    }
#pragma unroll
    for (int k = 0; k < UNR; ++k) {
      const uint32_t i = t0 + k * G + t;
      if (i < n16) __builtin_nontemporal_store(v[k], dst + i);
    }
  }
}

// Unit range of this launch; returns false when there is nothing to do.
template <bool kOut>
__device__ inline bool unit_range(const SwapArgs& s, uint32_t n, uint64_t* lo, uint64_t* hi) {
  const uint64_t LC = s.LC;
  const uint64_t total = (uint64_t)s.pg_base[n] * LC;
  const uint64_t nf = s.sum->pages_free_before + s.sum->pages_dropped;  // slots needing no wait
  *lo = 0;
  *hi = total;
  if (s.staging) {
    *lo = s.u_begin;
    *hi = s.u_end < total ? s.u_end : total;
  } else if (!kOut && s.part == 1) {
    uint32_t a = 0, b = n;  // number of moving programs whose first slot is below nf
    while (a < b) {
      const uint32_t mid = (a + b) >> 1;
      if (s.pg_base[mid] < nf) a = mid + 1;
      else b = mid;
    }
    *hi = (uint64_t)s.pg_base[a] * LC;
  } else if (!kOut && s.part == 2) {
    if (s.pg_base[n] <= nf) return false;  // no slot reaches a page that is free only later
    *lo = (uint64_t)s.pg_base[find_slice(s.pg_base, n, nf)] * LC;
  }
  return *lo < *hi;
}

// Decode state of one workgroup: the moving program of the current unit.  A
// workgroup's units only increase, so the program index only moves forward.
struct Cursor {
  uint32_t a;        // program (index into the direction's list)
  uint64_t first;    // its first page index / slot
  uint64_t nb;       // its blocks
  uint64_t u_first;  // its first unit
  uint8_t* side;     // its host buffer (direct mode)
};

__device__ inline void cursor_set(const SwapArgs& s, Cursor& c, uint32_t a) {
  c.a = a;
  c.first = s.pg_base[a];
  c.nb = (uint64_t)s.pg_base[a + 1] - c.first;
  c.u_first = c.first * s.LC;
  c.side = s.staging ? nullptr : reinterpret_cast<uint8_t*>(s.addr[s.prog[a]]);
}

// Source and destination of unit u (u >= the cursor's unit); false when the
// unit belongs to the other part of a two-part swap-in.
template <bool kOut>
__device__ inline bool unit_ends(const SwapArgs& s, Cursor& c, uint64_t u, uint64_t u_lo, uint64_t nf, const v4u** src,
                                 v4u** dst) {
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
  uint8_t* pool_run = s.pool + (q * s.NB + s.pages[slot]) * s.run;
  uint8_t* side = s.staging ? s.staging + (u - u_lo) * s.run : c.side + rem * s.run;
  *src = reinterpret_cast<const v4u*>(kOut ? pool_run : side);
  *dst = reinterpret_cast<v4u*>(kOut ? side : pool_run);
  return true;
}

// PER runs per pass (runs_per_pass below, chosen on the host from the run size)
template <bool kOut, uint32_t PER>
__global__ __launch_bounds__(NT) void swap_kernel(SwapArgs s) {
  // A swap-out stops on its own address errors only: the swap-in translates
  // concurrently on the other stream.  A swap-in also stops on the swap-out's
  // (ordered before it by the time it writes a page the swap-out reads): it
  // must not overwrite pages whose KV a failed swap-out did not save.
  if (s.sum->error || s.swap_err[0] || (!kOut && s.swap_err[1])) return;
  const uint32_t n = kOut ? s.sum->n_out : s.sum->n_in;
  uint64_t lo, hi;
  if (n == 0 || !unit_range<kOut>(s, n, &lo, &hi)) return;
  const uint32_t n16 = (uint32_t)(s.run / 16);
  constexpr uint32_t G = NT / PER;  // threads per run, whole wavefronts
  const uint32_t grp = threadIdx.x / G, t = threadIdx.x % G;
  const uint64_t stride = (uint64_t)gridDim.x * PER;
  uint64_t u = lo + (uint64_t)blockIdx.x * PER + grp;
  if (u >= hi) return;  // the group's whole wavefronts leave together
  const uint64_t nf = s.sum->pages_free_before + s.sum->pages_dropped;
  Cursor c;
  cursor_set(s, c, find_slice(s.pg_base, n, u / s.LC));
  const v4u* src;
  v4u* dst;
  bool ok = unit_ends<kOut>(s, c, u, lo, nf, &src, &dst);
  for (;;) {
    // decode the next unit first: its loads overlap this unit's copy
    const uint64_t un = u + stride;
    const v4u* nsrc = nullptr;
    v4u* ndst = nullptr;
    const bool more = un < hi;
    const bool nok = more && unit_ends<kOut>(s, c, un, lo, nf, &nsrc, &ndst);
    if (ok) copy_run<G>(src, dst, n16, t);
    if (!more) break;
    u = un;
    src = nsrc;
    dst = ndst;
    ok = nok;
  }
}

// Runs per pass: the most (a power of two, at most one per wavefront) whose
// vectors still fill two per thread of the workgroup.
uint32_t runs_per_pass(uint64_t run) {
  const uint64_t n16 = run / 16;
  uint32_t per = 1;
  while (per < MAX_RUNS_PER_PASS && 2ull * per * n16 <= (uint64_t)(NT * UNR)) per *= 2;
  return per;
}

template <bool kOut>
hipError_t launch_swap(const SwapArgs& a, uint32_t grid, hipStream_t s) {
  switch (runs_per_pass(a.run)) {
    case 1: hipLaunchKernelGGL((swap_kernel<kOut, 1>), dim3(grid), dim3(NT), 0, s, a); break;
    case 2: hipLaunchKernelGGL((swap_kernel<kOut, 2>), dim3(grid), dim3(NT), 0, s, a); break;
    case 4: hipLaunchKernelGGL((swap_kernel<kOut, 4>), dim3(grid), dim3(NT), 0, s, a); break;
    case 8: hipLaunchKernelGGL((swap_kernel<kOut, 8>), dim3(grid), dim3(NT), 0, s, a); break;
    default: hipLaunchKernelGGL((swap_kernel<kOut, 16>), dim3(grid), dim3(NT), 0, s, a); break;
  }
  return hipGetLastError();
}

}  // namespace

hipError_t launch_swap_out(const SwapArgs& a, uint32_t grid, hipStream_t s) { return launch_swap<true>(a, grid, s); }

hipError_t launch_swap_in(const SwapArgs& a, uint32_t grid, hipStream_t s) { return launch_swap<false>(a, grid, s); }

}  // namespace mori
