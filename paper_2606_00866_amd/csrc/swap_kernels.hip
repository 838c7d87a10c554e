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
// worth caching); the index arithmetic is wavefront-uniform and stays in
// scalar registers.  A persistent grid walks the units with a grid stride.
//
//   swap_out : pool page  -> host buffer (direct) or staging (copy engine)
//   swap_in  : host buffer (direct) or staging -> newly allocated pool page
//
// Swap-in is launched in two parts in direct mode: slots taken from pages
// that were free before the step, which no swap-out reads, and slots taken
// from pages released this step, which must wait for the swap-out (the host
// orders the second part after the swap-out's completion event).
#include "mori_internal.h"

namespace mori {
namespace {

typedef unsigned int v4u __attribute__((ext_vector_type(4)));

constexpr int NT = 256;  // threads per workgroup
constexpr int UNR = 8;   // 16-byte vectors in flight per thread per iteration

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

__device__ inline void copy_run(const v4u* __restrict__ src, v4u* __restrict__ dst, uint32_t n16) {
  for (uint32_t t0 = 0; t0 < n16; t0 += NT * UNR) {
    v4u v[UNR];
#pragma unroll
    for (int u = 0; u < UNR; ++u) {
      const uint32_t t = t0 + u * NT + threadIdx.x;
      if (t < n16) v[u] = __builtin_nontemporal_load(src + t);
    }
#pragma unroll
    for (int u = 0; u < UNR; ++u) {
      const uint32_t t = t0 + u * NT + threadIdx.x;
      if (t < n16) __builtin_nontemporal_store(v[u], dst + t);
    }
  }
}

template <bool kOut>
__global__ __launch_bounds__(NT) void swap_kernel(SwapArgs s) {
  if (s.sum->error || *s.swap_err) return;
  const uint32_t n = kOut ? s.sum->n_out : s.sum->n_in;
  if (n == 0) return;
  const uint64_t LC = s.LC;
  const uint64_t total = (uint64_t)s.pg_base[n] * LC;
  const uint64_t nf = s.sum->pages_free_before;
  uint64_t u_lo = 0, u_hi = total;
  if (s.staging) {
    u_lo = s.u_begin;
    u_hi = s.u_end < total ? s.u_end : total;
  } else if (!kOut && s.part == 1) {
    // programs whose first slot is below nf
    uint32_t a1 = 0;
    uint32_t lo = 0, hi = n;  // count of a with pg_base[a] < nf (pg_base is non-decreasing)
    while (lo < hi) {
      const uint32_t mid = (lo + hi) >> 1;
      if (s.pg_base[mid] < nf) lo = mid + 1;
      else hi = mid;
    }
    a1 = lo;
    u_hi = (uint64_t)s.pg_base[a1] * LC;
  } else if (!kOut && s.part == 2) {
    if (s.pg_base[n] <= nf) return;  // no slot reaches a released page
    u_lo = (uint64_t)s.pg_base[find_slice(s.pg_base, n, nf)] * LC;
  }
  const uint32_t n16 = (uint32_t)(s.run / 16);
  for (uint64_t u = u_lo + blockIdx.x; u < u_hi; u += gridDim.x) {
    const uint32_t a = find_slice(s.pg_base, n, u / LC);
    const uint64_t first = s.pg_base[a];
    const uint64_t nb = (uint64_t)s.pg_base[a + 1] - first;
    const uint64_t rem = u - first * LC;
    const uint64_t q = rem / nb, i = rem - q * nb;
    const uint64_t slot = first + i;
    if (!kOut && s.part == 1 && slot >= nf) continue;
    if (!kOut && s.part == 2 && slot < nf) continue;
    const uint64_t page = s.pages[slot];
    uint8_t* pool_run = s.pool + (q * s.NB + page) * s.run;
    uint8_t* side = s.staging ? s.staging + (u - u_lo) * s.run
                              : reinterpret_cast<uint8_t*>(s.addr[s.prog[a]]) + rem * s.run;
    if (kOut) copy_run(reinterpret_cast<const v4u*>(pool_run), reinterpret_cast<v4u*>(side), n16);
    else copy_run(reinterpret_cast<const v4u*>(side), reinterpret_cast<v4u*>(pool_run), n16);
  }
}

}  // namespace

hipError_t launch_swap_out(const SwapArgs& a, uint32_t grid, hipStream_t s) {
  hipLaunchKernelGGL(swap_kernel<true>, dim3(grid), dim3(NT), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_swap_in(const SwapArgs& a, uint32_t grid, hipStream_t s) {
  hipLaunchKernelGGL(swap_kernel<false>, dim3(grid), dim3(NT), 0, s, a);
  return hipGetLastError();
}

}  // namespace mori
