// Page side of one rebalance (sticky placement of Sec. 4.3 over the paged KV
// pool of Sec. 2.1), after the rank / boundary kernel (whose other workgroups
// set the page state from the caller's free map):
//
//   claim    walk every block-table entry: validate ownership (no page owned
//            twice, none both owned and free, none out of range, no page held
//            by a CPU/Waiting program), mark pages of programs leaving the
//            GPU as released, record the old page of every swap-out block;
//   count    per 512-page tile: pages free before the step, released pages
//            free at once (programs dropped to Waiting that are idle) and
//            released pages free only later (programs swapped out, and
//            programs dropped while they may still run an inference step:
//            Sec. 4.3.1 demotes a Reasoning victim lazily, so its step goes
//            on reading and appending to its pages); a page that is neither
//            free nor owned is a leak;
//   scan     exclusive prefix over tiles, totals, capacity; the summary is
//            final here and is stored into the host mirror.  Up to
//            SCAN_IN_ASSIGN tiles every assign workgroup does this itself
//            from the tile counts (one launch fewer); above, one workgroup
//            of a kernel of its own;
//   assign   slot j of the incoming programs takes the j-th page of
//            (free-before ++ free at once ++ free later, each ascending):
//            pages nothing uses come before pages still in use, so the
//            swap-in waits for the swap-out stream only for slots past the
//            first two groups; the free map after the step is what is left
//            of that sequence;
//   commit   rewrite the block tables (released -> no page, incoming -> their
//            slots' pages) and the tier vector.
//
// Validation happens in claim/count/scan; assign and commit write caller
// memory only when the plan's error word is still zero, so a rejected plan
// leaves the caller's state untouched.  All loops are grid-stride over sizes
// the host knows (tbl_len, num_blocks), bounded by device values read once.
#include "mori_internal.h"
#include "wave.h"

namespace mori {
namespace {

constexpr int WG = 256;
constexpr uint32_t SCAN_IN_ASSIGN = 1024;  // tiles (2^19 pages): each assign workgroup reads 16 B per tile

// Largest p in [0, P) with off[p] <= e (so off[p] <= e < off[p+1] when e < off[P]).
__device__ inline uint32_t find_program(const uint32_t* off, uint32_t P, uint32_t e) {
  uint32_t lo = 0, hi = P;  // invariant: off[lo] <= e, answer in [lo, hi)
  while (hi - lo > 1) {
    const uint32_t mid = (lo + hi) >> 1;
    if (off[mid] <= e) lo = mid;
    else hi = mid;
  }
  return lo;
}

__global__ __launch_bounds__(WG) void pages_claim_kernel(PlanArgs a) {
  if (a.sum->error) return;
  const uint32_t used = a.tbl_off[a.P];
  uint32_t err = 0;
  for (uint64_t e64 = (uint64_t)blockIdx.x * WG + threadIdx.x; e64 < used; e64 += (uint64_t)gridDim.x * WG) {
    const uint32_t e = (uint32_t)e64;  // 64-bit stride: no wrap near 2^32 entries
    const uint32_t p = find_program(a.tbl_off, a.P, e);
    const uint32_t pg = a.tbl[e];
    if (a.tier_old[p] != MORI_TIER_GPU) {
      if (pg != MORI_NO_PAGE) err |= MORI_DEV_NONRES_PAGE;
      continue;
    }
    if (pg >= a.NB) {
      err |= MORI_DEV_PAGE_RANGE;
      continue;
    }
    const uint8_t c = a.cat[p];
    // a program dropped while it may still run (with statuses: anything but
    // Acting) frees its pages only after its step, which the caller orders
    // before the swap-out on the swap-out stream
    const bool running = c == MORI_CAT_DROP_GPU && (a.flags & (MORI_F_STATUS_KEY | MORI_F_INCREMENTAL)) &&
                         a.status[p] != MORI_ST_ACTING;
    const uint32_t leaves =
        c == MORI_CAT_OUT || running ? (PS_REL | PS_LATER) : c == MORI_CAT_DROP_GPU ? PS_REL : 0u;
    const uint32_t old = atomicOr(&a.pstate[pg], PS_OWNED | leaves);
    if (old & (PS_FREE | PS_OWNED)) err |= MORI_DEV_PAGE_DUP;
    if (c == MORI_CAT_OUT) {
      const uint32_t k = a.base[p] + (e - a.tbl_off[p]);
      if (k < a.NB) a.out_src[k] = pg;  // more owned blocks than pages implies a duplicate
      else err |= MORI_DEV_PAGE_DUP;
    }
  }
  if (err) atomicOr(&a.sum->error, err);
}

__global__ __launch_bounds__(WG) void pages_count_kernel(PlanArgs a) {
  __shared__ uint32_t s_free, s_drop, s_copy, s_err;
  if (a.sum->error) return;
  if (threadIdx.x == 0) s_free = s_drop = s_copy = s_err = 0;
  __syncthreads();
  const uint32_t per = PAGE_TILE / WG;
  const uint64_t start = (uint64_t)blockIdx.x * PAGE_TILE + (uint64_t)threadIdx.x * per;
  uint32_t nf = 0, nd = 0, nc = 0, err = 0;
  for (uint32_t j = 0; j < per; ++j) {
    const uint64_t pg = start + j;
    if (pg >= a.NB) break;
    const uint32_t st = a.pstate[pg];
    if (st == PS_FREE) ++nf;
    else if (st & PS_LATER) ++nc;
    else if (st & PS_REL) ++nd;
    else if (st == 0) err |= MORI_DEV_PAGE_LEAK;
  }
  const uint32_t wf = wave::sum(nf), wd = wave::sum(nd), wc = wave::sum(nc);  // one LDS atomic per wavefront
  if ((threadIdx.x & 63) == 0) {
    if (wf) atomicAdd(&s_free, wf);
    if (wd) atomicAdd(&s_drop, wd);
    if (wc) atomicAdd(&s_copy, wc);
  }
  if (err) atomicOr(&s_err, err);
  __syncthreads();
  if (threadIdx.x == 0) {
    a.tile_cnt[blockIdx.x] = (uint64_t)s_free | ((uint64_t)s_drop << 32);
    a.tile_cnt[a.ntiles + blockIdx.x] = s_copy;
    if (s_err) atomicOr(&a.sum->error, s_err);
  }
}

// Workgroup-wide exclusive scan of one u64 per thread (WGS threads).
template <int WGS>
__device__ uint64_t wg_scan_excl(uint64_t v, uint64_t* s_wave, uint64_t* total) {
  constexpr int NWV = WGS / 64;
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
  const uint64_t x = wave::incl_add(v);
  if (lane == 63) s_wave[wid] = x;
  __syncthreads();
  if (wid == 0) {
    const uint64_t w = lane < NWV ? s_wave[lane] : 0ull;
    const uint64_t wi = wave::incl_add(w);
    if (lane < NWV) s_wave[lane] = wi - w;
    if (lane == NWV - 1) s_wave[NWV] = wi;
  }
  __syncthreads();
  const uint64_t res = s_wave[wid] + x - v;
  *total = s_wave[NWV];
  __syncthreads();
  return res;
}

// The page totals into the summary, the capacity check, and the summary into
// the host mirror (final from here).  One thread.
__device__ void finish_summary(const PlanArgs& a, uint64_t nf, uint64_t nd, uint64_t nc) {
  DevSummary* s = a.sum;
  s->pages_free_before = nf;
  s->pages_released = nd + nc;
  s->pages_dropped = nd;
  if (s->need > nf + nd + nc) {
    atomicOr(&s->error, MORI_DEV_NOSPC);
  } else {
    s->pages_recycled = s->need > nf ? s->need - nf : 0;
    s->pages_free_after = nf + nd + nc - s->need;
  }
  *host_mirror(a, s) = *s;
}

__global__ __launch_bounds__(1024) void pages_scan_kernel(PlanArgs a) {
  __shared__ uint64_t s_wave[1024 / 64 + 1];
  if (a.sum->error) {
    if (threadIdx.x == 0) *host_mirror(a, a.sum) = *a.sum;
    return;
  }
  uint64_t carry[2] = {0, 0};
  for (int half = 0; half < 2; ++half) {  // (free-before | dropped << 32), then free later
    const uint64_t* cnt = a.tile_cnt + (uint64_t)half * a.ntiles;
    uint64_t* out = a.tile_base + (uint64_t)half * a.ntiles;
    for (uint32_t t0 = 0; t0 < a.ntiles; t0 += 1024) {
      const uint32_t t = t0 + threadIdx.x;
      const uint64_t v = t < a.ntiles ? cnt[t] : 0ull;
      uint64_t tot;
      const uint64_t ex = wg_scan_excl<1024>(v, s_wave, &tot);
      if (t < a.ntiles) out[t] = carry[half] + ex;
      carry[half] += tot;
    }
  }
  if (threadIdx.x == 0) finish_summary(a, carry[0] & 0xFFFFFFFFull, carry[0] >> 32, carry[1]);
}

// SCAN: the tile scan is done here (every workgroup scans the counts of the
// tiles before its own and totals all of them; workgroup 0 finishes the
// summary), else it comes from pages_scan_kernel.
template <bool SCAN>
__global__ __launch_bounds__(WG) void pages_assign_kernel(PlanArgs a) {
  __shared__ uint64_t s_wave[WG / 64 + 1];
  __shared__ uint64_t s_red[WG / 64][4];
  if (a.sum->error) {
    if (SCAN && blockIdx.x == 0 && threadIdx.x == 0) *host_mirror(a, a.sum) = *a.sum;
    return;
  }
  const uint64_t need = a.sum->need;
  uint64_t tb, tbc, nf_all, nd_all;
  if constexpr (SCAN) {
    uint64_t v[4] = {0, 0, 0, 0};  // prefix (free | dropped << 32), prefix free-later, and the totals
    for (uint32_t t = threadIdx.x; t < a.ntiles; t += WG) {
      const uint64_t c0 = a.tile_cnt[t], c1 = a.tile_cnt[a.ntiles + t];
      if (t < blockIdx.x) v[0] += c0, v[1] += c1;
      v[2] += c0;
      v[3] += c1;
    }
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const uint64_t w = wave::sum(v[k]);
      if ((threadIdx.x & 63) == 0) s_red[threadIdx.x >> 6][k] = w;
    }
    __syncthreads();
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      v[k] = 0;
#pragma unroll
      for (int w = 0; w < WG / 64; ++w) v[k] += s_red[w][k];
    }
    tb = v[0];
    tbc = v[1];
    nf_all = v[2] & 0xFFFFFFFFull;
    nd_all = v[2] >> 32;
    if (blockIdx.x == 0 && threadIdx.x == 0) finish_summary(a, nf_all, nd_all, v[3]);
    if (need > nf_all + nd_all + v[3]) return;  // no room: workgroup 0 sets the error
  } else {
    tb = a.tile_base[blockIdx.x];
    tbc = a.tile_base[a.ntiles + blockIdx.x];
    nf_all = a.sum->pages_free_before;
    nd_all = a.sum->pages_dropped;
  }
  const uint32_t per = PAGE_TILE / WG;
  const uint64_t start = (uint64_t)blockIdx.x * PAGE_TILE + (uint64_t)threadIdx.x * per;
  uint32_t st[PAGE_TILE / WG];
  uint32_t nf = 0, nd = 0, nc = 0;
#pragma unroll
  for (uint32_t j = 0; j < per; ++j) {
    const uint64_t pg = start + j;
    st[j] = pg < a.NB ? a.pstate[pg] : PS_OWNED;
    if (st[j] == PS_FREE) ++nf;
    else if (st[j] & PS_LATER) ++nc;
    else if (st[j] & PS_REL) ++nd;
  }
  uint64_t tot;
  const uint64_t ex = wg_scan_excl<WG>((uint64_t)nf | ((uint64_t)nd << 32), s_wave, &tot);
  const uint64_t exc = wg_scan_excl<WG>(nc, s_wave, &tot);
  uint64_t fi = (tb & 0xFFFFFFFFull) + (ex & 0xFFFFFFFFull);
  uint64_t di = (tb >> 32) + (ex >> 32);
  uint64_t ci = tbc + exc;
#pragma unroll
  for (uint32_t j = 0; j < per; ++j) {
    const uint64_t pg = start + j;
    uint64_t slot;
    if (st[j] == PS_FREE) slot = fi++;
    else if (st[j] & PS_LATER) slot = nf_all + nd_all + ci++;
    else if (st[j] & PS_REL) slot = nf_all + di++;
    else continue;
    if (slot < need) {
      a.in_dst[slot] = (uint32_t)pg;
      a.free_map[pg] = 0;
    } else {
      a.free_map[pg] = 1;
    }
  }
}

__global__ __launch_bounds__(WG) void commit_kernel(PlanArgs a) {
  if (a.sum->error) return;
  const uint32_t used = a.tbl_off[a.P];
  for (uint64_t e64 = (uint64_t)blockIdx.x * WG + threadIdx.x; e64 < used; e64 += (uint64_t)gridDim.x * WG) {
    const uint32_t e = (uint32_t)e64;  // 64-bit stride: no wrap near 2^32 entries
    const uint32_t p = find_program(a.tbl_off, a.P, e);
    const uint8_t c = a.cat[p];
    if (c == MORI_CAT_OUT || c == MORI_CAT_DROP_GPU) a.tbl[e] = MORI_NO_PAGE;
    else if (c == MORI_CAT_IN || c == MORI_CAT_ADMIT_GPU) a.tbl[e] = a.in_dst[a.base[p] + (e - a.tbl_off[p])];
  }
  for (uint32_t p = blockIdx.x * WG + threadIdx.x; p < a.P; p += gridDim.x * WG) a.tier[p] = a.tier_new[p];
}

// Resolves every moving program's caller address through the registered
// ranges; a buffer that is not 16-B aligned or not wholly inside one range
// sets MORI_DEV_HOST_ADDR and the swap kernels then do nothing.
__global__ __launch_bounds__(WG) void translate_kernel(TranslateArgs t) {
  if (t.sum->error) return;
  const uint32_t n = t.dir_in ? t.sum->n_in : t.sum->n_out;
  uint32_t err = 0;
  for (uint32_t j = blockIdx.x * WG + threadIdx.x; j < n; j += gridDim.x * WG) {
    const uint32_t p = t.prog[j];
    const uint64_t bytes = (uint64_t)(t.tbl_off[p + 1] - t.tbl_off[p]) * t.block_bytes;
    const uint64_t h = t.addr_in[p];
    uint64_t dev = 0;
    bool ok = (h & 15ull) == 0 && h != 0;
    if (bytes == 0) ok = true;  // nothing to copy: any address will do
    else if (ok) {
      ok = false;
      for (uint32_t r = 0; r < t.nranges; ++r) {
        const DevRange rg = t.ranges[r];
        if (h >= rg.host_base && h - rg.host_base <= rg.bytes && bytes <= rg.bytes - (h - rg.host_base)) {
          dev = rg.dev_base + (h - rg.host_base);
          ok = true;
          break;
        }
      }
    }
    if (!ok) err |= MORI_DEV_HOST_ADDR;
    t.addr_out[p] = dev;
  }
  if (err) atomicOr(&t.swap_err[t.dir_in], err);
}

inline uint32_t grid_for(uint64_t n, uint32_t cap) {
  uint64_t g = (n + WG - 1) / WG;
  if (g < 1) g = 1;
  return (uint32_t)(g < cap ? g : cap);
}

}  // namespace

hipError_t launch_pages(const PlanArgs& a, hipStream_t s) {
  const uint32_t ge = grid_for(a.tbl_len > a.P ? a.tbl_len : a.P, 2048);
  hipLaunchKernelGGL(pages_claim_kernel, dim3(ge), dim3(WG), 0, s, a);
  hipLaunchKernelGGL(pages_count_kernel, dim3(a.ntiles), dim3(WG), 0, s, a);  // ntiles >= 1: the pool has a page
  if (a.ntiles <= SCAN_IN_ASSIGN) {
    hipLaunchKernelGGL(pages_assign_kernel<true>, dim3(a.ntiles), dim3(WG), 0, s, a);
  } else {
    hipLaunchKernelGGL(pages_scan_kernel, dim3(1), dim3(1024), 0, s, a);
    hipLaunchKernelGGL(pages_assign_kernel<false>, dim3(a.ntiles), dim3(WG), 0, s, a);
  }
  hipLaunchKernelGGL(commit_kernel, dim3(ge), dim3(WG), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_translate(const TranslateArgs& t, hipStream_t s) {
  hipLaunchKernelGGL(translate_kernel, dim3(16), dim3(WG), 0, s, t);
  return hipGetLastError();
}

}  // namespace mori
