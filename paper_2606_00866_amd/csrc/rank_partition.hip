// Rank / boundary step of one rebalance, in a single workgroup.
//
//   1. idleness of every program by Eq. 1 (Sec. 4.2), binary32, totals
//      accumulated oldest cycle first from +0, correctly rounded division;
//   2. a 64-bit key per program and a stable sort of (key, id): direct rank
//      counting for up to 256 programs, else an LSD radix sort with wave64
//      ballots.  Boundary policy: the key is the idleness bits,
//      optionally with the Acting bit of the demotion order of Sec. 4.3.1 --
//      the relative ranking, busiest first.  Incremental policy (Sec. 4.3.1):
//      the key is the program's listing group (old tier; Waiting split into
//      returning, new and Acting) above its priority in that group, so each
//      tier group lists its programs in reverse demotion order and the
//      promotion candidates come in promotion order;
//   3. an inclusive u64 scan of KV bytes in that order, then either the two
//      capacity boundaries (Sec. 4.1 per-tier capacity, Sec. 7.2 fill from the
//      busiest end) or the greedy skip-fit walk, or the incremental policy:
//      demote-until-fits is the tail of a tier group past its longest fitting
//      prefix, promote-while-fits a prefix of the candidates' byte scan;
//      victims that do not all fit the CPU room and skip-fit promotion are
//      walked one by one by one thread;
//   4. the sticky diff (Sec. 4.3): per-program transition category, the
//      swap-out and swap-in lists in that order and the page/slot bases.
//
// P <= 4096 programs fit in LDS (4 keys per thread), so the whole step is one
// launch: microseconds for tens of programs, about thirty for 4096, bound by
// the one workgroup's vector ALU and barriers; nothing here is bandwidth-bound.
#include "mori_internal.h"
#include "wave.h"

namespace mori {
namespace {

// Four shapes, chosen by P at launch: one wave (64 threads, so every barrier
// is a single wave's) for P <= 64, 256 threads x 1 item up to 256 (ranks
// counted directly in both), 1024 x 1 up to 1024 and
// 1024 threads x 4 items (striped: item x = it * RT + tid) up to 4096; fewer
// item slices mean fewer ballots per radix pass.
constexpr int RADIX_BITS = 8;
constexpr int RADIX = 1 << RADIX_BITS;
constexpr int KEY_BITS = 64;
constexpr int GROUP_SHIFT = 61;  // incremental keys: listing group in the top three bits
// Exclusive scans of the IPT x RT items in rank order (item it of thread tid
// has rank it * RT + tid), N values per item side by side: wave scans, the
// per-(slice, wave) totals scanned by the first wave, and three barriers in
// all, however many slices.  s_tot needs (IPT * NW + 1) * N entries; total[n]
// receives the sum of value n over all items.
template <int NW, int IPT, int N>
__device__ void scan_slices(const uint64_t (&v)[IPT][N], uint64_t (&ex)[IPT][N], uint64_t* s_tot,
                            uint64_t (&total)[N]) {
  constexpr int NS = IPT * NW;
  static_assert(NS <= 64, "one lane per (slice, wave) total");
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
  uint64_t inc[IPT][N];
#pragma unroll
  for (int it = 0; it < IPT; ++it)
#pragma unroll
    for (int n = 0; n < N; ++n) {
      const uint64_t x = wave::incl_add(v[it][n]);
      inc[it][n] = x;
      if (lane == 63) s_tot[(it * NW + wid) * N + n] = x;
    }
  __syncthreads();
  if (wid == 0) {
#pragma unroll
    for (int n = 0; n < N; ++n) {
      const uint64_t w = lane < NS ? s_tot[lane * N + n] : 0ull;
      const uint64_t wi = wave::incl_add(w);
      if (lane < NS) s_tot[lane * N + n] = wi - w;
      if (lane == NS - 1) s_tot[NS * N + n] = wi;
    }
  }
  __syncthreads();
#pragma unroll
  for (int it = 0; it < IPT; ++it)
#pragma unroll
    for (int n = 0; n < N; ++n) ex[it][n] = s_tot[(it * NW + wid) * N + n] + inc[it][n] - v[it][n];
#pragma unroll
  for (int n = 0; n < N; ++n) total[n] = s_tot[NS * N + n];
  __syncthreads();
}

// Adds every thread's v into an LDS total with one atomic per wavefront (the
// wave's sum by DPP); every thread of the workgroup calls it.
__device__ inline void add_to(uint32_t* dst, uint32_t v) {
  const uint32_t t = wave::sum(v);
  if ((threadIdx.x & 63) == 0 && t) atomicAdd(dst, t);
}
__device__ inline void add_to(unsigned long long* dst, uint64_t v) {
  const uint64_t t = wave::sum(v);
  if ((threadIdx.x & 63) == 0 && t) atomicAdd(dst, (unsigned long long)t);
}

// Transition category.  Leaving the GPU for a tier that keeps the KV (CPU,
// SSD) is a swap-out, the reverse a swap-in.
__device__ inline uint8_t category(uint8_t from, uint8_t to) {
  if (from == to) return MORI_CAT_KEPT;
  switch (from) {
    case MORI_TIER_GPU: return to == MORI_TIER_WAIT ? MORI_CAT_DROP_GPU : MORI_CAT_OUT;
    case MORI_TIER_CPU:
      return to == MORI_TIER_GPU ? MORI_CAT_IN : (to == MORI_TIER_SSD ? MORI_CAT_CPU_SSD : MORI_CAT_DROP_CPU);
    case MORI_TIER_SSD:
      return to == MORI_TIER_GPU ? MORI_CAT_IN : (to == MORI_TIER_CPU ? MORI_CAT_SSD_CPU : MORI_CAT_DROP_SSD);
    default:
      return to == MORI_TIER_GPU ? MORI_CAT_ADMIT_GPU : (to == MORI_TIER_CPU ? MORI_CAT_ADMIT_CPU : MORI_CAT_ADMIT_SSD);
  }
}

template <int RT, int IPT>
__global__ __launch_bounds__(RT) void rank_partition_kernel(PlanArgs a) {
  constexpr int NW = RT / 64;  // wavefronts
  constexpr int NCNT = RADIX * NW;  // digit counters, (digit, wave)
  constexpr int CPT = NCNT / RT;         // consecutive counters per thread in their scan
  static_assert(NCNT % RT == 0, "whole counters per thread");
  // counter c lives at c + c / 32: a thread's CPT consecutive counters then
  // fall in different banks from its neighbours'
  auto cidx = [](uint32_t c) { return c + (c >> 5); };
  __shared__ uint64_t s_key[RT * IPT];  // sort scratch, then the inclusive byte prefix by rank
  __shared__ uint32_t s_id[RT * IPT];   // sort scratch, then blocks by rank
  __shared__ uint32_t s_cnt[NCNT + NCNT / 32];
  __shared__ uint8_t s_tier[RT * IPT];
  __shared__ uint32_t s_nblk[RT * IPT];  // blocks of program x
  __shared__ uint8_t s_told[RT * IPT];   // old tier of program x
  __shared__ uint64_t s_tot[(IPT * NW + 1) * 2];
  __shared__ uint32_t s_w32[NW + 1];
  __shared__ unsigned long long s_or, s_and;
  __shared__ uint32_t s_err, s_m_gpu, s_m_cpu, s_m_ssd;
  __shared__ uint32_t s_grp[5], s_cpu_reasoning, s_k_gpu, s_k_cpu;
  __shared__ uint32_t s_n_drop_gpu, s_n_drop_cpu, s_n_admit_gpu, s_n_admit_cpu;
  __shared__ unsigned long long s_gpu_after, s_cpu_after, s_ssd_after, s_gpu_part, s_upper_part;

  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  if (blockIdx.x > 0) {
    // the other workgroups set up the page state for the page kernels (it
    // depends on the caller's free map only)
    const uint64_t stride = (uint64_t)(gridDim.x - 1) * RT;
    for (uint64_t pg = (uint64_t)(blockIdx.x - 1) * RT + tid; pg < a.NB; pg += stride)
      a.pstate[pg] = a.free_map[pg] ? PS_FREE : 0u;
    return;
  }
  const uint32_t P = a.P;
  const bool incremental = (a.flags & MORI_F_INCREMENTAL) != 0;
  const bool ssd = (a.flags & MORI_F_SSD_TIER) != 0;
  const uint8_t top_tier = ssd ? MORI_TIER_SSD : MORI_TIER_WAIT;
  if (tid == 0) {
    s_err = 0;
    s_or = 0;
    s_and = ~0ull;
    s_m_gpu = s_m_cpu = s_m_ssd = 0;
    for (int g = 0; g < 5; ++g) s_grp[g] = 0;
    s_cpu_reasoning = s_k_gpu = s_k_cpu = 0;
    s_n_drop_gpu = s_n_drop_cpu = s_n_admit_gpu = s_n_admit_cpu = 0;
    s_gpu_after = s_cpu_after = s_ssd_after = 0;
    s_gpu_part = s_upper_part = 0;
  }
  __syncthreads();

  // ---- 1. validation, Eq. 1, keys --------------------------------------
  uint64_t key[IPT];
  uint32_t id[IPT];
  uint32_t err = 0;
  if (tid == 0) {
    if (a.tbl_off[0] != 0u) err |= MORI_DEV_BAD_TBL_OFF;
    if (a.tbl_off[P] > a.tbl_len) err |= MORI_DEV_BAD_TBL_OFF;
  }
  unsigned long long k_or = 0, k_and = ~0ull;
#pragma unroll
  for (int it = 0; it < IPT; ++it) {
    const uint32_t x = it * RT + tid;
    key[it] = ~0ull;  // padding sorts after every real key
    id[it] = x;
    if (x >= P) continue;
    // every load of the program first, none behind a branch, so they are in
    // flight together: one memory latency instead of one per load
    const bool given = (a.flags & MORI_F_IDLENESS_GIVEN) != 0;
    const bool need_status = incremental || (a.flags & MORI_F_STATUS_KEY);
    const uint8_t told = a.tier[x];
    const uint32_t off0 = a.tbl_off[x], off1 = a.tbl_off[x + 1];
    const uint8_t st = need_status ? a.status[x] : 0;
    float rv[8], cv[8];  // the first eight cycles of the window (clamped indices: k >= 1)
    const float* w = given ? nullptr : a.window + (size_t)x * a.k * 2;
    if (!given) {
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const uint32_t j = min((uint32_t)u, a.k - 1);
        rv[u] = w[2 * j];
        cv[u] = w[2 * j + 1];
      }
    }
    if (told > top_tier) err |= MORI_DEV_BAD_TIER;
    if (off1 < off0) err |= MORI_DEV_BAD_TBL_OFF;
    s_nblk[x] = off1 - off0;
    s_told[x] = told;
    float v;
    if (given) {
      v = a.idleness[x];
      if (!(v >= 0.0f && v <= 1.0f)) err |= MORI_DEV_BAD_IDLENESS;
    } else {
      float t_reasoning = 0.0f, t_acting = 0.0f;
      for (uint32_t j0 = 0; j0 < a.k; j0 += 8) {  // eight cycles' loads in flight, then the sums in order
        if (j0 > 0) {
#pragma unroll
          for (int u = 0; u < 8; ++u) {
            const uint32_t j = min(j0 + u, a.k - 1);
            rv[u] = w[2 * j];
            cv[u] = w[2 * j + 1];
          }
        }
#pragma unroll
        for (int u = 0; u < 8; ++u) {
          if (j0 + u >= a.k) break;
          const float r = rv[u], c = cv[u];
          if (!(r >= 0.0f) || !(c >= 0.0f) || __builtin_isinf(r) || __builtin_isinf(c)) err |= MORI_DEV_BAD_WINDOW;
          t_reasoning = t_reasoning + r;
          t_acting = t_acting + c;
        }
      }
      const float total = t_reasoning + t_acting;
      if (__builtin_isinf(t_reasoning) || __builtin_isinf(t_acting) || __builtin_isinf(total))
        err |= MORI_DEV_BAD_WINDOW;
      v = (total > 0.0f) ? t_acting / total : 0.0f;
    }
    if (v == 0.0f) v = 0.0f;  // a negative zero keys like +0
    const uint32_t bits = __float_as_uint(v);  // < 2^30 for idleness in [0, 1]
    uint64_t k;
    if (incremental) {
      if (st > MORI_ST_NEW) err |= MORI_DEV_BAD_STATUS;
      const uint64_t acting = st == MORI_ST_ACTING;
      uint64_t grp;
      uint64_t sub = bits;
      if (told == MORI_TIER_GPU || told == MORI_TIER_CPU) {
        grp = told;  // Reasoning before Acting, then idleness: the reverse of the demotion order
        sub |= acting << 31;
      } else if (st == MORI_ST_NEW) {
        grp = 3;  // new arrivals: smallest context first
        const uint32_t nb = off1 - off0;
        if (nb >= 0x80000000u) err |= MORI_DEV_BAD_TBL_OFF;
        sub |= (uint64_t)nb << 30;
      } else {
        grp = acting ? 4 : 2;
      }
      k = (grp << GROUP_SHIFT) | sub;
    } else {
      k = bits;
      if ((a.flags & MORI_F_STATUS_KEY) && st == MORI_ST_ACTING) k |= 0x80000000u;
    }
    key[it] = k;
    k_or |= k;
    k_and &= k;
  }
  {
    const uint64_t w_or = wave::all_or<uint64_t>(k_or), w_and = wave::all_and<uint64_t>(k_and);
    if (lane == 0 && w_or) atomicOr(&s_or, (unsigned long long)w_or);
    if (lane == 0 && w_and != ~0ull) atomicAnd(&s_and, (unsigned long long)w_and);
  }
  if (err) atomicOr(&s_err, err);
  if constexpr (!(IPT == 1 && RT <= 256)) {  // the first radix pass's digit counters
#pragma unroll
    for (int j = 0; j < CPT; ++j) s_cnt[cidx(j * RT + tid)] = 0;
  }
  __syncthreads();
  if (s_err) {
    if (tid == 0) {
      DevSummary z = {};
      z.num_programs = P;
      z.error = s_err;
      *a.sum = z;
      *host_mirror(a, a.sum) = z;
      a.swap_err[0] = a.swap_err[1] = 0;
    }
    return;
  }

  // Incremental keys: the listing group moves down from the top bits to just
  // above the highest bit any program's priority uses (the same order), so the
  // radix sort spends no pass on the bits between.  OR and AND of the keys
  // follow, as the fields do not overlap.
  uint32_t gshift = GROUP_SHIFT;
  uint64_t kor = s_or, kand = s_and;
  if (incremental) {
    constexpr uint64_t SUB = (1ull << GROUP_SHIFT) - 1;
    const uint64_t sub_or = kor & SUB;
    gshift = sub_or ? 64u - (uint32_t)__clzll(sub_or) : 0u;
    auto pack = [&](uint64_t k) { return ((k >> GROUP_SHIFT) << gshift) | (k & SUB); };
#pragma unroll
    for (int it = 0; it < IPT; ++it)
      if (it * RT + tid < (int)P) key[it] = pack(key[it]);
    kor = pack(kor);
    kand = pack(kand);
  }

  // ---- 2. stable sort of (key, id) ---------------------------------------
  if constexpr (IPT == 1 && RT <= 256) {
    // P <= 256: each program's rank is the number of programs before it in
    // (key, id) order, counted against every key in LDS (the same address for
    // all lanes, a broadcast): P steps and four barriers, where the radix sort
    // takes up to sixteen passes of several barriers and a workgroup scan each.
    s_key[tid] = key[0];
    __syncthreads();
    uint32_t rank = tid;  // padding keeps its slot: every real rank is below P
    if ((uint32_t)tid < P) {
      // eight keys' loads in flight per step; the padding keys past P (all
      // ones, above every real key) count for nobody
      const uint64_t k = key[0];
      const uint32_t P8 = (P + 7u) & ~7u;
      rank = 0;
      for (uint32_t j0 = 0; j0 < P8; j0 += 8) {
        uint64_t kj[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) kj[u] = s_key[j0 + u];
#pragma unroll
        for (int u = 0; u < 8; ++u) rank += (kj[u] < k) | ((kj[u] == k) & (j0 + u < (uint32_t)tid));
      }
    }
    __syncthreads();
    s_key[rank] = key[0];
    s_id[rank] = id[0];
    __syncthreads();
    key[0] = s_key[tid];
    id[0] = s_id[tid];
    __syncthreads();
  } else {
    // LSD radix sort, 8-bit digits (at most four passes over idleness keys).
    // During the sort each wave holds a block of 64 * IPT consecutive
    // positions (slice it of wave w: positions w * 64 * IPT + it * 64 + lane)
    // and ranks its slices in order, a running count per (digit, wave) in LDS
    // carrying the ranks from slice to slice; those counters, scanned in
    // (digit, wave) order, give every group its output base, so a pass is
    // stable.  Items move to the blocked order before the first pass and back
    // to the striped one (item it of thread tid at it * RT + tid) in the last.
    // Digits on which every real key agrees are skipped; padding keeps the
    // tail.  Five barriers a pass: counts, wave totals, bases, scatter, and the
    // read-back that also clears the next pass's counters.
    const uint64_t varying = kor ^ kand;
    const uint64_t lanemask_lt = (1ull << lane) - 1ull;
    int last_shift = -1;
    for (int shift = 0; shift < KEY_BITS; shift += RADIX_BITS)
      if ((varying >> shift) & (RADIX - 1)) last_shift = shift;
    const uint32_t blk = (uint32_t)wid * 64 * IPT + lane;  // this lane's position in slice 0
    if (IPT > 1 && last_shift >= 0) {  // to the blocked order (positions are program ids here)
#pragma unroll
      for (int it = 0; it < IPT; ++it) {
        s_key[it * RT + tid] = key[it];
        s_id[it * RT + tid] = id[it];
      }
      __syncthreads();
#pragma unroll
      for (int it = 0; it < IPT; ++it) {
        key[it] = s_key[blk + it * 64];
        id[it] = s_id[blk + it * 64];
      }
      // the first pass overwrites s_key only after its first barriers
    }
    for (int shift = 0; shift <= last_shift; shift += RADIX_BITS) {
      if (((varying >> shift) & (RADIX - 1)) == 0) continue;
      uint32_t digit[IPT], lrank[IPT];
#pragma unroll
      for (int it = 0; it < IPT; ++it) {
        const uint32_t d = (uint32_t)(key[it] >> shift) & (RADIX - 1);
        const uint64_t same = ~wave::digit_differs<RADIX_BITS>(d);
        const uint32_t r = __popcll(same & lanemask_lt);
        const uint32_t c = cidx(d * NW + wid);
        const uint32_t before = s_cnt[c];  // keys of digit d in this wave's earlier slices
        __builtin_amdgcn_wave_barrier();
        if (r == 0) s_cnt[c] = before + __popcll(same);  // read by the next slice's lanes
        __builtin_amdgcn_wave_barrier();
        digit[it] = d;
        lrank[it] = before + r;
      }
      __syncthreads();
      uint32_t loc[CPT], sum = 0;
#pragma unroll
      for (int j = 0; j < CPT; ++j) {
        loc[j] = s_cnt[cidx(tid * CPT + j)];
        sum += loc[j];
      }
      // this thread's base: its wave's exclusive scan plus the totals of the
      // waves before it (lane w < wid reads wave w's total)
      const uint32_t incl = wave::incl_add(sum);
      if (lane == 63) s_w32[wid] = incl;
      __syncthreads();
      uint32_t base = incl - sum + wave::sum(lane < wid ? s_w32[lane] : 0u);
#pragma unroll
      for (int j = 0; j < CPT; ++j) {
        s_cnt[cidx(tid * CPT + j)] = base;
        base += loc[j];
      }
      __syncthreads();
#pragma unroll
      for (int it = 0; it < IPT; ++it) {
        const uint32_t pos = s_cnt[cidx(digit[it] * NW + wid)] + lrank[it];
        s_key[pos] = key[it];
        s_id[pos] = id[it];
      }
      __syncthreads();
#pragma unroll
      for (int it = 0; it < IPT; ++it) {
        const uint32_t x = shift == last_shift ? it * RT + tid : blk + it * 64;  // striped after the last pass
        key[it] = s_key[x];
        id[it] = s_id[x];
      }
#pragma unroll
      for (int j = 0; j < CPT; ++j) s_cnt[cidx(j * RT + tid)] = 0;  // every base of this pass is read
      __syncthreads();
    }
  }
  // item x now holds rank x: id[it] is the program at rank it * RT + tid
  uint32_t nb[IPT];
#pragma unroll
  for (int it = 0; it < IPT; ++it) {
    const uint32_t r = it * RT + tid;
    nb[it] = 0;
    if (r < P) nb[it] = s_nblk[id[it]];
  }
  __syncthreads();  // s_id is reused for blocks by rank
#pragma unroll
  for (int it = 0; it < IPT; ++it) s_id[it * RT + tid] = nb[it];

  // ---- 3. KV-byte prefix in that order and the placement ----------------
  uint64_t S[IPT];
  {
    uint64_t bytes[IPT][1], ex[IPT][1], tot[1];
#pragma unroll
    for (int it = 0; it < IPT; ++it) bytes[it][0] = (uint64_t)nb[it] * a.block_bytes;
    scan_slices<NW, IPT, 1>(bytes, ex, s_tot, tot);
#pragma unroll
    for (int it = 0; it < IPT; ++it) {
      S[it] = ex[it][0] + bytes[it][0];
      s_key[it * RT + tid] = S[it];
    }
  }
  if (incremental) {
    // listing groups: [0, g1) GPU, [g1, g2) CPU, [g2, g3) Waiting returning,
    // [g3, g4) new arrivals, [g4, P) Waiting Acting
    uint32_t gc[5] = {0, 0, 0, 0, 0}, cr = 0;
#pragma unroll
    for (int it = 0; it < IPT; ++it) {
      const uint32_t r = it * RT + tid;
      const uint32_t g = r < P ? (uint32_t)(key[it] >> gshift) : 5u;
      const uint64_t sub = gshift ? key[it] & ((1ull << gshift) - 1) : 0ull;  // priority: Acting bit 31
#pragma unroll
      for (int j = 0; j < 5; ++j) gc[j] += g == (uint32_t)j;
      cr += g == MORI_TIER_CPU && !((sub >> 31) & 1u);
    }
#pragma unroll
    for (int j = 0; j < 5; ++j) add_to(&s_grp[j], gc[j]);
    add_to(&s_cpu_reasoning, cr);
    __syncthreads();
    const uint32_t g1 = s_grp[0], g2 = g1 + s_grp[1], g3 = g2 + s_grp[2], g4 = g3 + s_grp[3];
    const uint64_t gpu_total = g1 ? s_key[g1 - 1] : 0;
    // (1) CPU admission control and (2) demotion from GPU: each tier keeps the
    // longest prefix of its group that fits its budget (the rest, in reverse,
    // is the demotion order's shortest prefix whose removal fits)
    uint32_t kg = 0, kc = 0;
#pragma unroll
    for (int it = 0; it < IPT; ++it) {
      const uint32_t r = it * RT + tid;
      if (r < g1 && S[it] <= a.gpu_bytes) ++kg;
      if (r >= g1 && r < g2 && S[it] - gpu_total <= a.cpu_bytes) ++kc;
    }
    add_to(&s_k_gpu, kg);
    add_to(&s_k_cpu, kc);
    __syncthreads();
    const uint32_t k_gpu = s_k_gpu, k_cpu = s_k_cpu;
    const uint64_t gpu_kept = k_gpu ? s_key[k_gpu - 1] : 0;
    const uint64_t cpu_kept = k_cpu ? s_key[g1 + k_cpu - 1] - gpu_total : 0;
    const uint64_t room_cpu = a.cpu_bytes - cpu_kept;
    const uint64_t room_gpu = a.gpu_bytes - gpu_kept;
    const bool victims_fit = gpu_total - gpu_kept <= room_cpu;
    const uint32_t c_end = g1 + min(k_cpu, s_cpu_reasoning);  // CPU candidates: [g1, c_end)
#pragma unroll
    for (int it = 0; it < IPT; ++it) {
      const uint32_t r = it * RT + tid;
      uint8_t t;
      if (r < k_gpu) t = MORI_TIER_GPU;
      else if (r < g1) t = victims_fit ? MORI_TIER_CPU : MORI_TIER_WAIT;  // else walked below
      else if (r < g1 + k_cpu) t = MORI_TIER_CPU;
      else t = MORI_TIER_WAIT;
      s_tier[r] = t;
    }
    // (3) promotion: a strict prefix of the candidates' byte scan
    if (!(a.flags & MORI_F_SKIP_FIT)) {
      uint64_t cb[IPT][1], ex[IPT][1], tot[1];
      bool cand[IPT];
#pragma unroll
      for (int it = 0; it < IPT; ++it) {
        const uint32_t r = it * RT + tid;
        cand[it] = (r >= g1 && r < c_end) || (r >= g2 && r < g4);
        cb[it][0] = cand[it] ? (uint64_t)nb[it] * a.block_bytes : 0;
      }
      scan_slices<NW, IPT, 1>(cb, ex, s_tot, tot);
#pragma unroll
      for (int it = 0; it < IPT; ++it)
        if (cand[it] && ex[it][0] + cb[it][0] <= room_gpu) s_tier[it * RT + tid] = MORI_TIER_GPU;
    }
    __syncthreads();
    if (tid == 0) {
      if (!victims_fit) {  // each victim, most demotable first, to the CPU tier if it still fits
        uint64_t room = room_cpu;
        for (uint32_t r = g1; r-- > k_gpu;) {
          const uint64_t b = (uint64_t)s_id[r] * a.block_bytes;
          if (b <= room) {
            room -= b;
            s_tier[r] = MORI_TIER_CPU;
          } else {
            s_tier[r] = MORI_TIER_WAIT;
          }
        }
      }
      if (a.flags & MORI_F_SKIP_FIT) {
        uint64_t room = room_gpu;
        for (int part = 0; part < 2; ++part) {
          const uint32_t lo = part ? g2 : g1, hi = part ? g4 : c_end;
          for (uint32_t r = lo; r < hi; ++r) {
            const uint64_t b = (uint64_t)s_id[r] * a.block_bytes;
            if (b <= room) {
              room -= b;
              s_tier[r] = MORI_TIER_GPU;
            }
          }
        }
      }
    }
    __syncthreads();
    uint32_t ng = 0, nc = 0;
#pragma unroll
    for (int it = 0; it < IPT; ++it) {
      const uint32_t r = it * RT + tid;
      if (r >= P) continue;
      ng += s_tier[r] == MORI_TIER_GPU;
      nc += s_tier[r] == MORI_TIER_CPU;
    }
    add_to(&s_m_gpu, ng);
    add_to(&s_m_cpu, nc);
  } else if (!(a.flags & MORI_F_SKIP_FIT)) {
    // S is non-decreasing in rank order, so the longest feasible prefix is
    // the number of ranks whose inclusive prefix fits the budget.
    uint32_t c = 0;
#pragma unroll
    for (int it = 0; it < IPT; ++it)
      if (it * RT + tid < (int)P && S[it] <= a.gpu_bytes) ++c;
    add_to(&s_m_gpu, c);
    __syncthreads();
    const uint32_t m_gpu = s_m_gpu;
#pragma unroll
    for (int it = 0; it < IPT; ++it)
      if (m_gpu > 0 && it * RT + tid == (int)m_gpu - 1) s_gpu_part = S[it];
    __syncthreads();
    const uint64_t gpu_part = s_gpu_part;
    c = 0;
#pragma unroll
    for (int it = 0; it < IPT; ++it) {
      const uint32_t r = it * RT + tid;
      if (r >= m_gpu && r < P && S[it] - gpu_part <= a.cpu_bytes) ++c;
    }
    add_to(&s_m_cpu, c);
    __syncthreads();
    const uint32_t m_cpu = s_m_cpu, upper = m_gpu + m_cpu;
    uint32_t m_ssd = 0;
    if (ssd) {  // Sec. 7.1: the run after the CPU tier's, within the SSD budget
#pragma unroll
      for (int it = 0; it < IPT; ++it)
        if (upper > 0 && it * RT + tid == (int)upper - 1) s_upper_part = S[it];
      __syncthreads();
      const uint64_t upper_part = s_upper_part;
      c = 0;
#pragma unroll
      for (int it = 0; it < IPT; ++it) {
        const uint32_t r = it * RT + tid;
        if (r >= upper && r < P && S[it] - upper_part <= a.ssd_bytes) ++c;
      }
      add_to(&s_m_ssd, c);
      __syncthreads();
      m_ssd = s_m_ssd;
    }
#pragma unroll
    for (int it = 0; it < IPT; ++it) {
      const uint32_t r = it * RT + tid;
      s_tier[r] = r < m_gpu ? MORI_TIER_GPU
                : r < upper ? MORI_TIER_CPU
                : r < upper + m_ssd ? MORI_TIER_SSD : MORI_TIER_WAIT;
    }
  } else {
    // Greedy walk in rank order: first tier that still has room.
    __syncthreads();
    if (tid == 0) {
      uint64_t room_gpu = a.gpu_bytes, room_cpu = a.cpu_bytes, room_ssd = a.ssd_bytes;
      uint32_t ng = 0, nc = 0, ns = 0;
      for (uint32_t r = 0; r < P; ++r) {
        const uint64_t bytes = (uint64_t)s_id[r] * a.block_bytes;
        if (bytes <= room_gpu) {
          room_gpu -= bytes;
          s_tier[r] = MORI_TIER_GPU;
          ++ng;
        } else if (bytes <= room_cpu) {
          room_cpu -= bytes;
          s_tier[r] = MORI_TIER_CPU;
          ++nc;
        } else if (ssd && bytes <= room_ssd) {
          room_ssd -= bytes;
          s_tier[r] = MORI_TIER_SSD;
          ++ns;
        } else {
          s_tier[r] = MORI_TIER_WAIT;
        }
      }
      s_m_gpu = ng;
      s_m_cpu = nc;
      s_m_ssd = ns;
    }
  }
  __syncthreads();

  // ---- 4. sticky diff: categories, lists in rank order, bases -----------
  // packed scans: A = pages_out | pages_in << 32, B = pages_admit | n_out << 32 | n_in << 48
  // Global stores wait until after the last barrier: a barrier waits for the
  // stores still in flight, so stores issued earlier would stall every one.
  uint64_t vab[IPT][2], exab[IPT][2], totab[2];
  uint8_t catv[IPT], tnewv[IPT];
  uint32_t n_dg = 0, n_dc = 0, n_ag = 0, n_ac = 0;
  uint64_t gpu_after = 0, cpu_after = 0, ssd_after = 0;
#pragma unroll
  for (int it = 0; it < IPT; ++it) {
    const uint32_t r = it * RT + tid;
    uint64_t va = 0, vb = 0;
    catv[it] = MORI_CAT_KEPT;
    if (r < P) {
      const uint32_t p = id[it];
      const uint8_t told = s_told[p], tnew = s_tier[r];
      const uint8_t c = category(told, tnew);
      catv[it] = c;
      tnewv[it] = tnew;
      if (c == MORI_CAT_OUT) va = nb[it], vb = 1ull << 32;
      if (c == MORI_CAT_IN) va = (uint64_t)nb[it] << 32, vb = 1ull << 48;
      if (c == MORI_CAT_ADMIT_GPU) vb = nb[it], ++n_ag;
      if (c == MORI_CAT_DROP_GPU) ++n_dg;
      if (c == MORI_CAT_DROP_CPU) ++n_dc;
      if (c == MORI_CAT_ADMIT_CPU) ++n_ac;
      if (tnew == MORI_TIER_GPU) gpu_after += (uint64_t)nb[it] * a.block_bytes;
      if (tnew == MORI_TIER_CPU) cpu_after += (uint64_t)nb[it] * a.block_bytes;
      if (tnew == MORI_TIER_SSD) ssd_after += (uint64_t)nb[it] * a.block_bytes;
    }
    vab[it][0] = va;
    vab[it][1] = vb;
  }
  scan_slices<NW, IPT, 2>(vab, exab, s_tot, totab);
  const uint64_t carryA = totab[0], carryB = totab[1];
  const uint32_t pages_out = (uint32_t)(carryA & 0xFFFFFFFFu), pages_in = (uint32_t)(carryA >> 32);
  const uint32_t pages_admit = (uint32_t)(carryB & 0xFFFFFFFFu);
  const uint32_t n_out = (uint32_t)((carryB >> 32) & 0xFFFFu), n_in = (uint32_t)(carryB >> 48);
  // program-indexed staging, so the per-program stores below are coalesced:
  // the new tier and the page base by program id (every read of the
  // rank-indexed s_tier and s_nblk came before the scan's first barrier)
#pragma unroll
  for (int it = 0; it < IPT; ++it) {
    const uint32_t r = it * RT + tid;
    if (r >= P) continue;
    const uint32_t p = id[it];
    const uint64_t exA = exab[it][0], exB = exab[it][1];
    s_tier[p] = tnewv[it];
    if (catv[it] == MORI_CAT_OUT) s_nblk[p] = (uint32_t)(exA & 0xFFFFFFFFu);
    if (catv[it] == MORI_CAT_IN) s_nblk[p] = (uint32_t)(exA >> 32);
    if (catv[it] == MORI_CAT_ADMIT_GPU) s_nblk[p] = pages_in + (uint32_t)(exB & 0xFFFFFFFFu);
  }
  add_to(&s_n_drop_gpu, n_dg);
  add_to(&s_n_drop_cpu, n_dc);
  add_to(&s_n_admit_gpu, n_ag);
  add_to(&s_n_admit_cpu, n_ac);
  add_to(&s_gpu_after, gpu_after);
  add_to(&s_cpu_after, cpu_after);
  add_to(&s_ssd_after, ssd_after);
  __syncthreads();

  // ---- 5. the plan's stores ------------------------------------------------
  // by rank: order, prefix and the swap lists
#pragma unroll
  for (int it = 0; it < IPT; ++it) {
    const uint32_t r = it * RT + tid;
    if (r >= P) continue;
    const uint32_t p = id[it];
    a.order[r] = p;
    a.prefix[r] = S[it];
    *host_mirror(a, a.order + r) = p;
    *host_mirror(a, a.prefix + r) = S[it];
    const uint64_t exA = exab[it][0], exB = exab[it][1];
    const uint32_t idx_out = (uint32_t)((exB >> 32) & 0xFFFFu), idx_in = (uint32_t)(exB >> 48);
    if (catv[it] == MORI_CAT_OUT) {
      const uint32_t pg = (uint32_t)(exA & 0xFFFFFFFFu);
      a.out_prog[idx_out] = p;
      a.out_pg_base[idx_out] = pg;
      *host_mirror(a, a.out_prog + idx_out) = p;
      *host_mirror(a, a.out_pg_base + idx_out) = pg;
    }
    if (catv[it] == MORI_CAT_IN) {  // programs promoted from the CPU (or SSD) tier take the first slots (Sec. 4.3.1)
      const uint32_t pg = (uint32_t)(exA >> 32);
      a.in_prog[idx_in] = p;
      a.in_pg_base[idx_in] = pg;
      *host_mirror(a, a.in_prog + idx_in) = p;
      *host_mirror(a, a.in_pg_base + idx_in) = pg;
    }
  }
  // by program id: tiers, categories and the page bases (swap-outs from their
  // first released page, swap-ins from theirs, then the programs admitted from
  // Waiting after every swap-in: priority (2))
#pragma unroll
  for (int it = 0; it < IPT; ++it) {
    const uint32_t x = it * RT + tid;
    if (x >= P) continue;
    const uint8_t told = s_told[x], tnew = s_tier[x], c = category(told, tnew);
    a.tier_old[x] = told;
    a.tier_new[x] = tnew;
    a.cat[x] = c;
    *host_mirror(a, a.tier_old + x) = told;
    *host_mirror(a, a.tier_new + x) = tnew;
    *host_mirror(a, a.cat + x) = c;
    if (c == MORI_CAT_OUT || c == MORI_CAT_IN || c == MORI_CAT_ADMIT_GPU) a.base[x] = s_nblk[x];
  }
  if (tid == 0) {
    a.out_pg_base[n_out] = pages_out;
    a.in_pg_base[n_in] = pages_in;
    *host_mirror(a, a.out_pg_base + n_out) = pages_out;
    *host_mirror(a, a.in_pg_base + n_in) = pages_in;
    DevSummary z = {};  // the page fields follow in the page kernels, which mirror the summary
    z.num_programs = P;
    z.m_gpu = s_m_gpu;
    z.m_cpu = s_m_cpu;
    z.m_ssd = s_m_ssd;
    z.n_out = n_out;
    z.n_in = n_in;
    z.n_drop_gpu = s_n_drop_gpu;
    z.n_drop_cpu = s_n_drop_cpu;
    z.n_admit_gpu = s_n_admit_gpu;
    z.n_admit_cpu = s_n_admit_cpu;
    z.pages_out = pages_out;
    z.pages_in = pages_in;
    z.pages_admit = pages_admit;
    z.bytes_out = (uint64_t)pages_out * a.block_bytes;
    z.bytes_in = (uint64_t)pages_in * a.block_bytes;
    z.gpu_bytes_after = s_gpu_after;
    z.cpu_bytes_after = s_cpu_after;
    z.ssd_bytes_after = s_ssd_after;
    z.need = (uint64_t)pages_in + pages_admit;
    *a.sum = z;
    a.swap_err[0] = a.swap_err[1] = 0;
  }
}

}  // namespace

hipError_t launch_rank(const PlanArgs& a, hipStream_t s) {
  static_assert(1024 * 4 == (int)MORI_MAX_PROGRAMS, "the large shape holds every program");
  // workgroup 0 ranks; the others (about four pages per thread) set up the page state
  auto grid = [&](uint32_t rt) {
    const uint64_t g = ((uint64_t)a.NB + 4ull * rt - 1) / (4ull * rt);
    return dim3(1 + (uint32_t)(g < 1024 ? g : 1024));
  };
  if (a.P <= 64) hipLaunchKernelGGL((rank_partition_kernel<64, 1>), grid(64), dim3(64), 0, s, a);
  else if (a.P <= 256) hipLaunchKernelGGL((rank_partition_kernel<256, 1>), grid(256), dim3(256), 0, s, a);
  else if (a.P <= 1024) hipLaunchKernelGGL((rank_partition_kernel<1024, 1>), grid(1024), dim3(1024), 0, s, a);
  else hipLaunchKernelGGL((rank_partition_kernel<1024, 4>), grid(1024), dim3(1024), 0, s, a);
  return hipGetLastError();
}

}  // namespace mori
