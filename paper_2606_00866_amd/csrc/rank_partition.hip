// Rank / boundary step of one rebalance, in a single 1024-thread workgroup.
//
//   1. idleness of every program by Eq. 1 (Sec. 4.2), binary32, totals
//      accumulated oldest cycle first from +0, correctly rounded division;
//   2. a 32-bit key per program (idleness bits, optionally the Acting bit of
//      the demotion order of Sec. 4.3.1) and a stable LSD radix sort of
//      (key, id) with wave64 ballots -- the relative ranking, busiest first;
//   3. an inclusive u64 scan of KV bytes in rank order and the two
//      capacity boundaries (Sec. 4.1 per-tier capacity, Sec. 7.2 fill from the
//      busiest end), or the greedy skip-fit walk;
//   4. the sticky diff (Sec. 4.3): per-program transition category, the
//      swap-out and swap-in lists in rank order and the page/slot bases.
//
// P <= 4096 programs fit in LDS (4 keys per thread), so the whole step is one
// launch of a few microseconds; nothing here is bandwidth-bound.
#include "mori_internal.h"

namespace mori {
namespace {

constexpr int RT = 1024;           // threads
constexpr int IPT = 4;             // items per thread, striped: item x = it * RT + tid
constexpr int NW = RT / 64;        // wavefronts
constexpr int RADIX_BITS = 4;
constexpr int RADIX = 1 << RADIX_BITS;
static_assert(RT * IPT == (int)MORI_MAX_PROGRAMS, "one key per thread slot");
static_assert(RADIX * IPT * NW == RT, "one digit counter per thread");

// Exclusive scan of one value per thread over the whole workgroup (thread
// order); *total receives the sum.  s_wave needs NW + 1 entries.
template <typename T>
__device__ T block_scan_excl(T v, T* s_wave, T* total) {
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
  T x = v;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    T y = __shfl_up(x, off, 64);
    if (lane >= off) x += y;
  }
  if (lane == 63) s_wave[wid] = x;
  __syncthreads();
  if (wid == 0) {
    T w = lane < NW ? s_wave[lane] : T(0);
    T wi = w;
#pragma unroll
    for (int off = 1; off < NW; off <<= 1) {
      T y = __shfl_up(wi, off, 64);
      if (lane >= off) wi += y;
    }
    if (lane < NW) s_wave[lane] = wi - w;
    if (lane == NW - 1) s_wave[NW] = wi;
  }
  __syncthreads();
  T res = s_wave[wid] + x - v;
  *total = s_wave[NW];
  __syncthreads();
  return res;
}

__device__ inline uint8_t category(uint8_t from, uint8_t to) {
  if (from == to) return MORI_CAT_KEPT;
  if (from == MORI_TIER_GPU) return to == MORI_TIER_CPU ? MORI_CAT_OUT : MORI_CAT_DROP_GPU;
  if (from == MORI_TIER_CPU) return to == MORI_TIER_GPU ? MORI_CAT_IN : MORI_CAT_DROP_CPU;
  return to == MORI_TIER_GPU ? MORI_CAT_ADMIT_GPU : MORI_CAT_ADMIT_CPU;
}

__global__ __launch_bounds__(RT) void rank_partition_kernel(PlanArgs a) {
  __shared__ uint32_t s_key[RT * IPT];
  __shared__ uint32_t s_id[RT * IPT];
  __shared__ uint32_t s_cnt[RT];
  __shared__ uint8_t s_tier[RT * IPT];
  __shared__ uint64_t s_w64[NW + 1];
  __shared__ uint32_t s_w32[NW + 1];
  __shared__ uint32_t s_err, s_or, s_and, s_m_gpu, s_m_cpu;
  __shared__ uint32_t s_n_drop_gpu, s_n_drop_cpu, s_n_admit_gpu, s_n_admit_cpu;
  __shared__ unsigned long long s_gpu_after, s_cpu_after, s_gpu_part;

  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  const uint32_t P = a.P;
  if (tid == 0) {
    s_err = 0;
    s_or = 0;
    s_and = 0xFFFFFFFFu;
    s_m_gpu = s_m_cpu = 0;
    s_n_drop_gpu = s_n_drop_cpu = s_n_admit_gpu = s_n_admit_cpu = 0;
    s_gpu_after = s_cpu_after = 0;
    s_gpu_part = 0;
    DevSummary z = {};
    z.num_programs = P;
    *a.sum = z;
    *a.swap_err = 0;
  }
  __syncthreads();

  // ---- 1. validation, Eq. 1, keys --------------------------------------
  uint32_t key[IPT], id[IPT];
  uint32_t err = 0;
  if (tid == 0) {
    if (a.tbl_off[0] != 0u) err |= MORI_DEV_BAD_TBL_OFF;
    if (a.tbl_off[P] > a.tbl_len) err |= MORI_DEV_BAD_TBL_OFF;
  }
#pragma unroll
  for (int it = 0; it < IPT; ++it) {
    const uint32_t x = it * RT + tid;
    key[it] = 0xFFFFFFFFu;  // padding sorts after every real key
    id[it] = x;
    if (x >= P) continue;
    if (a.tier[x] > MORI_TIER_WAIT) err |= MORI_DEV_BAD_TIER;
    if (a.tbl_off[x + 1] < a.tbl_off[x]) err |= MORI_DEV_BAD_TBL_OFF;
    float v;
    if (a.flags & MORI_F_IDLENESS_GIVEN) {
      v = a.idleness[x];
      if (!(v >= 0.0f && v <= 1.0f)) err |= MORI_DEV_BAD_IDLENESS;
    } else {
      float t_reasoning = 0.0f, t_acting = 0.0f;
      const float* w = a.window + (size_t)x * a.k * 2;
      for (uint32_t j = 0; j < a.k; ++j) {
        const float r = w[2 * j], c = w[2 * j + 1];
        if (!(r >= 0.0f) || !(c >= 0.0f) || __builtin_isinf(r) || __builtin_isinf(c)) err |= MORI_DEV_BAD_WINDOW;
        t_reasoning = t_reasoning + r;
        t_acting = t_acting + c;
      }
      const float total = t_reasoning + t_acting;
      if (__builtin_isinf(t_reasoning) || __builtin_isinf(t_acting) || __builtin_isinf(total))
        err |= MORI_DEV_BAD_WINDOW;
      v = (total > 0.0f) ? t_acting / total : 0.0f;
    }
    if (v == 0.0f) v = 0.0f;  // a negative zero keys like +0
    uint32_t bits = __float_as_uint(v);
    if ((a.flags & MORI_F_STATUS_KEY) && a.status[x] == 1) bits |= 0x80000000u;
    key[it] = bits;
    atomicOr(&s_or, bits);
    atomicAnd(&s_and, bits);
  }
  if (err) atomicOr(&s_err, err);
  __syncthreads();
  if (s_err) {
    if (tid == 0) atomicOr(&a.sum->error, s_err);
    return;
  }

  // ---- 2. stable LSD radix sort of (key, id), 4-bit digits ---------------
  // Digit counters are laid out (digit, it, wave) so an exclusive scan over
  // them in thread order gives every (digit, item slice, wave) its output base
  // in (digit, original position) order, i.e. a stable pass.  Digits on which
  // every real key agrees are skipped; padding keeps the tail.
  const uint32_t varying = s_or ^ s_and;
  const uint64_t lanemask_lt = (1ull << lane) - 1ull;
  for (int shift = 0; shift < 32; shift += RADIX_BITS) {
    if (((varying >> shift) & (RADIX - 1)) == 0) continue;
    uint32_t digit[IPT], lrank[IPT];
    s_cnt[tid] = 0;
    __syncthreads();
#pragma unroll
    for (int it = 0; it < IPT; ++it) {
      const uint32_t d = (key[it] >> shift) & (RADIX - 1);
      uint64_t same = ~0ull;
#pragma unroll
      for (int b = 0; b < RADIX_BITS; ++b) {
        const uint64_t bal = __ballot((d >> b) & 1u);
        same &= ((d >> b) & 1u) ? bal : ~bal;
      }
      const uint32_t r = __popcll(same & lanemask_lt);
      if (r == 0) s_cnt[(d * IPT + it) * NW + wid] = __popcll(same);
      digit[it] = d;
      lrank[it] = r;
    }
    __syncthreads();
    uint32_t tot;
    const uint32_t base = block_scan_excl<uint32_t>(s_cnt[tid], s_w32, &tot);
    s_cnt[tid] = base;
    __syncthreads();
#pragma unroll
    for (int it = 0; it < IPT; ++it) {
      const uint32_t pos = s_cnt[(digit[it] * IPT + it) * NW + wid] + lrank[it];
      s_key[pos] = key[it];
      s_id[pos] = id[it];
    }
    __syncthreads();
#pragma unroll
    for (int it = 0; it < IPT; ++it) {
      key[it] = s_key[it * RT + tid];
      id[it] = s_id[it * RT + tid];
    }
    __syncthreads();
  }
  // item x now holds rank x: id[it] is the program at rank it * RT + tid
  uint32_t nb[IPT];
#pragma unroll
  for (int it = 0; it < IPT; ++it) {
    const uint32_t r = it * RT + tid;
    nb[it] = 0;
    if (r < P) {
      a.order[r] = id[it];
      nb[it] = a.tbl_off[id[it] + 1] - a.tbl_off[id[it]];
    }
  }

  // ---- 3. KV-byte prefix in rank order and the boundaries ---------------
  uint64_t S[IPT];
  uint64_t carry = 0;
#pragma unroll
  for (int it = 0; it < IPT; ++it) {
    const uint64_t bytes = (uint64_t)nb[it] * a.block_bytes;
    uint64_t tot;
    const uint64_t ex = block_scan_excl<uint64_t>(bytes, s_w64, &tot);
    S[it] = carry + ex + bytes;
    carry += tot;
    const uint32_t r = it * RT + tid;
    if (r < P) a.prefix[r] = S[it];
  }
  if (!(a.flags & MORI_F_SKIP_FIT)) {
    // S is non-decreasing in rank order, so the longest feasible prefix is
    // the number of ranks whose inclusive prefix fits the budget.
    uint32_t c = 0;
#pragma unroll
    for (int it = 0; it < IPT; ++it)
      if (it * RT + tid < (int)P && S[it] <= a.gpu_bytes) ++c;
    if (c) atomicAdd(&s_m_gpu, c);
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
    if (c) atomicAdd(&s_m_cpu, c);
    __syncthreads();
    const uint32_t m_cpu = s_m_cpu;
#pragma unroll
    for (int it = 0; it < IPT; ++it) {
      const uint32_t r = it * RT + tid;
      s_tier[r] = r < m_gpu ? MORI_TIER_GPU : (r < m_gpu + m_cpu ? MORI_TIER_CPU : MORI_TIER_WAIT);
    }
  } else {
    // Greedy walk in rank order: first tier that still has room.
#pragma unroll
    for (int it = 0; it < IPT; ++it) s_key[it * RT + tid] = nb[it];
    __syncthreads();
    if (tid == 0) {
      uint64_t room_gpu = a.gpu_bytes, room_cpu = a.cpu_bytes;
      uint32_t ng = 0, nc = 0;
      for (uint32_t r = 0; r < P; ++r) {
        const uint64_t bytes = (uint64_t)s_key[r] * a.block_bytes;
        if (bytes <= room_gpu) {
          room_gpu -= bytes;
          s_tier[r] = MORI_TIER_GPU;
          ++ng;
        } else if (bytes <= room_cpu) {
          room_cpu -= bytes;
          s_tier[r] = MORI_TIER_CPU;
          ++nc;
        } else {
          s_tier[r] = MORI_TIER_WAIT;
        }
      }
      s_m_gpu = ng;
      s_m_cpu = nc;
    }
  }
  __syncthreads();

  // ---- 4. sticky diff: categories, lists in rank order, bases -----------
  // packed scans: A = pages_out | pages_in << 32, B = pages_admit | n_out << 32 | n_in << 48
  uint64_t exA[IPT], exB[IPT];
  uint8_t catv[IPT];
  uint64_t carryA = 0, carryB = 0;
  uint32_t n_dg = 0, n_dc = 0, n_ag = 0, n_ac = 0;
  uint64_t gpu_after = 0, cpu_after = 0;
#pragma unroll
  for (int it = 0; it < IPT; ++it) {
    const uint32_t r = it * RT + tid;
    uint64_t va = 0, vb = 0;
    catv[it] = MORI_CAT_KEPT;
    if (r < P) {
      const uint32_t p = id[it];
      const uint8_t told = a.tier[p], tnew = s_tier[r];
      const uint8_t c = category(told, tnew);
      catv[it] = c;
      a.tier_old[p] = told;
      a.tier_new[p] = tnew;
      a.cat[p] = c;
      if (c == MORI_CAT_OUT) va = nb[it], vb = 1ull << 32;
      if (c == MORI_CAT_IN) va = (uint64_t)nb[it] << 32, vb = 1ull << 48;
      if (c == MORI_CAT_ADMIT_GPU) vb = nb[it], ++n_ag;
      if (c == MORI_CAT_DROP_GPU) ++n_dg;
      if (c == MORI_CAT_DROP_CPU) ++n_dc;
      if (c == MORI_CAT_ADMIT_CPU) ++n_ac;
      if (tnew == MORI_TIER_GPU) gpu_after += (uint64_t)nb[it] * a.block_bytes;
      if (tnew == MORI_TIER_CPU) cpu_after += (uint64_t)nb[it] * a.block_bytes;
    }
    uint64_t tA, tB;
    exA[it] = carryA + block_scan_excl<uint64_t>(va, s_w64, &tA);
    exB[it] = carryB + block_scan_excl<uint64_t>(vb, s_w64, &tB);
    carryA += tA;
    carryB += tB;
  }
  const uint32_t pages_out = (uint32_t)(carryA & 0xFFFFFFFFu), pages_in = (uint32_t)(carryA >> 32);
  const uint32_t pages_admit = (uint32_t)(carryB & 0xFFFFFFFFu);
  const uint32_t n_out = (uint32_t)((carryB >> 32) & 0xFFFFu), n_in = (uint32_t)(carryB >> 48);
#pragma unroll
  for (int it = 0; it < IPT; ++it) {
    const uint32_t r = it * RT + tid;
    if (r >= P) continue;
    const uint32_t p = id[it];
    const uint32_t pg_out_ex = (uint32_t)(exA[it] & 0xFFFFFFFFu), pg_in_ex = (uint32_t)(exA[it] >> 32);
    const uint32_t pg_admit_ex = (uint32_t)(exB[it] & 0xFFFFFFFFu);
    const uint32_t idx_out = (uint32_t)((exB[it] >> 32) & 0xFFFFu), idx_in = (uint32_t)(exB[it] >> 48);
    switch (catv[it]) {
      case MORI_CAT_OUT:
        a.out_prog[idx_out] = p;
        a.out_pg_base[idx_out] = pg_out_ex;
        a.base[p] = pg_out_ex;
        break;
      case MORI_CAT_IN:  // promoted CPU programs take the first slots (priority (1) of Sec. 4.3.1)
        a.in_prog[idx_in] = p;
        a.in_pg_base[idx_in] = pg_in_ex;
        a.base[p] = pg_in_ex;
        break;
      case MORI_CAT_ADMIT_GPU:  // then programs admitted from Waiting (priority (2))
        a.base[p] = pages_in + pg_admit_ex;
        break;
      default:
        break;
    }
  }
  if (n_dg) atomicAdd(&s_n_drop_gpu, n_dg);
  if (n_dc) atomicAdd(&s_n_drop_cpu, n_dc);
  if (n_ag) atomicAdd(&s_n_admit_gpu, n_ag);
  if (n_ac) atomicAdd(&s_n_admit_cpu, n_ac);
  if (gpu_after) atomicAdd(&s_gpu_after, (unsigned long long)gpu_after);
  if (cpu_after) atomicAdd(&s_cpu_after, (unsigned long long)cpu_after);
  __syncthreads();
  if (tid == 0) {
    a.out_pg_base[n_out] = pages_out;
    a.in_pg_base[n_in] = pages_in;
    DevSummary* s = a.sum;
    s->m_gpu = s_m_gpu;
    s->m_cpu = s_m_cpu;
    s->n_out = n_out;
    s->n_in = n_in;
    s->n_drop_gpu = s_n_drop_gpu;
    s->n_drop_cpu = s_n_drop_cpu;
    s->n_admit_gpu = s_n_admit_gpu;
    s->n_admit_cpu = s_n_admit_cpu;
    s->pages_out = pages_out;
    s->pages_in = pages_in;
    s->pages_admit = pages_admit;
    s->bytes_out = (uint64_t)pages_out * a.block_bytes;
    s->bytes_in = (uint64_t)pages_in * a.block_bytes;
    s->gpu_bytes_after = s_gpu_after;
    s->cpu_bytes_after = s_cpu_after;
    s->need = (uint64_t)pages_in + pages_admit;
  }
}

}  // namespace

hipError_t launch_rank(const PlanArgs& a, hipStream_t s) {
  hipLaunchKernelGGL(rank_partition_kernel, dim3(1), dim3(RT), 0, s, a);
  return hipGetLastError();
}

}  // namespace mori
