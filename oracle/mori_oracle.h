/*
 * mori_oracle.h -- plain CPU oracle for MORI's idleness-ranked KV tier placement
 * (arXiv 2606.00866, "Idleness is Relative").
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing on the product path may include, link or
 * call this code; only the tests, the smoke check and the benchmark's CPU
 * baseline leg use it.  It shares no code, header or constant with the HIP
 * library: every definition below is restated from the paper on its own.
 *
 * What it computes, in the paper's order:
 *   1. idleness of every program, Eq. 1 (Sec. 4.2), over a window of k cycles;
 *   2. the relative ranking of all programs by idleness, busiest first
 *      (Sec. 1 and Sec. 4.3: idleness is relative, programs are ranked);
 *   3. the capacity-matched boundary: fill the GPU tier from the busiest end of
 *      the ranking until its byte budget is reached, then the CPU tier the same
 *      way; the rest waits (Sec. 4.1 three-tier queues, Sec. 4.3, Sec. 7.2);
 *   4. sticky placement: only programs whose tier changes move (Sec. 4.3), with
 *      KV pages of paged attention (Sec. 2.1) allocated lowest id first, pages
 *      free before the step ahead of released ones and, among those, pages
 *      nothing reads ahead of pages a swap-out reads;
 *   5. the byte movement this implies: demoted programs' pages copied into
 *      their contiguous host buffers, promoted programs' bytes copied back into
 *      newly allocated pages (Sec. 4.1: the CPU tier resumes over PCIe).
 *
 * Readings where the paper is silent are listed with each function.
 * Floating point: idleness is computed in IEEE binary32 because it decides an
 * integer (the ranking) and the GPU path takes that decision in binary32; the
 * oracle therefore uses the same precision and the same summation order.
 */
#ifndef MORI_ORACLE_H
#define MORI_ORACLE_H
#include <stdint.h>
#include <stddef.h>

#ifdef __cplusplus
extern "C" {
#endif

/* tiers (Sec. 4.1: GPU queue, CPU queue, Waiting queue; Sec. 7.1: an SSD
   tier below the CPU tier) */
#define ORC_GPU 0u
#define ORC_CPU 1u
#define ORC_WAIT 2u
#define ORC_SSD 3u
#define ORC_NONE 0xFFFFFFFFu /* table entry of a block that has no HBM page */

/* flags */
#define ORC_F_STATUS_KEY 1u     /* Acting programs rank after Reasoning ones (Sec. 4.3.1, demotion) */
#define ORC_F_SKIP_FIT 2u       /* greedy fit instead of a strict prefix boundary */
#define ORC_F_IDLENESS_GIVEN 4u /* idleness supplied directly instead of windows */
#define ORC_F_INCREMENTAL 8u    /* incremental sticky policy (Sec. 4.3.1) instead of the boundary */
#define ORC_F_SSD_TIER 16u      /* a third boundary: SSD tier after the CPU tier (Sec. 7.1) */

/* program status (Sec. 4.1): Reasoning = running or waiting for inference,
   Acting = inside a tool call, New = arrived and not yet run (waits for its
   first inference, no KV anywhere) */
#define ORC_ST_REASONING 0u
#define ORC_ST_ACTING 1u
#define ORC_ST_NEW 2u

/* result classes */
#define ORC_OK 0
#define ORC_E_INPUT 1  /* malformed program data: windows, idleness, tiers or table offsets */
#define ORC_E_POOL 2   /* inconsistent page pool: bad/duplicate/leaked/free-but-owned page */
#define ORC_E_NOSPC 3  /* not enough pages for the promoted programs */

/* transition categories, old tier -> new tier */
#define ORC_KEPT 0u
#define ORC_OUT 1u       /* GPU -> CPU or SSD: swap-out into the program's host buffer */
#define ORC_IN 2u        /* CPU or SSD -> GPU: swap-in from the program's host buffer */
#define ORC_DROP_GPU 3u  /* GPU -> WAIT: pages released, KV discarded */
#define ORC_DROP_CPU 4u  /* CPU -> WAIT */
#define ORC_ADMIT_GPU 5u /* WAIT -> GPU: pages reserved, no copy (prefill recomputes) */
#define ORC_ADMIT_CPU 6u /* WAIT -> CPU */
#define ORC_CPU_SSD 7u   /* CPU -> SSD: host buffer written to storage, no GPU work */
#define ORC_SSD_CPU 8u   /* SSD -> CPU */
#define ORC_DROP_SSD 9u  /* SSD -> WAIT */
#define ORC_ADMIT_SSD 10u /* WAIT -> SSD */

typedef struct {
  uint32_t layers, planes, block_tokens, row_bytes, num_blocks;
} orc_geometry;

typedef struct {
  uint32_t m_gpu, m_cpu, m_ssd;
  uint32_t n_out, n_in, n_drop_gpu, n_drop_cpu, n_admit_gpu, n_admit_cpu;
  uint64_t pages_out, pages_in, pages_admit;
  uint64_t pages_free_before, pages_released, pages_recycled, pages_free_after;
  uint64_t bytes_out, bytes_in, gpu_bytes_after, cpu_bytes_after, ssd_bytes_after;
  uint64_t pages_dropped; /* released pages of programs dropped to Waiting: reusable at once */
} orc_summary;

/* Eq. 1 for every program.  window is [P][k][2] (reasoning s, acting s), oldest first. */
int orc_idleness(uint32_t P, uint32_t k, const float* window, float* iota);

/* 32-bit ranking key from idleness (and status when ORC_F_STATUS_KEY is set). */
int orc_keys(uint32_t P, const float* iota, const uint8_t* status, uint32_t flags, uint32_t* key);

/* Ascending (key, program id) order; rank is its inverse permutation. */
void orc_order(uint32_t P, const uint32_t* key, uint32_t* order, uint32_t* rank);

/* Capacity-matched boundary over the ranking.  prefix[r] = KV bytes of the
 * first r+1 programs in rank order.  With ORC_F_SSD_TIER a third run after the
 * CPU tier's goes to the SSD tier (ssd_budget, m_ssd); otherwise m_ssd = 0. */
void orc_boundary(uint32_t P, const uint32_t* order, const uint32_t* nblk, uint64_t block_bytes,
                  uint64_t gpu_budget, uint64_t cpu_budget, uint64_t ssd_budget, uint32_t flags,
                  uint64_t* prefix, uint8_t* tier_new, uint32_t* m_gpu, uint32_t* m_cpu, uint32_t* m_ssd);

/* Incremental sticky placement (Sec. 4.3 and Sec. 4.3.1), the alternative to
 * the boundary: tiers change only to repair a capacity violation or to fill
 * free GPU capacity.
 *   1. CPU admission control: while the CPU tier holds more than its budget,
 *      its programs go to Waiting in demotion order.
 *   2. Demotion from GPU: while the GPU tier holds more than its budget, the
 *      next program in demotion order (Acting before Reasoning, then highest
 *      idleness) leaves the GPU; it goes to the CPU tier if it fits in what
 *      the CPU budget has left, otherwise to Waiting.  A Reasoning victim is
 *      demoted lazily (after its current inference step) by the caller.
 *   3. Promotion to GPU into the room left: CPU-tier programs waiting for
 *      inference, then returning Waiting programs waiting for inference, then
 *      new arrivals smallest context first; lowest idleness first within a
 *      level.  Programs moved in steps 1-2 are not candidates.  The walk stops
 *      at the first candidate that does not fit (ORC_F_SKIP_FIT: skips it).
 * order[] lists all programs by old tier and the priorities above (GPU and CPU
 * programs: Reasoning before Acting, then idleness; Waiting programs: returning
 * Reasoning ones by idleness, new arrivals by context then idleness, Acting
 * ones by idleness; ties lowest id first), so demotion runs from its end of a
 * tier group and promotion from the start; prefix[] accumulates bytes along it.
 * Rejects (ORC_E_INPUT) a status above 2, idleness outside [0, 1] and a new
 * arrival with 2^31 or more blocks. */
int orc_incremental(uint32_t P, const float* iota, const uint8_t* status, const uint8_t* tier_old,
                    const uint32_t* nblk, uint64_t block_bytes, uint64_t gpu_budget, uint64_t cpu_budget,
                    uint32_t flags, uint32_t* order, uint32_t* rank, uint64_t* prefix, uint8_t* tier_new,
                    uint32_t* m_gpu, uint32_t* m_cpu);

/* One whole rebalance: Eq. 1 -> ranking -> boundary -> sticky diff -> page
 * allocation -> table rewrite -> byte movement.  All state arrays are updated
 * in place only when the result is ORC_OK; on an error nothing is modified.
 *
 * pool_bytes [layers*planes][num_blocks][block_tokens*row_bytes] and host_bufs
 * [P] (one contiguous [layers*planes][nblk_p][block_tokens*row_bytes] buffer per
 * program) may both be NULL to compute the placement only.
 * Optional outputs (may be NULL): order, rank, tier_old_out, category, prefix, summary.
 * With ORC_F_INCREMENTAL the placement comes from orc_incremental (status
 * required) instead of the ranking and boundary.  With ORC_F_SSD_TIER tier 3
 * (SSD) is a valid tier, the boundary has a third run (ssd_budget), and an SSD
 * program's KV lives in its host buffer as a CPU program's does (the storage
 * I/O is the caller's); ORC_F_SSD_TIER with ORC_F_INCREMENTAL is rejected. */
int orc_rebalance(const orc_geometry* g, uint8_t* pool_bytes, uint32_t P, uint32_t k,
                  const float* window, const float* iota_given, const uint8_t* status,
                  const uint32_t* tbl_off, uint32_t tbl_len, uint32_t* tbl, uint8_t* tier,
                  uint8_t* free_map, uint64_t gpu_budget, uint64_t cpu_budget, uint64_t ssd_budget, uint32_t flags,
                  uint8_t* const* host_bufs, uint32_t* order, uint32_t* rank, uint8_t* tier_old_out,
                  uint8_t* category, uint64_t* prefix, orc_summary* summary);

/* ------------------------------------------------------------------------ */
/* Typed eviction order (Sec. 4.3.2, typed offloading on the engine).        */
/* Every KV block carries its program's type label -- busy (GPU queue), idle */
/* (CPU queue) or inactive (Waiting) -- and its last access time.  Eviction */
/* is least-recently-used within a type, with the type as the higher key,    */
/* in tier-reversed order: the GPU tier evicts inactive, then idle, then     */
/* busy blocks; the CPU tier evicts inactive, then busy, then idle blocks.   */
/* ------------------------------------------------------------------------ */
#define ORC_TYPE_BUSY 0u
#define ORC_TYPE_IDLE 1u
#define ORC_TYPE_INACTIVE 2u

/* order[j] = block evicted j-th from `tier` (ORC_GPU or ORC_CPU).  prefix[j] =
 * bytes freed by the first j+1 evictions (size[b] * unit_bytes each; size may
 * be NULL for one unit per block).  *count = fewest evictions that free at
 * least need_bytes (all N when even all of them free less).  Reading: equal
 * type and time go lowest block id first.  Returns ORC_E_INPUT for a type
 * label above 2 or a tier other than GPU/CPU. */
int orc_evict_order(uint32_t N, const uint8_t* type, const uint64_t* last_access, const uint32_t* size,
                    uint64_t unit_bytes, uint32_t tier, uint64_t need_bytes, uint32_t* order, uint64_t* prefix,
                    uint32_t* count);

/* ------------------------------------------------------------------------ */
/* Multi-replica admission of the shared Waiting queue (Sec. 4.1: one global */
/* Waiting queue, a GPU and a CPU queue per replica; Sec. 4.3.1: Waiting     */
/* promotions are bin-packed across replicas in decreasing size order, onto  */
/* the replica with the most available capacity; CPU-tier programs keep     */
/* their replica and are promoted there).                                     */
/* Candidates: status Reasoning (returning) before New; Acting programs stay */
/* waiting.  Within a level: larger KV first, then lower idleness, then id.  */
/* Each goes to the replica with the most room that can hold it (with        */
/* ORC_ADMIT_BEST_FIT: the least room that can), ties to the lower replica   */
/* index; if none can, it stays waiting (-1) and the next is tried.          */
/* ------------------------------------------------------------------------ */
#define ORC_ADMIT_BEST_FIT 1u

/* replica[p] in [0, R) or -1; room_after[R] = room minus what was admitted.
 * ORC_E_INPUT for R == 0, a status above 2 or idleness outside [0, 1]. */
int orc_replica_admit(uint32_t P, const uint64_t* bytes, const float* iota, const uint8_t* status, uint32_t R,
                      const uint64_t* room, uint32_t flags, int32_t* replica, uint64_t* room_after);

#ifdef __cplusplus
}
#endif
#endif
