/*
 * mori.h -- C ABI of libmori: the MI355X (gfx950) hot path of MORI's
 * idleness-ranked KV-cache placement (arXiv 2606.00866, "Idleness is
 * Relative: Exploiting Tool-Call Idle Windows for Offloading in Agentic
 * Systems with MORI").
 *
 * One rebalance of the three-tier placement of Sec. 4.1 (GPU HBM, CPU DRAM,
 * Waiting), as three calls:
 *
 *   mori_rank_partition  Eq. 1 idleness of every program (Sec. 4.2), the
 *                        relative ranking (Sec. 1, Sec. 4.3), the
 *                        capacity-matched GPU and CPU boundaries (Sec. 4.1
 *                        per-tier capacity, Sec. 7.2 fill from the busiest
 *                        end), the sticky diff (Sec. 4.3: only programs that
 *                        cross the boundary move), page allocation and the
 *                        block-table rewrite.
 *   mori_kv_swap_out     gathers the demoted programs' scattered KV pages into
 *                        one contiguous buffer per program (GPU -> CPU).
 *   mori_kv_swap_in      scatters the promoted programs' bytes into the pages
 *                        allocated for them (CPU -> GPU, Sec. 4.1: a CPU-tier
 *                        program resumes over PCIe).
 *
 * Conventions
 *   - Every call returns an int: MORI_OK (0) or a negative MORI_E* code.
 *     Nothing throws across the ABI.  Errors found on the host are reported
 *     before anything is enqueued and leave all caller memory untouched.
 *   - Device-side validation (program data, pool consistency, host
 *     addresses) sets bits of a device error word (MORI_DEV_*).  A plan that
 *     fails validation modifies no caller memory; its error is returned by
 *     mori_plan_wait and mori_query.
 *   - Streams are hipStream_t values passed as void*; NULL is the default
 *     stream.  The library never synchronises the device.  It blocks the host
 *     in mori_plan_wait, in copy-engine swaps (which need the plan), in
 *     mori_query(MORI_Q_DEVICE_ERROR), mori_profile_read, mori_register and
 *     mori_destroy; a kernel-mode swap waits until the previous one of its
 *     direction has read its address table.
 *   - Threads: a context is driven by one host thread at a time (its calls
 *     are not synchronised against each other); distinct contexts share no
 *     state, and mori_evict_order and mori_replica_admit keep none.
 *   - Ownership: the caller owns the pool, the program arrays, the host
 *     buffers and the streams.  The context owns its device scratch, a small
 *     pinned mirror of the plan and, for copy-engine swaps, device staging
 *     buffers, all allocated in mori_create and freed in mori_destroy.
 *
 * Layouts
 *   pool   [layers * planes][num_blocks][block_tokens][row_bytes] bytes in
 *          HBM.  A "run" is one (plane, page): block_tokens * row_bytes
 *          contiguous bytes.  A page of a program spans every plane.
 *   host   one contiguous buffer per CPU-resident program p:
 *          [layers * planes][nblk_p][block_tokens][row_bytes], so each
 *          program's runs of one plane are adjacent.
 *   nblk_p = tbl_off[p+1] - tbl_off[p] whole blocks; a program is never split
 *          across tiers (Sec. 1: a program sits in exactly one tier at a time).
 */
#ifndef MORI_H
#define MORI_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* ---- return codes ---------------------------------------------------- */
#define MORI_OK 0
#define MORI_EINVAL (-1)  /* bad argument: null/misaligned pointer, size, flag or mode */
#define MORI_ENOSPC (-2)  /* capacity: too many programs, staging too small, registry full */
#define MORI_ESTATE (-3)  /* call out of order (swap without a plan, swap twice, ...) */
#define MORI_EHIP (-4)    /* a HIP runtime call failed; mori_query(MORI_Q_LAST_HIP_ERROR) */
#define MORI_EDEVICE (-5) /* device-side validation failed; see the MORI_DEV_* bits */

/* ---- device error word bits ------------------------------------------- */
#define MORI_DEV_BAD_WINDOW 0x001u    /* window value negative, NaN or inf, or a total overflowed */
#define MORI_DEV_BAD_IDLENESS 0x002u  /* given idleness outside [0, 1] */
#define MORI_DEV_BAD_TIER 0x004u      /* tier value > 2 */
#define MORI_DEV_BAD_TBL_OFF 0x008u   /* tbl_off not starting at 0, decreasing, or past tbl_len */
#define MORI_DEV_PAGE_RANGE 0x010u    /* a GPU program's page id >= num_blocks */
#define MORI_DEV_PAGE_DUP 0x020u      /* a page owned twice, or owned and marked free */
#define MORI_DEV_PAGE_LEAK 0x040u     /* a page neither free nor owned */
#define MORI_DEV_NONRES_PAGE 0x080u   /* a CPU/Waiting program's table holds a page */
#define MORI_DEV_NOSPC 0x100u         /* not enough pages (unreachable for a consistent pool) */
#define MORI_DEV_HOST_ADDR 0x200u     /* swap address not 16-B aligned or outside registered memory */
#define MORI_DEV_BAD_BLOCK 0x400u     /* eviction order: type label > 2 or last access >= 2^62 */
#define MORI_DEV_BAD_STATUS 0x800u    /* incremental policy: status value > 2 */
#define MORI_DEV_STALL 0x1000u        /* eviction order: a sort pass waited too long on another
                                         workgroup (not expected; the result is not valid) */
/* classes: program data = 0x00F and 0x800, pool state = 0x0F0, capacity = 0x100, swap = 0x200,
   blocks = 0x400 */

/* ---- tiers, table sentinel, flags, copy modes -------------------------- */
#define MORI_TIER_GPU 0u
#define MORI_TIER_CPU 1u
#define MORI_TIER_WAIT 2u
#define MORI_TIER_SSD 3u /* only with MORI_F_SSD_TIER (Sec. 7.1: storage below the CPU tier) */
#define MORI_NO_PAGE 0xFFFFFFFFu

#define MORI_F_STATUS_KEY 1u     /* Acting programs (status 1) rank after all Reasoning ones */
#define MORI_F_SKIP_FIT 2u       /* greedy fit in rank order instead of a strict prefix */
#define MORI_F_IDLENESS_GIVEN 4u /* use programs.idleness instead of windows */
#define MORI_F_INCREMENTAL 8u    /* incremental sticky policy of Sec. 4.3.1 instead of the boundary */
#define MORI_F_SSD_TIER 16u      /* a third boundary in the ranking: the SSD tier (Sec. 7.1) */

/* program status (Sec. 4.1), read with MORI_F_STATUS_KEY or MORI_F_INCREMENTAL */
#define MORI_ST_REASONING 0u /* running inference or waiting for it */
#define MORI_ST_ACTING 1u    /* inside a tool call */
#define MORI_ST_NEW 2u       /* newly arrived, waiting for its first inference (Reasoning elsewhere) */

#define MORI_COPY_AUTO 0u   /* copy engines (chosen by measurement on MI355X) */
#define MORI_COPY_KERNEL 1u /* kernels load/store host-mapped memory directly; no host sync */
#define MORI_COPY_CE 2u     /* kernel gather/scatter through device staging + SDMA copies */

/* transition categories (mori_plan.category) */
#define MORI_CAT_KEPT 0u
#define MORI_CAT_OUT 1u       /* GPU -> CPU or SSD: bytes gathered to the host */
#define MORI_CAT_IN 2u        /* CPU or SSD -> GPU: bytes scattered into new pages */
#define MORI_CAT_DROP_GPU 3u  /* GPU -> Waiting: pages released, KV discarded */
#define MORI_CAT_DROP_CPU 4u  /* CPU -> Waiting */
#define MORI_CAT_ADMIT_GPU 5u /* Waiting -> GPU: pages reserved, no copy */
#define MORI_CAT_ADMIT_CPU 6u /* Waiting -> CPU: no copy */
#define MORI_CAT_CPU_SSD 7u   /* CPU -> SSD: the caller writes the host buffer to storage */
#define MORI_CAT_SSD_CPU 8u   /* SSD -> CPU: the caller reads it back into a host buffer */
#define MORI_CAT_DROP_SSD 9u  /* SSD -> Waiting */
#define MORI_CAT_ADMIT_SSD 10u /* Waiting -> SSD: no copy */

#define MORI_MAX_PROGRAMS 4096u
#define MORI_MAX_WINDOW 64u
#define MORI_MAX_RANGES 64u

typedef struct mori_ctx mori_ctx;

/* The paged KV pool in HBM (PagedAttention-style blocks, Sec. 2.1). */
typedef struct {
  uint32_t layers;       /* >= 1 */
  uint32_t planes;       /* >= 1: 2 for K and V, 1 for a compressed latent */
  uint32_t block_tokens; /* >= 1 tokens per block */
  uint32_t row_bytes;    /* bytes per token per (layer, plane); multiple of 16 */
  uint32_t num_blocks;   /* pages in the pool, < 2^32 - 1 */
  void* base;            /* device pointer, 256-B aligned, layout in the header comment */
} mori_pool;

/* Per-program state (Sec. 4.1: status, context size and recent durations). */
typedef struct {
  uint32_t num_programs;   /* P <= max_programs of the context */
  uint32_t window_k;       /* cycles per idleness window, 1..MORI_MAX_WINDOW (the paper uses 5) */
  const float* window;     /* device [P][window_k][2]: (reasoning s, acting s), oldest cycle
                              first; the newest acting entry is the ongoing call's elapsed time */
  const float* idleness;   /* device [P]; read only with MORI_F_IDLENESS_GIVEN */
  const uint8_t* status;   /* device [P] MORI_ST_*; read only with MORI_F_STATUS_KEY (where only
                              MORI_ST_ACTING counts) or MORI_F_INCREMENTAL */
  const uint32_t* tbl_off; /* device [P+1] CSR offsets into tbl; nblk_p = tbl_off[p+1]-tbl_off[p] */
  uint32_t tbl_len;        /* entries allocated in tbl (>= tbl_off[P]) */
  uint32_t* tbl;           /* device [tbl_len], in/out: page id of each logical block of a
                              GPU-resident program, MORI_NO_PAGE for every other program */
  uint8_t* tier;           /* device [P], in/out: current tier -> new tier */
  uint8_t* free_map;       /* device [num_blocks], in/out: 1 = page free */
} mori_programs;

/* Per-tier capacity (Sec. 4.1: neither tier may exceed its memory). */
typedef struct {
  uint64_t gpu_bytes; /* <= num_blocks * block bytes */
  uint64_t cpu_bytes;
  uint32_t flags;     /* MORI_F_* */
  uint64_t ssd_bytes; /* read only with MORI_F_SSD_TIER */
} mori_budget;

/* The plan of the last mori_rank_partition, as mirrored on the host.  The
 * array pointers refer to context-owned pinned memory, valid until the next
 * mori_rank_partition or mori_destroy. */
typedef struct {
  uint32_t num_programs, m_gpu, m_cpu;
  uint32_t n_out, n_in, n_drop_gpu, n_drop_cpu, n_admit_gpu, n_admit_cpu;
  uint32_t device_error; /* MORI_DEV_* bits; 0 when the plan is valid */
  uint32_t m_ssd;        /* programs on the SSD tier (0 without MORI_F_SSD_TIER) */
  uint64_t pages_out, pages_in, pages_admit;
  uint64_t pages_free_before, pages_released, pages_recycled, pages_free_after;
  uint64_t bytes_out, bytes_in, gpu_bytes_after, cpu_bytes_after, ssd_bytes_after;
  uint64_t pages_dropped; /* released pages of idle programs dropped to Waiting (nothing uses them) */
  const uint32_t* order;        /* [P] program ids, busiest first (incremental: see below) */
  const uint64_t* prefix;       /* [P] inclusive KV-byte prefix in rank order */
  const uint8_t* tier_old;      /* [P] */
  const uint8_t* tier_new;      /* [P] */
  const uint8_t* category;      /* [P] MORI_CAT_* */
  const uint32_t* out_programs; /* [n_out] in rank order */
  const uint32_t* in_programs;  /* [n_in] in rank order */
} mori_plan;

/* ---- context ----------------------------------------------------------- */

/* Creates a context for one pool on the current HIP device.  max_programs <=
 * MORI_MAX_PROGRAMS bounds P of every later call.  staging_bytes is the
 * device staging of copy-engine swaps per direction (0: 512 MiB), used as two
 * halves of whole runs (it must hold at least two runs); copy-engine swaps
 * move the bytes in chunks of one half.  flags:
 *   MORI_CREATE_COPY_STREAMS  the context owns one copy stream per direction,
 *     so the copy engines drain one staging half while the gather/scatter
 *     kernel works on the other.  HIP maps a process's streams onto
 *     GPU_MAX_HW_QUEUES hardware queues (4 by default, read when HIP starts)
 *     and streams beyond that share queues, where one stream's waits block
 *     the other's work and the two swap directions serialise; set the flag
 *     only when the process has at least 8 queues (the two swap streams, the
 *     two copy streams).  Without it the copies run on the caller's stream,
 *     in order with the kernels.
 * The two streams given to the swaps should be distinct and created early
 * (streams beyond the queue count share queues).  *out is set on success.
 * EINVAL: null pool/out, unknown flags, bad geometry or alignment; EHIP:
 * allocation. */
#define MORI_CREATE_COPY_STREAMS 1u
int mori_create(const mori_pool* pool, uint32_t max_programs, uint64_t staging_bytes, uint32_t flags,
                mori_ctx** out);

/* Waits for the context's outstanding work and frees it.  NULL is a no-op. */
int mori_destroy(mori_ctx* ctx);

/* Registers a range that swap buffers may live in: pinned host memory from
 * hipHostMalloc / mori_host_alloc (used through its device mapping), or
 * device memory (then swaps are device-to-device gathers and scatters).  The
 * swap kernels touch no address outside registered ranges.  EINVAL: null,
 * zero size, or memory HIP does not know; ENOSPC: MORI_MAX_RANGES reached. */
int mori_register(mori_ctx* ctx, void* ptr, uint64_t bytes);

/* Pinned, device-mapped host memory for the CPU tier (hipHostMalloc with the
 * mapped and portable flags), and its release. */
int mori_host_alloc(uint64_t bytes, void** out);
int mori_host_free(void* ptr);

/* ---- the hot path ------------------------------------------------------ */

/* Computes the new placement and rewrites tbl, tier and free_map in stream
 * order.  Waits (on the stream) for the previous plan's swaps.  The plan is
 * stored into the context's pinned host mirror by the kernels; read it with
 * mori_plan_wait.
 *
 * Pages for programs entering the GPU are handed out in this order: pages
 * free before the step; then pages of programs dropped to Waiting that
 * nothing uses any more; then, together, pages of swapped-out programs (free
 * once the swap-out has read them) and pages of programs dropped while they
 * may still be running an inference step (free once that step has ended);
 * each group in ascending page id.  A dropped program counts as running when
 * the plan reads statuses (MORI_F_STATUS_KEY or MORI_F_INCREMENTAL) and its
 * status is not MORI_ST_ACTING (Sec. 4.3.1 demotes a Reasoning victim lazily:
 * its current step is not interrupted); without statuses the caller vouches
 * that dropped programs are idle.  The caller orders such a program's current
 * step before mori_kv_swap_out on the swap-out stream.  Programs promoted
 * from a lower tier take the pages first, then programs admitted from
 * Waiting, each group in rank order, blocks in logical order.  A slot at or
 * past pages_free_before + pages_dropped is on a page still in use: the
 * swap-in waits for the swap-out stream before writing it, and the caller
 * (MORI_Q_OUT_EVENT) before prefilling it.
 *
 * Default policy (Sec. 4.3, Sec. 7.2): rank all programs by idleness (Eq. 1),
 * busiest first, and fill the GPU tier, then the CPU tier, from the busiest
 * end; a program moves only when it crosses a boundary.
 *
 * MORI_F_INCREMENTAL (Sec. 4.3.1; status required): tiers change only to
 * repair a capacity violation or to fill free GPU room.  (1) While the CPU
 * tier exceeds its budget, its programs go to Waiting in demotion order
 * (Acting before Reasoning, highest idleness first, ties highest id first).
 * (2) While the GPU tier exceeds its budget, the next program in demotion
 * order leaves it, to the CPU tier if it fits in the CPU room left, else to
 * Waiting; a Reasoning victim is demoted lazily: the caller lets its current
 * inference step finish (orders it before the swap-out on the swap-out
 * stream), and its pages are handed out only after that (see above).
 * (3) The GPU room left is filled from, in order: CPU programs waiting for
 * inference, returning Waiting programs waiting for inference, new arrivals
 * smallest context first; lowest idleness first within a level, ties lowest
 * id.  Programs moved by (1)-(2) and Acting programs are no candidates; the
 * walk stops at the first candidate that does not fit (MORI_F_SKIP_FIT:
 * skips it).  Waiting programs are never placed on the CPU tier.  plan.order
 * then lists programs by old tier -- GPU, CPU, then Waiting as returning,
 * new (by context size), Acting -- each group by (Reasoning before Acting,
 * idleness, id) or, for new arrivals, (context size, idleness, id); m_gpu and
 * m_cpu count the programs on each tier afterwards.  A new arrival must have
 * fewer than 2^31 blocks (MORI_DEV_BAD_TBL_OFF otherwise).
 *
 * MORI_F_SSD_TIER (Sec. 7.1, boundary policy only): tier 3 is valid and the
 * ranking gets a third run -- after the CPU tier's, the longest run within
 * ssd_bytes goes to the SSD tier (skip-fit: the first of GPU, CPU, SSD with
 * room).  An SSD program owns no page; its KV is the caller's, in storage.
 * A program leaving the GPU for the SSD tier is swapped out like one going to
 * the CPU tier (into a host buffer the caller then writes to storage), and one
 * coming back is swapped in from a host buffer the caller has filled; page
 * slots go to every swapped-in program (from CPU or SSD) in rank order.
 *
 * A new plan supersedes the last one.  It waits (on the stream) for the last
 * plan's swaps that were enqueued; swaps that were not are abandoned, and the
 * tables, tiers and free map stand as that plan wrote them -- programs it sent
 * off the GPU then have no copy of their KV (placement-only use).
 *
 * EINVAL: null pointers (status with MORI_F_STATUS_KEY or MORI_F_INCREMENTAL),
 * window_k out of range, unknown flags, MORI_F_SSD_TIER with
 * MORI_F_INCREMENTAL, gpu_bytes > num_blocks * block bytes.  ENOSPC: P above
 * the context's max_programs.  Both are raised before anything is enqueued. */
int mori_rank_partition(mori_ctx* ctx, const mori_programs* programs, const mori_budget* budget,
                        void* stream);

/* Blocks the host until the last plan is on the host and fills *out.
 * Returns MORI_EDEVICE (with out->device_error set) if the plan was rejected
 * on the device, ESTATE if there is no plan. */
int mori_plan_wait(mori_ctx* ctx, mori_plan* out);

/* Swap-out of the last plan: for every program p with category OUT, copies
 * each run (plane q, logical block i) from its old page to
 * host_dst[p] + (q * nblk_p + i) * run_bytes.  host_dst is a host array of P
 * addresses (read during the call; entries of other programs are ignored),
 * each 16-B aligned inside a registered range with room for nblk_p * block
 * bytes.  Pages released by these programs may be reused only after this
 * swap completes.  ESTATE: no plan, or swap-out already enqueued for it. */
int mori_kv_swap_out(mori_ctx* ctx, const uint64_t* host_dst, uint32_t mode, void* stream);

/* Swap-in of the last plan: for every program p with category IN, copies
 * host_src[p] + (q * nblk_p + i) * run_bytes into its newly allocated page of
 * block i, plane q.  Waits (on the stream) for the plan and, before writing a
 * page that is still in use (the swap-out of the same plan reads it, or a
 * dropped program's step ordered before that swap-out uses it), for that
 * swap-out (pages free before the step and pages of idle dropped programs
 * need no wait).  The host buffers may be reused after it completes.  ESTATE: no plan, swap-in already
 * enqueued, or swap-out of the plan not yet enqueued. */
int mori_kv_swap_in(mori_ctx* ctx, const uint64_t* host_src, uint32_t mode, void* stream);

/* ---- introspection ----------------------------------------------------- */
#define MORI_Q_LAST_HIP_ERROR 1 /* last hipError_t seen by the context */
#define MORI_Q_DEVICE_ERROR 2   /* device error word of the last plan and swaps (waits for them) */
#define MORI_Q_LAST_MODE 3      /* copy mode actually used by the last swap */
#define MORI_Q_PLAN_EVENT 4     /* hipEvent_t recorded when the plan is complete */
#define MORI_Q_OUT_EVENT 5      /* hipEvent_t recorded when the last swap-out is complete */
#define MORI_Q_IN_EVENT 6       /* hipEvent_t recorded when the last swap-in is complete */
int mori_query(mori_ctx* ctx, int what, uint64_t* value);

/* Static description of a return code. */
const char* mori_strerror(int code);

/* ---- typed eviction order (Sec. 4.3.2) -------------------------------------- */
/* The engine-side companion of the placement: every KV block carries the type
 * label of its program -- busy (GPU queue), idle (CPU queue), inactive
 * (Waiting) -- and its last access time.  A tier evicts by type first, in
 * tier-reversed order (GPU: inactive, idle, busy; CPU: inactive, busy, idle),
 * least recently used first within a type, so each tier keeps the programs
 * the placement assigned to it.  Equal type and time: lowest block id first. */
#define MORI_TYPE_BUSY 0u
#define MORI_TYPE_IDLE 1u
#define MORI_TYPE_INACTIVE 2u

typedef struct {
  uint32_t num_blocks;          /* N */
  const uint8_t* type;          /* device [N] MORI_TYPE_* */
  const uint64_t* last_access;  /* device [N] access times, larger = more recent, < 2^62 */
  const uint32_t* size;         /* device [N] block sizes in units of unit_bytes, or NULL: one unit each */
  uint64_t unit_bytes;
} mori_blocks;

/* Bytes of device workspace mori_evict_order needs for num_blocks blocks
 * (about 36 bytes per block, plus 1 MiB). */
int mori_evict_workspace(uint32_t num_blocks, uint64_t* bytes);

/* Eviction order of one tier (MORI_TIER_GPU or MORI_TIER_CPU), enqueued on
 * `stream`: order[j] (device [N]) = block evicted j-th; prefix[j] (device [N],
 * may be NULL) = bytes freed by the first j+1 evictions; result (device [2]) =
 * {fewest evictions that free at least need_bytes (N if all of them free
 * less, 0 when need_bytes is 0), MORI_DEV_* error bits}.  workspace: device
 * memory of at least mori_evict_workspace bytes, 256-B aligned, owned by the
 * caller and used only while the call's work runs.  Nothing is allocated.
 * EINVAL: null pointers, misaligned or short workspace, bad tier. */
int mori_evict_order(const mori_blocks* blocks, uint32_t tier, uint64_t need_bytes, void* workspace,
                     uint64_t workspace_bytes, uint32_t* order, uint64_t* prefix, uint32_t* result,
                     void* stream);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, serving loops that forbid allocation): mori_evict_order with the
 * workspace in a device array the library holds on each GPU for the life of
 * the process, instead of a caller buffer.  Same result for the same input;
 * at most MORI_EVICT_NOALLOC_MAX_BLOCKS blocks (ENOSPC above; the array is
 * about 19.5 MiB per GPU).  Nothing is allocated: the array's device address
 * is looked up on the first call on each GPU (call it once before a capture
 * starts), and each call enqueues kernels only, which clear what must start
 * at zero.  Every call on one GPU uses the same array: calls whose work
 * overlaps on one GPU (other streams, other host threads) race and give
 * wrong results, so the caller serialises them, e.g. on one stream.
 * EINVAL: null pointers, bad tier; EHIP: the address lookup failed. */
#define MORI_EVICT_NOALLOC_MAX_BLOCKS 524288u /* 2^19 */
int mori_evict_order_noalloc(const mori_blocks* blocks, uint32_t tier, uint64_t need_bytes, uint32_t* order,
                             uint64_t* prefix, uint32_t* result, void* stream);

/* ---- kernel timing ------------------------------------------------------ */
/* With profiling on, every gather/scatter kernel launch of the swaps is
 * bracketed by timing events recorded on the stream it is launched on (up to
 * 4096 launches per direction between reads).  mori_profile_read waits for
 * those events and returns, for direction 0 (swap-out) or 1 (swap-in), the
 * number of launches, the payload bytes they moved and their summed duration
 * in milliseconds, then clears the record.  EINVAL: null pointers or a bad
 * direction; ENOSPC (from a swap) is never raised: launches beyond the record
 * capacity are simply not timed. */
int mori_profile(mori_ctx* ctx, int enable);
int mori_profile_read(mori_ctx* ctx, int direction, uint64_t* launches, uint64_t* payload_bytes,
                      double* kernel_ms);

/* ---- multi-replica admission (host) ----------------------------------- */
#define MORI_MAX_REPLICAS 1024u
#define MORI_ADMIT_BEST_FIT 1u /* least room that holds the program, instead of the most */

/* Admission of the Waiting queue that all replicas share (Sec. 4.1: a GPU and
 * a CPU queue per replica, one global Waiting queue; Sec. 4.3.1: Waiting
 * promotions are bin-packed across replicas in decreasing size onto the
 * replica with the most available capacity, while CPU-tier programs keep their
 * replica -- each replica's own mori_rank_partition promotes those).  Host
 * memory only; no GPU work.
 *   bytes[P], idleness[P], status[P]: the Waiting programs' KV bytes, Eq. 1
 *     idleness in [0, 1] and MORI_ST_* status.  Candidates are the Reasoning
 *     (returning) programs, then the new arrivals; Acting programs stay.
 *     Within a level: larger KV first, then lower idleness, then lower index.
 *   room[R]: free GPU bytes of each replica after its own plan.
 *   flags: 0 or MORI_ADMIT_BEST_FIT.
 *   replica[P] (out): the replica each program goes to, -1 if it stays
 *     waiting (it fits no replica when its turn comes; later ones are tried).
 *   room_after[R] (out; may be room itself): room less what was admitted.
 * Ties between replicas go to the lower index.  Each replica then admits its
 * programs as Waiting->GPU in its next plan (prefill rebuilds their KV).
 * EINVAL: num_replicas 0 or above MORI_MAX_REPLICAS, null arrays, unknown
 * flags, a status above 2 or idleness outside [0, 1]. */
int mori_replica_admit(uint32_t num_programs, const uint64_t* bytes, const float* idleness, const uint8_t* status,
                       uint32_t num_replicas, const uint64_t* room, uint32_t flags, int32_t* replica,
                       uint64_t* room_after);

#ifdef __cplusplus
}
#endif
#endif /* MORI_H */
