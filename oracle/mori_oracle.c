/*
 * mori_oracle.c -- plain CPU oracle for MORI's idleness-ranked KV tier placement
 * (arXiv 2606.00866).  TEST INFRASTRUCTURE ONLY: used by the tests, the smoke
 * check and the benchmark's CPU-baseline leg, never by the product path.
 *
 * Deliberately simple: whole-array loops in the order the paper describes the
 * method, a library sort, memcpy per KV run.  No blocking, fusion or
 * reordering beyond what the definitions state.  Readings of points the paper
 * leaves open are marked "Reading:".
 */
#include "mori_oracle.h"

#include <math.h>
#include <stdlib.h>
#include <string.h>

/* ------------------------------------------------------------------------ */
/* Step 1 -- idleness, Eq. 1 (Sec. 4.2 "Idleness Metric").                   */
/*   iota = T_acting / (T_reasoning + T_acting), both totals over the last k   */
/*   reasoning/tool-call cycles, the ongoing call's elapsed time included.     */
/* Reading: binary32 throughout; each total is accumulated oldest cycle first */
/* starting from +0; a program with no recorded time (denominator 0) gets     */
/* idleness 0; a zero result is +0.  Inputs must be finite and >= 0 and the    */
/* totals must stay finite, otherwise the program data is rejected.          */
/* ------------------------------------------------------------------------ */
int orc_idleness(uint32_t P, uint32_t k, const float* window, float* iota) {
  for (uint32_t p = 0; p < P; ++p) {
    float t_reasoning = 0.0f;
    float t_acting = 0.0f;
    for (uint32_t j = 0; j < k; ++j) {
      float r = window[((size_t)p * k + j) * 2 + 0];
      float a = window[((size_t)p * k + j) * 2 + 1];
      if (!(r >= 0.0f) || !(a >= 0.0f) || isinf(r) || isinf(a)) return ORC_E_INPUT;
      t_reasoning = t_reasoning + r;
      t_acting = t_acting + a;
    }
    float total = t_reasoning + t_acting;
    if (isinf(t_reasoning) || isinf(t_acting) || isinf(total)) return ORC_E_INPUT;
    float value = (total > 0.0f) ? t_acting / total : 0.0f;
    if (value == 0.0f) value = 0.0f; /* drop the sign of a negative zero */
    iota[p] = value;
  }
  return ORC_OK;
}

/* ------------------------------------------------------------------------ */
/* Ranking key.  Programs are ranked busiest (lowest idleness) first.        */
/* Reading: the key is the binary32 bit pattern of idleness, which orders    */
/* like the value because idleness lies in [0, 1].  With ORC_F_STATUS_KEY an */
/* Acting program (status 1) is placed after every Reasoning program, since  */
/* Acting programs are demoted first (Sec. 4.3.1, demotion from GPU).        */
/* ------------------------------------------------------------------------ */
int orc_keys(uint32_t P, const float* iota, const uint8_t* status, uint32_t flags, uint32_t* key) {
  for (uint32_t p = 0; p < P; ++p) {
    float v = iota[p];
    if (!(v >= 0.0f && v <= 1.0f)) return ORC_E_INPUT;
    if (v == 0.0f) v = 0.0f;
    uint32_t bits;
    memcpy(&bits, &v, sizeof bits);
    if ((flags & ORC_F_STATUS_KEY) && status != NULL && status[p] == 1) bits |= 0x80000000u;
    key[p] = bits;
  }
  return ORC_OK;
}

/* ------------------------------------------------------------------------ */
/* Relative ranking (Sec. 1, Sec. 4.3): order all programs by key.          */
/* Reading: ties go to the lower program id, i.e. the sort is on the pair    */
/* (key, id), which is a total order.                                        */
/* ------------------------------------------------------------------------ */
typedef struct {
  uint32_t key, id;
} orc_pair;

static int orc_pair_cmp(const void* a, const void* b) {
  const orc_pair* x = (const orc_pair*)a;
  const orc_pair* y = (const orc_pair*)b;
  if (x->key != y->key) return x->key < y->key ? -1 : 1;
  if (x->id != y->id) return x->id < y->id ? -1 : 1;
  return 0;
}

void orc_order(uint32_t P, const uint32_t* key, uint32_t* order, uint32_t* rank) {
  orc_pair* pairs = (orc_pair*)malloc(sizeof(orc_pair) * (P ? P : 1));
  for (uint32_t p = 0; p < P; ++p) {
    pairs[p].key = key[p];
    pairs[p].id = p;
  }
  qsort(pairs, P, sizeof(orc_pair), orc_pair_cmp);
  for (uint32_t r = 0; r < P; ++r) {
    order[r] = pairs[r].id;
    if (rank) rank[pairs[r].id] = r;
  }
  free(pairs);
}

/* ------------------------------------------------------------------------ */
/* Capacity-matched boundary (Sec. 1; Sec. 4.1 three-tier queues and their   */
/* capacity invariants; Sec. 7.2: fill from the busiest end of the ranking   */
/* until capacity is reached).                                               */
/* Reading: a program is placed whole (never split across tiers) with       */
/* ceil(context/tokens-per-block) blocks; the boundary is a strict prefix of */
/* the ranking: the GPU tier takes the longest prefix whose bytes do not     */
/* exceed the GPU budget, the CPU tier the longest following run that does   */
/* not exceed the CPU budget, the rest go to Waiting.  ORC_F_SKIP_FIT walks  */
/* the ranking once and puts each program in the first tier it still fits.  */
/* ------------------------------------------------------------------------ */
void orc_boundary(uint32_t P, const uint32_t* order, const uint32_t* nblk, uint64_t block_bytes,
                  uint64_t gpu_budget, uint64_t cpu_budget, uint64_t ssd_budget, uint32_t flags,
                  uint64_t* prefix, uint8_t* tier_new, uint32_t* m_gpu, uint32_t* m_cpu, uint32_t* m_ssd) {
  const int ssd = (flags & ORC_F_SSD_TIER) != 0;
  uint64_t running = 0;
  for (uint32_t r = 0; r < P; ++r) {
    running += (uint64_t)nblk[order[r]] * block_bytes;
    prefix[r] = running;
  }
  uint32_t n_gpu = 0, n_cpu = 0, n_ssd = 0;
  if (flags & ORC_F_SKIP_FIT) {
    uint64_t room_gpu = gpu_budget, room_cpu = cpu_budget, room_ssd = ssd_budget;
    for (uint32_t r = 0; r < P; ++r) {
      uint32_t p = order[r];
      uint64_t bytes = (uint64_t)nblk[p] * block_bytes;
      if (bytes <= room_gpu) {
        room_gpu -= bytes;
        tier_new[p] = ORC_GPU;
        ++n_gpu;
      } else if (bytes <= room_cpu) {
        room_cpu -= bytes;
        tier_new[p] = ORC_CPU;
        ++n_cpu;
      } else if (ssd && bytes <= room_ssd) {
        room_ssd -= bytes;
        tier_new[p] = ORC_SSD;
        ++n_ssd;
      } else {
        tier_new[p] = ORC_WAIT;
      }
    }
  } else {
    while (n_gpu < P && prefix[n_gpu] <= gpu_budget) ++n_gpu;
    uint64_t gpu_part = n_gpu ? prefix[n_gpu - 1] : 0;
    while (n_gpu + n_cpu < P && prefix[n_gpu + n_cpu] - gpu_part <= cpu_budget) ++n_cpu;
    if (ssd) { /* Sec. 7.1: the programs between the second and a third threshold go to SSD */
      uint64_t upper_part = (n_gpu + n_cpu) ? prefix[n_gpu + n_cpu - 1] : 0;
      while (n_gpu + n_cpu + n_ssd < P && prefix[n_gpu + n_cpu + n_ssd] - upper_part <= ssd_budget) ++n_ssd;
    }
    for (uint32_t r = 0; r < P; ++r) {
      uint32_t p = order[r];
      tier_new[p] = (r < n_gpu) ? ORC_GPU
                  : (r < n_gpu + n_cpu) ? ORC_CPU
                  : (r < n_gpu + n_cpu + n_ssd) ? ORC_SSD : ORC_WAIT;
    }
  }
  *m_gpu = n_gpu;
  *m_cpu = n_cpu;
  *m_ssd = n_ssd;
}

/* Transition category, old tier -> new tier.  Leaving the GPU for a lower
   tier that keeps the KV (CPU, SSD) is a swap-out, the reverse a swap-in. */
static uint8_t orc_category(uint8_t from, uint8_t to) {
  static const uint8_t table[4][4] = {
      /* to:           GPU            CPU            WAIT           SSD */
      /* GPU  */ {ORC_KEPT, ORC_OUT, ORC_DROP_GPU, ORC_OUT},
      /* CPU  */ {ORC_IN, ORC_KEPT, ORC_DROP_CPU, ORC_CPU_SSD},
      /* WAIT */ {ORC_ADMIT_GPU, ORC_ADMIT_CPU, ORC_KEPT, ORC_ADMIT_SSD},
      /* SSD  */ {ORC_IN, ORC_SSD_CPU, ORC_DROP_SSD, ORC_KEPT},
  };
  return table[from][to];
}

/* ------------------------------------------------------------------------ */
/* Incremental sticky placement (Sec. 4.3 "sticky placement"; Sec. 4.3.1     */
/* demotion from GPU and promotion to GPU).  Written as the loops the paper  */
/* describes: pick the next victim while a tier is over budget, then promote */
/* while the next candidate fits.                                            */
/* Readings: programs of equal status and idleness are demoted highest id    */
/* first and promoted lowest id first (the reverse of each other, as in the  */
/* ranking); the CPU tier is brought within its budget before the GPU's      */
/* victims are placed; each victim goes to the CPU tier if it fits in what   */
/* is left there (the paper's per-program rule); promotion stops at the      */
/* first candidate that does not fit so that no lower-priority program       */
/* overtakes it (ORC_F_SKIP_FIT skips it instead); a program moved by this   */
/* step is not promoted again in it; a new arrival found outside Waiting     */
/* counts as Reasoning; Waiting programs are never placed on the CPU tier    */
/* (their KV is rebuilt by prefill on the GPU).                              */
/* ------------------------------------------------------------------------ */
static int orc_is_acting(const uint8_t* status, uint32_t p) { return status[p] == ORC_ST_ACTING; }

/* nonzero when program x is demoted before program y */
static int orc_demote_before(const float* iota, const uint8_t* status, uint32_t x, uint32_t y) {
  int ax = orc_is_acting(status, x), ay = orc_is_acting(status, y);
  if (ax != ay) return ax; /* Acting (KV idle on the GPU) before Reasoning */
  if (iota[x] != iota[y]) return iota[x] > iota[y];
  return x > y;
}

/* promotion level of a candidate: 0 CPU tier, 1 returning Waiting, 2 new arrival */
static uint32_t orc_promote_level(const uint8_t* status, const uint8_t* tier_old, uint32_t p) {
  if (tier_old[p] == ORC_CPU) return 0;
  return status[p] == ORC_ST_NEW ? 2 : 1;
}

/* comparison context for qsort, one per thread so concurrent calls are safe */
static _Thread_local const float* orc_sort_iota;
static _Thread_local const uint8_t* orc_sort_status;
static _Thread_local const uint8_t* orc_sort_tier;
static _Thread_local const uint32_t* orc_sort_nblk;

static int orc_promote_cmp(const void* a, const void* b) {
  uint32_t x = *(const uint32_t*)a, y = *(const uint32_t*)b;
  uint32_t lx = orc_promote_level(orc_sort_status, orc_sort_tier, x);
  uint32_t ly = orc_promote_level(orc_sort_status, orc_sort_tier, y);
  if (lx != ly) return lx < ly ? -1 : 1;
  if (lx == 2 && orc_sort_nblk[x] != orc_sort_nblk[y]) return orc_sort_nblk[x] < orc_sort_nblk[y] ? -1 : 1;
  if (orc_sort_iota[x] != orc_sort_iota[y]) return orc_sort_iota[x] < orc_sort_iota[y] ? -1 : 1;
  return x < y ? -1 : (x > y);
}

/* listing group of a program: 0 GPU, 1 CPU, 2 Waiting Reasoning, 3 Waiting new, 4 Waiting Acting */
static uint32_t orc_list_group(uint32_t p) {
  if (orc_sort_tier[p] == ORC_GPU) return 0;
  if (orc_sort_tier[p] == ORC_CPU) return 1;
  if (orc_sort_status[p] == ORC_ST_ACTING) return 4;
  return orc_sort_status[p] == ORC_ST_NEW ? 3 : 2;
}

static int orc_list_cmp(const void* a, const void* b) {
  uint32_t x = *(const uint32_t*)a, y = *(const uint32_t*)b;
  uint32_t gx = orc_list_group(x), gy = orc_list_group(y);
  if (gx != gy) return gx < gy ? -1 : 1;
  if (gx <= 1) { /* the reverse of the demotion order */
    if (x == y) return 0;
    return orc_demote_before(orc_sort_iota, orc_sort_status, x, y) ? 1 : -1;
  }
  if (gx == 3 && orc_sort_nblk[x] != orc_sort_nblk[y]) return orc_sort_nblk[x] < orc_sort_nblk[y] ? -1 : 1;
  if (orc_sort_iota[x] != orc_sort_iota[y]) return orc_sort_iota[x] < orc_sort_iota[y] ? -1 : 1;
  return x < y ? -1 : (x > y);
}

int orc_incremental(uint32_t P, const float* iota_in, const uint8_t* status, const uint8_t* tier_old,
                    const uint32_t* nblk, uint64_t block_bytes, uint64_t gpu_budget, uint64_t cpu_budget,
                    uint32_t flags, uint32_t* order, uint32_t* rank, uint64_t* prefix, uint8_t* tier_new,
                    uint32_t* m_gpu, uint32_t* m_cpu) {
  const size_t np = P ? P : 1;
  float* iota = (float*)malloc(sizeof(float) * np);
  for (uint32_t p = 0; p < P; ++p) {
    float v = iota_in[p];
    if (!(v >= 0.0f && v <= 1.0f) || status[p] > ORC_ST_NEW ||
        (tier_old[p] == ORC_WAIT && status[p] == ORC_ST_NEW && nblk[p] >= 0x80000000u)) {
      free(iota);
      return ORC_E_INPUT;
    }
    iota[p] = (v == 0.0f) ? 0.0f : v;
  }
  uint8_t* moved = (uint8_t*)calloc(np, 1);
  uint32_t* cand = (uint32_t*)malloc(sizeof(uint32_t) * np);
  uint64_t used_gpu = 0, used_cpu = 0;
  for (uint32_t p = 0; p < P; ++p) {
    tier_new[p] = tier_old[p];
    uint64_t bytes = (uint64_t)nblk[p] * block_bytes;
    if (tier_old[p] == ORC_GPU) used_gpu += bytes;
    if (tier_old[p] == ORC_CPU) used_cpu += bytes;
  }

  /* 1. CPU admission control */
  while (used_cpu > cpu_budget) {
    uint32_t v = P;
    for (uint32_t p = 0; p < P; ++p)
      if (tier_new[p] == ORC_CPU && tier_old[p] == ORC_CPU && !moved[p] &&
          (v == P || orc_demote_before(iota, status, p, v)))
        v = p;
    tier_new[v] = ORC_WAIT;
    moved[v] = 1;
    used_cpu -= (uint64_t)nblk[v] * block_bytes;
  }

  /* 2. demotion from GPU */
  while (used_gpu > gpu_budget) {
    uint32_t v = P;
    for (uint32_t p = 0; p < P; ++p)
      if (tier_new[p] == ORC_GPU && (v == P || orc_demote_before(iota, status, p, v))) v = p;
    uint64_t bytes = (uint64_t)nblk[v] * block_bytes;
    used_gpu -= bytes;
    moved[v] = 1;
    if (bytes <= cpu_budget - used_cpu) {
      tier_new[v] = ORC_CPU;
      used_cpu += bytes;
    } else {
      tier_new[v] = ORC_WAIT;
    }
  }

  /* 3. promotion to GPU */
  uint32_t nc = 0;
  for (uint32_t p = 0; p < P; ++p)
    if (!moved[p] && tier_old[p] != ORC_GPU && status[p] != ORC_ST_ACTING) cand[nc++] = p;
  orc_sort_iota = iota;
  orc_sort_status = status;
  orc_sort_tier = tier_old;
  orc_sort_nblk = nblk;
  qsort(cand, nc, sizeof(uint32_t), orc_promote_cmp);
  uint64_t room = gpu_budget - used_gpu;
  for (uint32_t j = 0; j < nc; ++j) {
    uint32_t p = cand[j];
    uint64_t bytes = (uint64_t)nblk[p] * block_bytes;
    if (bytes <= room) {
      room -= bytes;
      tier_new[p] = ORC_GPU;
    } else if (!(flags & ORC_F_SKIP_FIT)) {
      break;
    }
  }

  /* the listing order and the byte prefix along it */
  for (uint32_t p = 0; p < P; ++p) order[p] = p;
  qsort(order, P, sizeof(uint32_t), orc_list_cmp);
  uint64_t running = 0;
  uint32_t ng = 0, nk = 0;
  for (uint32_t r = 0; r < P; ++r) {
    running += (uint64_t)nblk[order[r]] * block_bytes;
    prefix[r] = running;
    if (rank) rank[order[r]] = r;
  }
  for (uint32_t p = 0; p < P; ++p) {
    ng += tier_new[p] == ORC_GPU;
    nk += tier_new[p] == ORC_CPU;
  }
  *m_gpu = ng;
  *m_cpu = nk;
  free(iota);
  free(moved);
  free(cand);
  return ORC_OK;
}

/* ------------------------------------------------------------------------ */
/* One rebalance.                                                            */
/* ------------------------------------------------------------------------ */
int orc_rebalance(const orc_geometry* g, uint8_t* pool_bytes, uint32_t P, uint32_t k,
                  const float* window, const float* iota_given, const uint8_t* status,
                  const uint32_t* tbl_off, uint32_t tbl_len, uint32_t* tbl, uint8_t* tier,
                  uint8_t* free_map, uint64_t gpu_budget, uint64_t cpu_budget, uint64_t ssd_budget, uint32_t flags,
                  uint8_t* const* host_bufs, uint32_t* order_out, uint32_t* rank_out,
                  uint8_t* tier_old_out, uint8_t* category_out, uint64_t* prefix_out,
                  orc_summary* summary) {
  const uint32_t NB = g->num_blocks;
  const uint64_t planes = (uint64_t)g->layers * g->planes;
  const uint64_t run = (uint64_t)g->block_tokens * g->row_bytes; /* bytes of one (plane, page) */
  const uint64_t block_bytes = planes * run;                      /* bytes of one page, all planes */
  const size_t np = P ? P : 1;
  int rc = ORC_OK;

  float* iota = (float*)calloc(np, sizeof(float));
  uint32_t* key = (uint32_t*)malloc(sizeof(uint32_t) * np);
  uint32_t* order = (uint32_t*)malloc(sizeof(uint32_t) * np);
  uint32_t* rank = (uint32_t*)malloc(sizeof(uint32_t) * np);
  uint32_t* nblk = (uint32_t*)malloc(sizeof(uint32_t) * np);
  uint64_t* prefix = (uint64_t*)malloc(sizeof(uint64_t) * np);
  uint8_t* tier_new = (uint8_t*)malloc(np);
  uint8_t* cat = (uint8_t*)malloc(np);
  uint8_t* page_state = (uint8_t*)calloc(NB ? NB : 1, 1); /* bit0 free, bit1 owned, bit2 released, bit3 free only later */
  uint32_t* pages_avail = (uint32_t*)malloc(sizeof(uint32_t) * (NB ? NB : 1));
  uint32_t* new_tbl = NULL;

  /* -- program data: tiers and the block-table offsets -- */
  const uint8_t top_tier = (flags & ORC_F_SSD_TIER) ? ORC_SSD : ORC_WAIT;
  if ((flags & ORC_F_SSD_TIER) && (flags & ORC_F_INCREMENTAL)) rc = ORC_E_INPUT;
  for (uint32_t p = 0; p < P && rc == ORC_OK; ++p)
    if (tier[p] > top_tier) rc = ORC_E_INPUT;
  if (rc == ORC_OK && tbl_off[0] != 0) rc = ORC_E_INPUT;
  for (uint32_t p = 0; p < P && rc == ORC_OK; ++p) {
    if (tbl_off[p + 1] < tbl_off[p]) rc = ORC_E_INPUT;
    else nblk[p] = tbl_off[p + 1] - tbl_off[p];
  }
  if (rc == ORC_OK && tbl_off[P] > tbl_len) rc = ORC_E_INPUT;

  /* -- steps 1-3: idleness, ranking, boundary -- */
  if (rc == ORC_OK) {
    if (flags & ORC_F_IDLENESS_GIVEN) {
      for (uint32_t p = 0; p < P; ++p) iota[p] = iota_given[p];
    } else {
      rc = orc_idleness(P, k, window, iota);
    }
  }
  uint32_t m_gpu = 0, m_cpu = 0, m_ssd = 0;
  if (rc == ORC_OK && (flags & ORC_F_INCREMENTAL)) {
    if (status == NULL && P) rc = ORC_E_INPUT;
    else rc = orc_incremental(P, iota, status, tier, nblk, block_bytes, gpu_budget, cpu_budget, flags, order,
                              rank, prefix, tier_new, &m_gpu, &m_cpu);
  } else if (rc == ORC_OK) {
    rc = orc_keys(P, iota, status, flags, key);
    if (rc == ORC_OK) {
      orc_order(P, key, order, rank);
      orc_boundary(P, order, nblk, block_bytes, gpu_budget, cpu_budget, ssd_budget, flags, prefix, tier_new,
                   &m_gpu, &m_cpu, &m_ssd);
    }
  }
  if (rc == ORC_OK)
    for (uint32_t p = 0; p < P; ++p) cat[p] = orc_category(tier[p], tier_new[p]);

  /* -- which programs dropped from the GPU may still be using their pages.
        Reading (Sec. 4.3.1, lazy demotion): a Reasoning victim is not
        interrupted; its current inference step ends first, so its pages are
        not free at once.  When the plan reads statuses (ORC_F_STATUS_KEY or
        ORC_F_INCREMENTAL), every status other than Acting counts as running
        (a new arrival found on the GPU counts as Reasoning); without
        statuses the caller vouches that dropped programs are idle. -- */
  uint8_t* may_run = (uint8_t*)calloc(np, 1);
  if (rc == ORC_OK && status != NULL && (flags & (ORC_F_STATUS_KEY | ORC_F_INCREMENTAL)))
    for (uint32_t p = 0; p < P; ++p) may_run[p] = status[p] != ORC_ST_ACTING;

  /* -- pool consistency: every page is either free or owned by exactly one
        GPU-resident program; non-resident programs hold no page -- */
  if (rc == ORC_OK) {
    for (uint32_t pg = 0; pg < NB; ++pg)
      if (free_map[pg]) page_state[pg] |= 1u;
    for (uint32_t p = 0; p < P && rc == ORC_OK; ++p) {
      for (uint32_t i = 0; i < nblk[p] && rc == ORC_OK; ++i) {
        uint32_t pg = tbl[tbl_off[p] + i];
        if (tier[p] != ORC_GPU) {
          if (pg != ORC_NONE) rc = ORC_E_POOL;
          continue;
        }
        if (pg >= NB || (page_state[pg] & 3u)) {
          rc = ORC_E_POOL;
          continue;
        }
        page_state[pg] |= 2u;
        if (cat[p] == ORC_DROP_GPU && !may_run[p]) page_state[pg] |= 4u; /* released, nothing reads it */
        if (cat[p] == ORC_DROP_GPU && may_run[p]) page_state[pg] |= 4u | 8u; /* free once its step ended */
        if (cat[p] == ORC_OUT) page_state[pg] |= 4u | 8u;      /* released once the swap-out read it */
      }
    }
    for (uint32_t pg = 0; pg < NB && rc == ORC_OK; ++pg)
      if (!(page_state[pg] & 3u)) rc = ORC_E_POOL;
  }
  if (rc == ORC_OK && pool_bytes && host_bufs) {
    for (uint32_t p = 0; p < P && rc == ORC_OK; ++p)
      if ((cat[p] == ORC_OUT || cat[p] == ORC_IN) && nblk[p] && host_bufs[p] == NULL) rc = ORC_E_INPUT;
  }

  /* -- step 4: page allocation (Reading: pages free before this step in
        ascending id order, then the pages of programs dropped from the GPU to
        Waiting that nothing reads any more, then the pages that are free only
        later -- those of programs swapped out (once the swap-out has read
        them) and those of dropped programs that may still be running (once
        their step has ended) -- together in ascending id order; they are
        handed out first to the programs promoted from a lower tier, then to
        those admitted from Waiting, following the promotion priority of
        Sec. 4.3.1, each group in rank order, each program's blocks in logical
        order) -- */
  uint64_t n_free0 = 0, n_rel = 0, n_drop = 0, need = 0;
  if (rc == ORC_OK) {
    for (uint32_t pg = 0; pg < NB; ++pg)
      if (page_state[pg] & 1u) pages_avail[n_free0++] = pg;
    for (uint32_t pg = 0; pg < NB; ++pg)
      if ((page_state[pg] & 4u) && !(page_state[pg] & 8u)) pages_avail[n_free0 + n_rel++] = pg;
    n_drop = n_rel;
    for (uint32_t pg = 0; pg < NB; ++pg)
      if (page_state[pg] & 8u) pages_avail[n_free0 + n_rel++] = pg;
    for (uint32_t p = 0; p < P; ++p)
      if (cat[p] == ORC_IN || cat[p] == ORC_ADMIT_GPU) need += nblk[p];
    if (need > n_free0 + n_rel) rc = ORC_E_NOSPC;
  }

  if (rc == ORC_OK) {
    /* -- step 5a: swap-out, reading the tables as they were before this step -- */
    if (pool_bytes && host_bufs) {
      for (uint32_t p = 0; p < P; ++p) {
        if (cat[p] != ORC_OUT) continue;
        for (uint64_t q = 0; q < planes; ++q)
          for (uint32_t i = 0; i < nblk[p]; ++i) {
            uint64_t page = tbl[tbl_off[p] + i];
            memcpy(host_bufs[p] + (q * nblk[p] + i) * run, pool_bytes + (q * NB + page) * run, run);
          }
      }
    }
    /* -- table rewrite and the free map after the step -- */
    new_tbl = (uint32_t*)malloc(sizeof(uint32_t) * (tbl_off[P] ? tbl_off[P] : 1));
    memcpy(new_tbl, tbl, sizeof(uint32_t) * tbl_off[P]);
    uint64_t slot = 0;
    for (int pass = 0; pass < 2; ++pass) {
      uint8_t want = pass == 0 ? ORC_IN : ORC_ADMIT_GPU;
      for (uint32_t r = 0; r < P; ++r) {
        uint32_t p = order[r];
        if (cat[p] != want) continue;
        for (uint32_t i = 0; i < nblk[p]; ++i) new_tbl[tbl_off[p] + i] = pages_avail[slot++];
      }
    }
    for (uint32_t p = 0; p < P; ++p)
      if (cat[p] == ORC_OUT || cat[p] == ORC_DROP_GPU)
        for (uint32_t i = 0; i < nblk[p]; ++i) new_tbl[tbl_off[p] + i] = ORC_NONE;
    for (uint64_t j = 0; j < n_free0 + n_rel; ++j) free_map[pages_avail[j]] = (j >= need) ? 1 : 0;
    memcpy(tbl, new_tbl, sizeof(uint32_t) * tbl_off[P]);

    /* -- step 5b: swap-in into the newly allocated pages -- */
    if (pool_bytes && host_bufs) {
      for (uint32_t p = 0; p < P; ++p) {
        if (cat[p] != ORC_IN) continue;
        for (uint64_t q = 0; q < planes; ++q)
          for (uint32_t i = 0; i < nblk[p]; ++i) {
            uint64_t page = tbl[tbl_off[p] + i];
            memcpy(pool_bytes + (q * NB + page) * run, host_bufs[p] + (q * nblk[p] + i) * run, run);
          }
      }
    }

    if (summary) {
      memset(summary, 0, sizeof *summary);
      summary->m_gpu = m_gpu;
      summary->m_cpu = m_cpu;
      summary->m_ssd = m_ssd;
      for (uint32_t p = 0; p < P; ++p) {
        uint64_t pages = nblk[p];
        switch (cat[p]) {
          case ORC_OUT: summary->n_out++; summary->pages_out += pages; break;
          case ORC_IN: summary->n_in++; summary->pages_in += pages; break;
          case ORC_DROP_GPU: summary->n_drop_gpu++; break;
          case ORC_DROP_CPU: summary->n_drop_cpu++; break;
          case ORC_ADMIT_GPU: summary->n_admit_gpu++; summary->pages_admit += pages; break;
          case ORC_ADMIT_CPU: summary->n_admit_cpu++; break;
          default: break;
        }
        if (tier_new[p] == ORC_GPU) summary->gpu_bytes_after += pages * block_bytes;
        if (tier_new[p] == ORC_CPU) summary->cpu_bytes_after += pages * block_bytes;
        if (tier_new[p] == ORC_SSD) summary->ssd_bytes_after += pages * block_bytes;
      }
      summary->pages_free_before = n_free0;
      summary->pages_released = n_rel;
      summary->pages_recycled = need > n_free0 ? need - n_free0 : 0;
      summary->pages_free_after = n_free0 + n_rel - need;
      summary->pages_dropped = n_drop;
      summary->bytes_out = summary->pages_out * block_bytes;
      summary->bytes_in = summary->pages_in * block_bytes;
    }
    if (tier_old_out) memcpy(tier_old_out, tier, P);
    if (category_out) memcpy(category_out, cat, P);
    if (order_out) memcpy(order_out, order, sizeof(uint32_t) * P);
    if (rank_out) memcpy(rank_out, rank, sizeof(uint32_t) * P);
    if (prefix_out) memcpy(prefix_out, prefix, sizeof(uint64_t) * P);
    memcpy(tier, tier_new, P);
  }

  free(iota);
  free(key);
  free(order);
  free(rank);
  free(nblk);
  free(prefix);
  free(tier_new);
  free(cat);
  free(page_state);
  free(may_run);
  free(pages_avail);
  free(new_tbl);
  return rc;
}

/* ------------------------------------------------------------------------ */
/* Typed eviction order (Sec. 4.3.2).                                         */
/* ------------------------------------------------------------------------ */
typedef struct {
  uint32_t rank_of_type; /* position of the block's type in the tier's eviction order */
  uint64_t time;
  uint32_t id;
} orc_victim;

static int orc_victim_cmp(const void* a, const void* b) {
  const orc_victim* x = (const orc_victim*)a;
  const orc_victim* y = (const orc_victim*)b;
  if (x->rank_of_type != y->rank_of_type) return x->rank_of_type < y->rank_of_type ? -1 : 1;
  if (x->time != y->time) return x->time < y->time ? -1 : 1; /* least recently used first */
  if (x->id != y->id) return x->id < y->id ? -1 : 1;
  return 0;
}

int orc_evict_order(uint32_t N, const uint8_t* type, const uint64_t* last_access, const uint32_t* size,
                    uint64_t unit_bytes, uint32_t tier, uint64_t need_bytes, uint32_t* order, uint64_t* prefix,
                    uint32_t* count) {
  /* tier-reversed type order: GPU evicts inactive, idle, busy; CPU evicts inactive, busy, idle */
  static const uint32_t gpu_rank[3] = {2, 1, 0}; /* indexed by type: busy, idle, inactive */
  static const uint32_t cpu_rank[3] = {1, 2, 0};
  if (tier != ORC_GPU && tier != ORC_CPU) return ORC_E_INPUT;
  const uint32_t* rank_of = tier == ORC_GPU ? gpu_rank : cpu_rank;
  for (uint32_t b = 0; b < N; ++b)
    if (type[b] > ORC_TYPE_INACTIVE) return ORC_E_INPUT;
  orc_victim* v = (orc_victim*)malloc(sizeof(orc_victim) * (N ? N : 1));
  for (uint32_t b = 0; b < N; ++b) {
    v[b].rank_of_type = rank_of[type[b]];
    v[b].time = last_access[b];
    v[b].id = b;
  }
  qsort(v, N, sizeof(orc_victim), orc_victim_cmp);
  uint64_t freed = 0;
  uint32_t m = N;
  int found = 0;
  for (uint32_t j = 0; j < N; ++j) {
    order[j] = v[j].id;
    freed += (uint64_t)(size ? size[v[j].id] : 1u) * unit_bytes;
    if (prefix) prefix[j] = freed;
    if (!found && freed >= need_bytes) {
      m = j + 1;
      found = 1;
    }
  }
  if (need_bytes == 0) m = 0;
  *count = m;
  free(v);
  return ORC_OK;
}

/* ------------------------------------------------------------------------ */
/* Multi-replica admission (Sec. 4.1 global Waiting queue; Sec. 4.3.1,        */
/* promotion to GPU, multi-replica deployments).                             */
/* Reading: the paper names Best-Fit-Decreasing but selects the replica with  */
/* the most available capacity; that stated selection is the default, the   */
/* textbook best fit (least sufficient room) is ORC_ADMIT_BEST_FIT.  The     */
/* single-replica level order is kept (returning before new) and each level  */
/* is taken in decreasing size, the "decreasing" of the packing.             */
/* ------------------------------------------------------------------------ */
/* nonzero when candidate x is packed before candidate y */
static int orc_pack_before(const uint64_t* bytes, const float* iota, const uint8_t* status, uint32_t x, uint32_t y) {
  uint32_t lx = status[x] == ORC_ST_NEW, ly = status[y] == ORC_ST_NEW;
  if (lx != ly) return lx < ly;
  if (bytes[x] != bytes[y]) return bytes[x] > bytes[y];
  if (iota[x] != iota[y]) return iota[x] < iota[y];
  return x < y;
}

int orc_replica_admit(uint32_t P, const uint64_t* bytes, const float* iota, const uint8_t* status, uint32_t R,
                      const uint64_t* room, uint32_t flags, int32_t* replica, uint64_t* room_after) {
  if (R == 0) return ORC_E_INPUT;
  for (uint32_t p = 0; p < P; ++p)
    if (status[p] > ORC_ST_NEW || !(iota[p] >= 0.0f && iota[p] <= 1.0f)) return ORC_E_INPUT;
  for (uint32_t r = 0; r < R; ++r) room_after[r] = room[r];
  uint8_t* done = (uint8_t*)calloc(P ? P : 1, 1);
  for (uint32_t p = 0; p < P; ++p) {
    replica[p] = -1;
    if (status[p] == ORC_ST_ACTING) done[p] = 1; /* in a tool call: no inference to admit */
  }
  for (;;) {
    /* the next candidate in packing order */
    uint32_t c = P;
    for (uint32_t p = 0; p < P; ++p)
      if (!done[p] && (c == P || orc_pack_before(bytes, iota, status, p, c))) c = p;
    if (c == P) break;
    done[c] = 1;
    /* the replica it goes to */
    uint32_t best = R;
    for (uint32_t r = 0; r < R; ++r) {
      if (room_after[r] < bytes[c]) continue;
      if (best == R) best = r;
      else if (!(flags & ORC_ADMIT_BEST_FIT) && room_after[r] > room_after[best]) best = r;
      else if ((flags & ORC_ADMIT_BEST_FIT) && room_after[r] < room_after[best]) best = r;
    }
    if (best < R) {
      replica[c] = (int32_t)best;
      room_after[best] -= bytes[c];
    }
  }
  free(done);
  return ORC_OK;
}
