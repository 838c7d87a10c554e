// Host side of libmori: argument validation, the context (device scratch,
// pinned plan mirror, staging), stream/event ordering of the three calls, and
// the two copy modes of the swaps.
//
//   plan       rank kernel (and the page state) -> page kernels, which also
//              store the plan into its pinned host mirror -> plan event.
//   swap-out   direct: translate addresses -> gather kernel storing straight
//              into host-mapped memory; copy engine: per chunk, gather kernel
//              into one half of a device staging buffer (caller's stream) ->
//              hipMemcpyAsync of each program segment to its host buffer on
//              the context's copy stream, while the next gather fills the
//              other half.
//   swap-in    direct: translate -> scatter of slots on pages free before the
//              step or released by idle dropped programs -> wait for the
//              swap-out -> scatter of slots on pages that were still in use
//              (read by the swap-out, or by a dropped program's inference step
//              ordered before it); copy engine: per chunk,
//              hipMemcpyAsync host -> staging half on the copy stream -> scatter
//              kernel on the caller's stream (after the swap-out event from the
//              first chunk that writes a page the swap-out reads), the next
//              chunk loading into the other half meanwhile.
//   next plan  waits on the stream for both swaps of the previous plan.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstring>
#include <new>
#include <vector>

#include "mori_internal.h"

using namespace mori;

namespace {

constexpr uint64_t kDefaultStaging = 512ull << 20;
constexpr uint32_t kGridHost = 128;     // enough outstanding 16-B accesses to fill the host link
// Workgroups of an HBM-to-HBM gather (d = 0) or scatter (d = 1).  Measured in
// the full-size pipelined rebalance: on runs of 32 KiB and more the gather is
// fastest with one run per workgroup (a 1 GiB staging half of 32 KiB runs:
// 32 768 workgroups, 4-5% faster than 16 384 and 6% faster than 8 192) while
// the scatter loses 1-2% there against 16 384; on 16 KiB runs 16 384
// workgroups (about four runs each) beat 32 768 by 2% and 8 192 by 3%.
uint32_t grid_device(uint64_t run, int d) { return run >= (32u << 10) && d == 0 ? 32768u : 16384u; }
constexpr uint64_t kTimeOnly = ~0ull;

struct BlobLayout {
  size_t sum, order, prefix, tier_old, tier_new, cat, out_prog, in_prog, out_base, in_base, total;
};

BlobLayout blob_layout(uint32_t pm) {
  BlobLayout L{};
  size_t o = 0;
  auto take = [&](size_t bytes) {
    const size_t r = o;
    o += (bytes + 255) & ~size_t(255);
    return r;
  };
  L.sum = take(sizeof(DevSummary));
  L.order = take(4ull * pm);
  L.prefix = take(8ull * pm);
  L.tier_old = take(pm);
  L.tier_new = take(pm);
  L.cat = take(pm);
  L.out_prog = take(4ull * pm);
  L.in_prog = take(4ull * pm);
  L.out_base = take(4ull * (pm + 1));
  L.in_base = take(4ull * (pm + 1));
  L.total = o;
  return L;
}

}  // namespace

struct mori_ctx {
  int device = 0;
  mori_pool pool{};
  uint64_t run = 0, block_bytes = 0;
  uint32_t LC = 0, max_programs = 0, ntiles = 0;
  BlobLayout L{};
  uint8_t* blob_dev = nullptr;   // plan blob on the device
  uint8_t* blob_host = nullptr;  // pinned mirror
  uint8_t* blob_host_dev = nullptr;  // the mirror as the device addresses it
  uint8_t* scratch = nullptr;    // device-only arrays
  uint32_t* base = nullptr;
  uint32_t* pstate = nullptr;
  uint32_t* out_src = nullptr;
  uint32_t* in_dst = nullptr;
  uint64_t* tile_cnt = nullptr;
  uint64_t* tile_base = nullptr;
  uint64_t* addr_stage[2] = {nullptr, nullptr};
  uint64_t* addr_dev[2] = {nullptr, nullptr};
  uint32_t* swap_err = nullptr;  // [2] per direction
  DevRange* ranges_dev = nullptr;
  uint64_t* addr_pinned = nullptr;  // [2][max_programs]
  uint8_t* staging[2] = {nullptr, nullptr};  // per direction, two halves
  uint64_t staging_bytes = 0;
  hipStream_t cstream[2] = {nullptr, nullptr};  // per direction: the copy-engine copies
  hipEvent_t ev_half_ready[2][2] = {};          // [dir][half]: gathered (out) / loaded (in)
  hipEvent_t ev_half_free[2][2] = {};           // [dir][half]: copied out (out) / scattered (in)
  hipEvent_t ev_start[2] = {nullptr, nullptr};
  std::vector<DevRange> ranges;
  hipEvent_t ev_plan = nullptr, ev_out = nullptr, ev_in = nullptr, ev_addr[2] = {nullptr, nullptr};
  bool have_plan = false, out_enqueued = false, in_enqueued = false;
  bool out_recorded = false, in_recorded = false, addr_pending[2] = {false, false};
  uint32_t P = 0;
  const uint32_t* tbl_off = nullptr;
  int last_hip_error = 0;
  uint32_t last_mode = 0;
  // kernel timing (opt-in)
  static constexpr int kProfCap = 4096;
  bool profiling = false;
  std::vector<hipEvent_t> prof_ev[2];  // pairs: [2 * i] start, [2 * i + 1] stop
  uint32_t prof_n[2] = {0, 0};
  uint64_t prof_bytes[2] = {0, 0};
  uint32_t prof_direct[2] = {0, 0};    // launches whose payload is the plan's whole direction

  DevSummary* sum_dev() const { return reinterpret_cast<DevSummary*>(blob_dev + L.sum); }
  const DevSummary* sum_host() const { return reinterpret_cast<const DevSummary*>(blob_host + L.sum); }
  template <typename T>
  T* dev(size_t off) const { return reinterpret_cast<T*>(blob_dev + off); }
  template <typename T>
  const T* host(size_t off) const { return reinterpret_cast<const T*>(blob_host + off); }
};

#define HIP_TRY(ctx, expr)                                          \
  do {                                                              \
    hipError_t e_ = (expr);                                         \
    if (e_ != hipSuccess) {                                         \
      if (ctx) (ctx)->last_hip_error = (int)e_;                     \
      (void)hipGetLastError();                                      \
      return MORI_EHIP;                                             \
    }                                                               \
  } while (0)

// Direct-mode swap launches move their plan's whole direction, whose size the
// host learns only from that plan; fold it into the profile record before a
// new plan replaces the host mirror (and when the record is read).
static int fold_direct_bytes(mori_ctx* c) {
  if (!c->have_plan || (!c->prof_direct[0] && !c->prof_direct[1])) return MORI_OK;
  HIP_TRY(c, hipEventSynchronize(c->ev_plan));
  const DevSummary* s = c->sum_host();
  c->prof_bytes[0] += c->prof_direct[0] * s->bytes_out;
  c->prof_bytes[1] += c->prof_direct[1] * s->bytes_in;
  c->prof_direct[0] = c->prof_direct[1] = 0;
  return MORI_OK;
}

static void destroy_profile_events(mori_ctx* c) {
  for (int d = 0; d < 2; ++d) {
    for (hipEvent_t e : c->prof_ev[d])
      if (e) {
        (void)hipEventSynchronize(e);
        (void)hipEventDestroy(e);
      }
    c->prof_ev[d].clear();
    c->prof_n[d] = 0;
  }
}

static void free_ctx(mori_ctx* c) {
  if (!c) return;
  // everything the context enqueued has finished before its memory goes
  if (c->ev_plan) (void)hipEventSynchronize(c->ev_plan);
  if (c->ev_out) (void)hipEventSynchronize(c->ev_out);
  if (c->ev_in) (void)hipEventSynchronize(c->ev_in);
  for (int d = 0; d < 2; ++d)
    if (c->ev_addr[d]) (void)hipEventSynchronize(c->ev_addr[d]);
  for (int d = 0; d < 2; ++d)
    if (c->cstream[d]) (void)hipStreamSynchronize(c->cstream[d]);
  destroy_profile_events(c);
  if (c->blob_dev) (void)hipFree(c->blob_dev);
  if (c->scratch) (void)hipFree(c->scratch);
  for (int d = 0; d < 2; ++d)
    if (c->staging[d]) (void)hipFree(c->staging[d]);
  if (c->blob_host) (void)hipHostFree(c->blob_host);
  if (c->addr_pinned) (void)hipHostFree(c->addr_pinned);
  hipEvent_t evs[] = {c->ev_plan,          c->ev_out,           c->ev_in,           c->ev_addr[0],
                      c->ev_addr[1],       c->ev_start[0],      c->ev_start[1],     c->ev_half_ready[0][0],
                      c->ev_half_ready[0][1], c->ev_half_ready[1][0], c->ev_half_ready[1][1],
                      c->ev_half_free[0][0], c->ev_half_free[0][1], c->ev_half_free[1][0], c->ev_half_free[1][1]};
  for (hipEvent_t e : evs)
    if (e) (void)hipEventDestroy(e);
  for (int d = 0; d < 2; ++d)
    if (c->cstream[d]) (void)hipStreamDestroy(c->cstream[d]);
  delete c;
}

extern "C" int mori_create(const mori_pool* pool, uint32_t max_programs, uint64_t staging_bytes, uint32_t flags,
                           mori_ctx** out) {
  if (!pool || !out) return MORI_EINVAL;
  *out = nullptr;
  if (flags & ~MORI_CREATE_COPY_STREAMS) return MORI_EINVAL;
  if (!pool->base || (reinterpret_cast<uintptr_t>(pool->base) & 255u)) return MORI_EINVAL;
  if (!pool->layers || !pool->planes || !pool->block_tokens || !pool->row_bytes || (pool->row_bytes & 15u))
    return MORI_EINVAL;
  if (!pool->num_blocks || pool->num_blocks == MORI_NO_PAGE) return MORI_EINVAL;
  if (max_programs == 0 || max_programs > MORI_MAX_PROGRAMS) return MORI_EINVAL;
  const uint64_t LC = (uint64_t)pool->layers * pool->planes;
  const uint64_t run = (uint64_t)pool->block_tokens * pool->row_bytes;
  if (LC > 0xFFFFu || run > (1ull << 31) || LC * run >= (1ull << 32)) return MORI_EINVAL;
  if (staging_bytes == 0) staging_bytes = kDefaultStaging;
  staging_bytes = staging_bytes / (2 * run) * (2 * run);  // two halves of whole runs
  if (staging_bytes == 0) return MORI_EINVAL;

  mori_ctx* c = new (std::nothrow) mori_ctx();
  if (!c) return MORI_ENOSPC;
  c->pool = *pool;
  c->LC = (uint32_t)LC;
  c->run = run;
  c->block_bytes = LC * run;
  c->max_programs = max_programs;
  c->ntiles = (uint32_t)((pool->num_blocks + (uint64_t)PAGE_TILE - 1) / PAGE_TILE);
  c->L = blob_layout(max_programs);
  c->staging_bytes = staging_bytes;
  int rc = MORI_OK;
  auto fail = [&](hipError_t e) {
    c->last_hip_error = (int)e;
    (void)hipGetLastError();
    free_ctx(c);
    return MORI_EHIP;
  };
  hipError_t e;
  if ((e = hipGetDevice(&c->device)) != hipSuccess) return fail(e);
  if ((e = hipMalloc(&c->blob_dev, c->L.total)) != hipSuccess) return fail(e);
  if ((e = hipHostMalloc(&c->blob_host, c->L.total, hipHostMallocMapped)) != hipSuccess) return fail(e);
  std::memset(c->blob_host, 0, c->L.total);
  if ((e = hipHostGetDevicePointer(reinterpret_cast<void**>(&c->blob_host_dev), c->blob_host, 0)) != hipSuccess)
    return fail(e);
  // device-only scratch, 256-B aligned pieces
  const uint64_t NB = pool->num_blocks, pm = max_programs;
  size_t o = 0;
  auto take = [&](size_t bytes) {
    const size_t r = o;
    o += (bytes + 255) & ~size_t(255);
    return r;
  };
  const size_t o_base = take(4 * pm), o_pstate = take(4 * NB), o_out_src = take(4 * NB), o_in_dst = take(4 * NB);
  const size_t o_tc = take(16ull * c->ntiles), o_tb = take(16ull * c->ntiles);
  const size_t o_as0 = take(8 * pm), o_as1 = take(8 * pm), o_ad0 = take(8 * pm), o_ad1 = take(8 * pm);
  const size_t o_err = take(8), o_rng = take(sizeof(DevRange) * MORI_MAX_RANGES);
  if ((e = hipMalloc(&c->scratch, o)) != hipSuccess) return fail(e);
  c->base = reinterpret_cast<uint32_t*>(c->scratch + o_base);
  c->pstate = reinterpret_cast<uint32_t*>(c->scratch + o_pstate);
  c->out_src = reinterpret_cast<uint32_t*>(c->scratch + o_out_src);
  c->in_dst = reinterpret_cast<uint32_t*>(c->scratch + o_in_dst);
  c->tile_cnt = reinterpret_cast<uint64_t*>(c->scratch + o_tc);
  c->tile_base = reinterpret_cast<uint64_t*>(c->scratch + o_tb);
  c->addr_stage[0] = reinterpret_cast<uint64_t*>(c->scratch + o_as0);
  c->addr_stage[1] = reinterpret_cast<uint64_t*>(c->scratch + o_as1);
  c->addr_dev[0] = reinterpret_cast<uint64_t*>(c->scratch + o_ad0);
  c->addr_dev[1] = reinterpret_cast<uint64_t*>(c->scratch + o_ad1);
  c->swap_err = reinterpret_cast<uint32_t*>(c->scratch + o_err);
  c->ranges_dev = reinterpret_cast<DevRange*>(c->scratch + o_rng);
  if ((e = hipMemset(c->scratch, 0, o)) != hipSuccess) return fail(e);
  if ((e = hipMemset(c->blob_dev, 0, c->L.total)) != hipSuccess) return fail(e);
  if ((e = hipHostMalloc(&c->addr_pinned, 16 * pm, hipHostMallocDefault)) != hipSuccess) return fail(e);
  for (int d = 0; d < 2; ++d)
    if ((e = hipMalloc(&c->staging[d], staging_bytes)) != hipSuccess) return fail(e);
  for (hipEvent_t* ev : {&c->ev_plan, &c->ev_out, &c->ev_in, &c->ev_addr[0], &c->ev_addr[1], &c->ev_start[0],
                         &c->ev_start[1], &c->ev_half_ready[0][0], &c->ev_half_ready[0][1],
                         &c->ev_half_ready[1][0], &c->ev_half_ready[1][1], &c->ev_half_free[0][0],
                         &c->ev_half_free[0][1], &c->ev_half_free[1][0], &c->ev_half_free[1][1]})
    if ((e = hipEventCreateWithFlags(ev, hipEventDisableTiming)) != hipSuccess) return fail(e);
  // Copy streams (default priority) only when the caller says the process has
  // hardware queues to spare: HIP maps streams onto GPU_MAX_HW_QUEUES queues
  // (4 by default) and streams beyond that share a queue, where each stream's
  // waits block the other's work and the two swap directions serialise.
  // Without them the copies run on the caller's stream, in order with the
  // gathers/scatters.
  if (flags & MORI_CREATE_COPY_STREAMS)
    for (int d = 0; d < 2; ++d)
      if ((e = hipStreamCreateWithFlags(&c->cstream[d], hipStreamNonBlocking)) != hipSuccess) return fail(e);
  *out = c;
  return rc;
}

extern "C" int mori_destroy(mori_ctx* ctx) {
  free_ctx(ctx);
  return MORI_OK;
}

extern "C" int mori_register(mori_ctx* ctx, void* ptr, uint64_t bytes) {
  if (!ctx || !ptr || bytes == 0) return MORI_EINVAL;
  if (ctx->ranges.size() >= MORI_MAX_RANGES) return MORI_ENOSPC;
  hipPointerAttribute_t a0{}, a1{};
  if (hipPointerGetAttributes(&a0, ptr) != hipSuccess) {
    (void)hipGetLastError();
    return MORI_EINVAL;
  }
  uint8_t* last = static_cast<uint8_t*>(ptr) + (bytes - 1);
  if (hipPointerGetAttributes(&a1, last) != hipSuccess) {
    (void)hipGetLastError();
    return MORI_EINVAL;
  }
  const bool host = a0.type == hipMemoryTypeHost, device = a0.type == hipMemoryTypeDevice;
  if (!(host || device) || a1.type != a0.type) return MORI_EINVAL;
  if (device && a0.device != ctx->device) return MORI_EINVAL;
  if (!a0.devicePointer || !a1.devicePointer) return MORI_EINVAL;
  const uint64_t d0 = reinterpret_cast<uint64_t>(a0.devicePointer);
  const uint64_t d1 = reinterpret_cast<uint64_t>(a1.devicePointer);
  if (d1 - d0 != bytes - 1) return MORI_EINVAL;  // one contiguous mapping
  DevRange r{reinterpret_cast<uint64_t>(ptr), bytes, d0, device ? 1ull : 0ull};
  // the new entry goes to the device first, then to the host list, so a
  // failure registers nothing; entries a swap may be reading are not written
  HIP_TRY(ctx, hipSetDevice(ctx->device));
  HIP_TRY(ctx, hipMemcpy(ctx->ranges_dev + ctx->ranges.size(), &r, sizeof r, hipMemcpyHostToDevice));
  ctx->ranges.push_back(r);
  return MORI_OK;
}

extern "C" int mori_host_alloc(uint64_t bytes, void** out) {
  if (!out || bytes == 0) return MORI_EINVAL;
  *out = nullptr;
  hipError_t e = hipHostMalloc(out, bytes, hipHostMallocMapped | hipHostMallocPortable);
  if (e != hipSuccess) {
    (void)hipGetLastError();
    *out = nullptr;
    return MORI_EHIP;
  }
  return MORI_OK;
}

extern "C" int mori_host_free(void* ptr) {
  if (!ptr) return MORI_OK;
  return hipHostFree(ptr) == hipSuccess ? MORI_OK : MORI_EHIP;
}

extern "C" int mori_rank_partition(mori_ctx* ctx, const mori_programs* pr, const mori_budget* b, void* stream) {
  if (!ctx || !pr || !b) return MORI_EINVAL;
  const uint32_t P = pr->num_programs;
  if (P > ctx->max_programs) return MORI_ENOSPC;
  if (b->flags & ~(MORI_F_STATUS_KEY | MORI_F_SKIP_FIT | MORI_F_IDLENESS_GIVEN | MORI_F_INCREMENTAL |
                   MORI_F_SSD_TIER))
    return MORI_EINVAL;
  if ((b->flags & MORI_F_SSD_TIER) && (b->flags & MORI_F_INCREMENTAL)) return MORI_EINVAL;
  if (!pr->tbl_off || !pr->free_map) return MORI_EINVAL;
  if (P && (!pr->tier || (pr->tbl_len && !pr->tbl))) return MORI_EINVAL;
  if (b->flags & MORI_F_IDLENESS_GIVEN) {
    if (P && !pr->idleness) return MORI_EINVAL;
  } else {
    if (pr->window_k == 0 || pr->window_k > MORI_MAX_WINDOW) return MORI_EINVAL;
    if (P && !pr->window) return MORI_EINVAL;
  }
  if ((b->flags & (MORI_F_STATUS_KEY | MORI_F_INCREMENTAL)) && P && !pr->status) return MORI_EINVAL;
  if (b->gpu_bytes > (uint64_t)ctx->pool.num_blocks * ctx->block_bytes) return MORI_EINVAL;
  hipStream_t s = static_cast<hipStream_t>(stream);
  HIP_TRY(ctx, hipSetDevice(ctx->device));
  if (int rc = fold_direct_bytes(ctx)) return rc;
  if (ctx->out_recorded) HIP_TRY(ctx, hipStreamWaitEvent(s, ctx->ev_out, 0));
  if (ctx->in_recorded) HIP_TRY(ctx, hipStreamWaitEvent(s, ctx->ev_in, 0));
  // from here the previous plan is superseded: a launch that fails leaves none
  ctx->have_plan = false;

  PlanArgs a{};
  a.window = pr->window;
  a.idleness = pr->idleness;
  a.status = pr->status;
  a.tbl_off = pr->tbl_off;
  a.tbl = pr->tbl;
  a.tier = pr->tier;
  a.free_map = pr->free_map;
  a.tbl_len = pr->tbl_len;
  a.P = P;
  a.k = (b->flags & MORI_F_IDLENESS_GIVEN) ? 0 : pr->window_k;
  a.flags = b->flags;
  a.NB = ctx->pool.num_blocks;
  a.ntiles = ctx->ntiles;
  a.block_bytes = ctx->block_bytes;
  a.gpu_bytes = b->gpu_bytes;
  a.cpu_bytes = b->cpu_bytes;
  a.ssd_bytes = (b->flags & MORI_F_SSD_TIER) ? b->ssd_bytes : 0;
  a.sum = ctx->sum_dev();
  a.order = ctx->dev<uint32_t>(ctx->L.order);
  a.prefix = ctx->dev<uint64_t>(ctx->L.prefix);
  a.tier_old = ctx->dev<uint8_t>(ctx->L.tier_old);
  a.tier_new = ctx->dev<uint8_t>(ctx->L.tier_new);
  a.cat = ctx->dev<uint8_t>(ctx->L.cat);
  a.out_prog = ctx->dev<uint32_t>(ctx->L.out_prog);
  a.in_prog = ctx->dev<uint32_t>(ctx->L.in_prog);
  a.out_pg_base = ctx->dev<uint32_t>(ctx->L.out_base);
  a.in_pg_base = ctx->dev<uint32_t>(ctx->L.in_base);
  a.base = ctx->base;
  a.pstate = ctx->pstate;
  a.out_src = ctx->out_src;
  a.in_dst = ctx->in_dst;
  a.tile_cnt = ctx->tile_cnt;
  a.tile_base = ctx->tile_base;
  a.swap_err = ctx->swap_err;
  a.host_delta = reinterpret_cast<int64_t>(ctx->blob_host_dev) - reinterpret_cast<int64_t>(ctx->blob_dev);
  HIP_TRY(ctx, launch_rank(a, s));
  HIP_TRY(ctx, launch_pages(a, s));
  HIP_TRY(ctx, hipEventRecord(ctx->ev_plan, s));
  ctx->have_plan = true;
  ctx->out_enqueued = ctx->in_enqueued = false;
  ctx->P = P;
  ctx->tbl_off = pr->tbl_off;
  return MORI_OK;
}

extern "C" int mori_plan_wait(mori_ctx* ctx, mori_plan* out) {
  if (!ctx || !out) return MORI_EINVAL;
  if (!ctx->have_plan) return MORI_ESTATE;
  HIP_TRY(ctx, hipEventSynchronize(ctx->ev_plan));
  const DevSummary* s = ctx->sum_host();
  mori_plan p{};
  p.num_programs = s->num_programs;
  p.m_gpu = s->m_gpu;
  p.m_cpu = s->m_cpu;
  p.n_out = s->n_out;
  p.n_in = s->n_in;
  p.n_drop_gpu = s->n_drop_gpu;
  p.n_drop_cpu = s->n_drop_cpu;
  p.n_admit_gpu = s->n_admit_gpu;
  p.n_admit_cpu = s->n_admit_cpu;
  p.device_error = s->error;
  p.pages_out = s->pages_out;
  p.pages_in = s->pages_in;
  p.pages_admit = s->pages_admit;
  p.pages_free_before = s->pages_free_before;
  p.pages_released = s->pages_released;
  p.pages_recycled = s->pages_recycled;
  p.pages_dropped = s->pages_dropped;
  p.pages_free_after = s->pages_free_after;
  p.bytes_out = s->bytes_out;
  p.bytes_in = s->bytes_in;
  p.gpu_bytes_after = s->gpu_bytes_after;
  p.cpu_bytes_after = s->cpu_bytes_after;
  p.ssd_bytes_after = s->ssd_bytes_after;
  p.m_ssd = s->m_ssd;
  p.order = ctx->host<uint32_t>(ctx->L.order);
  p.prefix = ctx->host<uint64_t>(ctx->L.prefix);
  p.tier_old = ctx->host<uint8_t>(ctx->L.tier_old);
  p.tier_new = ctx->host<uint8_t>(ctx->L.tier_new);
  p.category = ctx->host<uint8_t>(ctx->L.cat);
  p.out_programs = ctx->host<uint32_t>(ctx->L.out_prog);
  p.in_programs = ctx->host<uint32_t>(ctx->L.in_prog);
  *out = p;
  return s->error ? MORI_EDEVICE : MORI_OK;
}

namespace {

const DevRange* find_range(const mori_ctx* c, uint64_t addr, uint64_t bytes) {
  for (const DevRange& r : c->ranges)
    if (addr >= r.host_base && addr - r.host_base <= r.bytes && bytes <= r.bytes - (addr - r.host_base)) return &r;
  return nullptr;
}

// Chooses the copy mode: AUTO resolves to the copy engines for host memory
// (measured faster on MI355X when both directions run together) and to
// kernels for device-memory buffers.  Returns false on an invalid mode.
bool resolve_mode(const mori_ctx* c, const uint64_t* addr, uint32_t mode, uint32_t* resolved, bool* device_only) {
  if (mode > MORI_COPY_CE) return false;
  bool any = false, all_dev = true;
  for (uint32_t p = 0; p < c->P; ++p) {
    if (!addr[p]) continue;
    const DevRange* r = find_range(c, addr[p], 0);
    if (!r) continue;
    any = true;
    if (!r->is_device) all_dev = false;
  }
  *device_only = any && all_dev;
  *resolved = mode == MORI_COPY_AUTO ? (*device_only ? MORI_COPY_KERNEL : MORI_COPY_CE) : mode;
  return true;
}

// Host-side check of every moving program's buffer (copy-engine mode).
bool host_check(const mori_ctx* c, const uint64_t* addr, const uint32_t* progs, uint32_t n, const uint32_t* pg_base) {
  for (uint32_t j = 0; j < n; ++j) {
    const uint64_t bytes = (uint64_t)(pg_base[j + 1] - pg_base[j]) * c->block_bytes;
    if (!bytes) continue;
    const uint64_t h = addr[progs[j]];
    if (!h || (h & 15u) || !find_range(c, h, bytes)) return false;
  }
  return true;
}

int stage_addresses(mori_ctx* c, int d, const uint64_t* addr, hipStream_t s) {
  if (c->addr_pending[d]) HIP_TRY(c, hipEventSynchronize(c->ev_addr[d]));
  uint64_t* pin = c->addr_pinned + (size_t)d * c->max_programs;
  std::memcpy(pin, addr, sizeof(uint64_t) * c->P);
  if (c->P) HIP_TRY(c, hipMemcpyAsync(c->addr_stage[d], pin, sizeof(uint64_t) * c->P, hipMemcpyHostToDevice, s));
  HIP_TRY(c, hipEventRecord(c->ev_addr[d], s));
  c->addr_pending[d] = true;
  return MORI_OK;
}

// Copies of one staging half, issued in unit order; a segment that continues
// the previous one on both sides (host buffers of consecutive programs that
// are adjacent, as a first-fit arena hands them out) joins it, so a half
// takes as few copy-engine commands as its host layout allows.
struct CopyRun {
  uint8_t* dst = nullptr;
  const uint8_t* src = nullptr;
  uint64_t bytes = 0;
};

int copy_flush(mori_ctx* c, CopyRun& r, hipMemcpyKind kind, hipStream_t s) {
  if (r.bytes) HIP_TRY(c, hipMemcpyAsync(r.dst, r.src, r.bytes, kind, s));
  r.bytes = 0;
  return MORI_OK;
}

int copy_add(mori_ctx* c, CopyRun& r, uint8_t* dst, const uint8_t* src, uint64_t bytes, hipMemcpyKind kind,
             hipStream_t s) {
  if (r.bytes && r.dst + r.bytes == dst && r.src + r.bytes == src) {
    // joined only inside one registered range: one allocation for the copy
    const uint64_t host = reinterpret_cast<uint64_t>(kind == hipMemcpyDeviceToHost ? r.dst : r.src);
    if (find_range(c, host, r.bytes + bytes)) {
      r.bytes += bytes;
      return MORI_OK;
    }
  }
  if (int rc = copy_flush(c, r, kind, s)) return rc;
  r.dst = dst;
  r.src = src;
  r.bytes = bytes;
  return MORI_OK;
}

SwapArgs swap_args(const mori_ctx* c, int d) {
  SwapArgs a{};
  a.pool = static_cast<uint8_t*>(c->pool.base);
  a.NB = c->pool.num_blocks;
  a.run = c->run;
  a.LC = c->LC;
  a.sum = c->sum_dev();
  a.prog = c->dev<uint32_t>(d ? c->L.in_prog : c->L.out_prog);
  a.pg_base = c->dev<uint32_t>(d ? c->L.in_base : c->L.out_base);
  a.pages = d ? c->in_dst : c->out_src;
  a.addr = c->addr_dev[d];
  a.swap_err = c->swap_err;
  return a;
}

// Launches one gather (d = 0) or scatter (d = 1) kernel, bracketed by timing
// events on the same stream when profiling is on.  payload = bytes moved; 0
// for a direct launch whose payload is the whole direction of the plan;
// kTimeOnly for the second part of a direct swap-in (its bytes are already
// counted with the first part).
int timed_swap_launch(mori_ctx* c, int d, const SwapArgs& a, uint32_t grid, hipStream_t s, uint64_t payload) {
  const bool rec = c->profiling && c->prof_n[d] < (uint32_t)mori_ctx::kProfCap;
  if (rec) HIP_TRY(c, hipEventRecord(c->prof_ev[d][2 * c->prof_n[d]], s));
  HIP_TRY(c, d ? launch_swap_in(a, grid, s) : launch_swap_out(a, grid, s));
  if (rec) {
    HIP_TRY(c, hipEventRecord(c->prof_ev[d][2 * c->prof_n[d] + 1], s));
    ++c->prof_n[d];
    if (payload == kTimeOnly) {
    } else if (payload) {
      c->prof_bytes[d] += payload;
    } else {
      ++c->prof_direct[d];
    }
  }
  return MORI_OK;
}

int translate(mori_ctx* c, int d, hipStream_t s) {
  TranslateArgs t{};
  t.sum = c->sum_dev();
  t.prog = c->dev<uint32_t>(d ? c->L.in_prog : c->L.out_prog);
  t.dir_in = d;
  t.tbl_off = c->tbl_off;
  t.block_bytes = c->block_bytes;
  t.addr_in = c->addr_stage[d];
  t.addr_out = c->addr_dev[d];
  t.ranges = c->ranges_dev;
  t.nranges = (uint32_t)c->ranges.size();
  t.swap_err = c->swap_err;
  HIP_TRY(c, launch_translate(t, s));
  return MORI_OK;
}

}  // namespace

extern "C" int mori_kv_swap_out(mori_ctx* ctx, const uint64_t* host_dst, uint32_t mode, void* stream) {
  if (!ctx || !host_dst) return MORI_EINVAL;
  if (!ctx->have_plan || ctx->out_enqueued) return MORI_ESTATE;
  uint32_t m;
  bool device_only;
  if (!resolve_mode(ctx, host_dst, mode, &m, &device_only)) return MORI_EINVAL;
  hipStream_t s = static_cast<hipStream_t>(stream);
  HIP_TRY(ctx, hipSetDevice(ctx->device));
  if (m == MORI_COPY_KERNEL) {
    HIP_TRY(ctx, hipStreamWaitEvent(s, ctx->ev_plan, 0));
    int rc = stage_addresses(ctx, 0, host_dst, s);
    if (rc) return rc;
    if ((rc = translate(ctx, 0, s))) return rc;
    SwapArgs a = swap_args(ctx, 0);
    a.host_link = !device_only;
    if ((rc = timed_swap_launch(ctx, 0, a, device_only ? grid_device(ctx->run, 0) : kGridHost, s, 0))) return rc;
  } else {
    HIP_TRY(ctx, hipEventSynchronize(ctx->ev_plan));
    const DevSummary* sh = ctx->sum_host();
    if (sh->error) return MORI_EDEVICE;
    const uint32_t n = sh->n_out;
    const uint32_t* progs = ctx->host<uint32_t>(ctx->L.out_prog);
    const uint32_t* base = ctx->host<uint32_t>(ctx->L.out_base);
    if (!host_check(ctx, host_dst, progs, n, base)) return MORI_EINVAL;
    HIP_TRY(ctx, hipStreamWaitEvent(s, ctx->ev_plan, 0));
    const uint64_t LC = ctx->LC, run = ctx->run;
    const uint64_t total = n ? (uint64_t)base[n] * LC : 0;
    const uint64_t cu = ctx->staging_bytes / 2 / run;  // chunk = one staging half
    hipStream_t cs = ctx->cstream[0] ? ctx->cstream[0] : s;
    SwapArgs a = swap_args(ctx, 0);
    uint32_t j = 0;  // first program that may overlap the chunk
    uint64_t c = 0;
    // Double buffering: the gather of chunk c (stream s) fills one half while the
    // copy engines drain the other half (copy stream), so the gathers leave the
    // copy chain only at its start.  With no copy stream (cs == s) the same
    // sequence runs in stream order.
    for (uint64_t u0 = 0; u0 < total; u0 += cu, ++c) {
      const uint64_t u1 = std::min(total, u0 + cu);
      const int h = (int)(c & 1);
      uint8_t* half = ctx->staging[0] + (uint64_t)h * cu * run;
      if (c >= 2) HIP_TRY(ctx, hipStreamWaitEvent(s, ctx->ev_half_free[0][h], 0));
      a.staging = half;
      a.u_begin = u0;
      a.u_end = u1;
      const int rc = timed_swap_launch(ctx, 0, a, (uint32_t)std::min<uint64_t>(u1 - u0, grid_device(ctx->run, 0)), s,
                                       (u1 - u0) * run);
      if (rc) return rc;
      HIP_TRY(ctx, hipEventRecord(ctx->ev_half_ready[0][h], s));
      HIP_TRY(ctx, hipStreamWaitEvent(cs, ctx->ev_half_ready[0][h], 0));
      while (j < n && (uint64_t)base[j + 1] * LC <= u0) ++j;
      CopyRun cr;
      for (uint32_t k = j; k < n && (uint64_t)base[k] * LC < u1; ++k) {
        const uint64_t b0 = (uint64_t)base[k] * LC, b1 = (uint64_t)base[k + 1] * LC;
        const uint64_t lo = std::max(u0, b0), hi = std::min(u1, b1);
        if (hi <= lo) continue;
        uint8_t* dst = reinterpret_cast<uint8_t*>(host_dst[progs[k]]) + (lo - b0) * run;
        if (int rc = copy_add(ctx, cr, dst, half + (lo - u0) * run, (hi - lo) * run, hipMemcpyDeviceToHost, cs))
          return rc;
      }
      if (int rc = copy_flush(ctx, cr, hipMemcpyDeviceToHost, cs)) return rc;
      HIP_TRY(ctx, hipEventRecord(ctx->ev_half_free[0][h], cs));
    }
    // join: the copy stream's last copy implies all earlier ones
    if (c) HIP_TRY(ctx, hipStreamWaitEvent(s, ctx->ev_half_free[0][(c - 1) & 1], 0));
  }
  HIP_TRY(ctx, hipEventRecord(ctx->ev_out, s));
  ctx->out_enqueued = ctx->out_recorded = true;
  ctx->last_mode = m;
  return MORI_OK;
}

extern "C" int mori_kv_swap_in(mori_ctx* ctx, const uint64_t* host_src, uint32_t mode, void* stream) {
  if (!ctx || !host_src) return MORI_EINVAL;
  if (!ctx->have_plan || ctx->in_enqueued || !ctx->out_enqueued) return MORI_ESTATE;
  uint32_t m;
  bool device_only;
  if (!resolve_mode(ctx, host_src, mode, &m, &device_only)) return MORI_EINVAL;
  hipStream_t s = static_cast<hipStream_t>(stream);
  HIP_TRY(ctx, hipSetDevice(ctx->device));
  if (m == MORI_COPY_KERNEL) {
    HIP_TRY(ctx, hipStreamWaitEvent(s, ctx->ev_plan, 0));
    int rc = stage_addresses(ctx, 1, host_src, s);
    if (rc) return rc;
    if ((rc = translate(ctx, 1, s))) return rc;
    SwapArgs a = swap_args(ctx, 1);
    a.host_link = !device_only;
    const uint32_t grid = device_only ? grid_device(ctx->run, 1) : kGridHost;
    a.part = 1;  // slots on pages that were free before the step
    if ((rc = timed_swap_launch(ctx, 1, a, grid, s, 0))) return rc;
    HIP_TRY(ctx, hipStreamWaitEvent(s, ctx->ev_out, 0));
    a.part = 2;  // slots on pages released by this step's swap-out
    if ((rc = timed_swap_launch(ctx, 1, a, grid, s, kTimeOnly))) return rc;
  } else {
    HIP_TRY(ctx, hipEventSynchronize(ctx->ev_plan));
    const DevSummary* sh = ctx->sum_host();
    if (sh->error) return MORI_EDEVICE;
    const uint32_t n = sh->n_in;
    const uint32_t* progs = ctx->host<uint32_t>(ctx->L.in_prog);
    const uint32_t* base = ctx->host<uint32_t>(ctx->L.in_base);
    if (!host_check(ctx, host_src, progs, n, base)) return MORI_EINVAL;
    HIP_TRY(ctx, hipStreamWaitEvent(s, ctx->ev_plan, 0));
    // slots below `ready` are on pages free before the step or released by an
    // idle dropped program; the rest are on pages still in use until the
    // swap-out stream has passed
    const uint64_t LC = ctx->LC, run = ctx->run, ready = sh->pages_free_before + sh->pages_dropped;
    const uint64_t total = n ? (uint64_t)base[n] * LC : 0;
    const uint64_t cu = ctx->staging_bytes / 2 / run;  // chunk = one staging half
    // first unit of the first program with a slot on a page the swap-out reads
    uint64_t u_recycled = total;
    for (uint32_t k = 0; k < n; ++k)
      if (base[k + 1] > ready && base[k + 1] > base[k]) {
        u_recycled = (uint64_t)base[k] * LC;
        break;
      }
    hipStream_t cs = ctx->cstream[1] ? ctx->cstream[1] : s;
    // the copies start after everything already ordered before this swap-in on s
    // (the plan, hence the previous plan's swaps and their use of the staging)
    HIP_TRY(ctx, hipEventRecord(ctx->ev_start[1], s));
    HIP_TRY(ctx, hipStreamWaitEvent(cs, ctx->ev_start[1], 0));
    bool waited = false;
    SwapArgs a = swap_args(ctx, 1);
    uint32_t j = 0;
    uint64_t c = 0;
    // The first chunk is half a staging half: the copy engines then finish
    // the swap-in's chunks half a chunk period away from the swap-out's, so
    // a scatter kernel (launched when its chunk has arrived) falls between
    // the gather kernels (launched when a chunk has left) instead of on top
    // of them, and neither shares HBM with the other.
    const uint64_t cu0 = total > cu ? std::max<uint64_t>(1, cu / 2) : cu;
    for (uint64_t u0 = 0, u1 = 0; u0 < total; u0 = u1, ++c) {
      u1 = std::min(total, u0 + (c == 0 ? cu0 : cu));
      const int h = (int)(c & 1);
      uint8_t* half = ctx->staging[1] + (uint64_t)h * cu * run;
      if (c >= 2) HIP_TRY(ctx, hipStreamWaitEvent(cs, ctx->ev_half_free[1][h], 0));
      while (j < n && (uint64_t)base[j + 1] * LC <= u0) ++j;
      CopyRun cr;
      for (uint32_t k = j; k < n && (uint64_t)base[k] * LC < u1; ++k) {
        const uint64_t b0 = (uint64_t)base[k] * LC, b1 = (uint64_t)base[k + 1] * LC;
        const uint64_t lo = std::max(u0, b0), hi = std::min(u1, b1);
        if (hi <= lo) continue;
        const uint8_t* src = reinterpret_cast<const uint8_t*>(host_src[progs[k]]) + (lo - b0) * run;
        if (int rc = copy_add(ctx, cr, half + (lo - u0) * run, src, (hi - lo) * run, hipMemcpyHostToDevice, cs))
          return rc;
      }
      if (int rc = copy_flush(ctx, cr, hipMemcpyHostToDevice, cs)) return rc;
      HIP_TRY(ctx, hipEventRecord(ctx->ev_half_ready[1][h], cs));
      HIP_TRY(ctx, hipStreamWaitEvent(s, ctx->ev_half_ready[1][h], 0));
      if (!waited && u1 > u_recycled) {
        HIP_TRY(ctx, hipStreamWaitEvent(s, ctx->ev_out, 0));
        waited = true;
      }
      a.staging = half;
      a.u_begin = u0;
      a.u_end = u1;
      const int rc = timed_swap_launch(ctx, 1, a, (uint32_t)std::min<uint64_t>(u1 - u0, grid_device(ctx->run, 1)), s,
                                       (u1 - u0) * run);
      if (rc) return rc;
      HIP_TRY(ctx, hipEventRecord(ctx->ev_half_free[1][h], s));
    }
  }
  HIP_TRY(ctx, hipEventRecord(ctx->ev_in, s));
  ctx->in_enqueued = ctx->in_recorded = true;
  ctx->last_mode = m;
  return MORI_OK;
}

extern "C" int mori_query(mori_ctx* ctx, int what, uint64_t* value) {
  if (!ctx || !value) return MORI_EINVAL;
  switch (what) {
    case MORI_Q_LAST_HIP_ERROR:
      *value = (uint64_t)(uint32_t)ctx->last_hip_error;
      return MORI_OK;
    case MORI_Q_DEVICE_ERROR: {
      if (ctx->have_plan) HIP_TRY(ctx, hipEventSynchronize(ctx->ev_plan));
      if (ctx->out_recorded) HIP_TRY(ctx, hipEventSynchronize(ctx->ev_out));
      if (ctx->in_recorded) HIP_TRY(ctx, hipEventSynchronize(ctx->ev_in));
      uint32_t swap_err[2] = {0, 0};
      HIP_TRY(ctx, hipMemcpy(swap_err, ctx->swap_err, sizeof swap_err, hipMemcpyDeviceToHost));
      *value = (uint64_t)(ctx->have_plan ? ctx->sum_host()->error : 0u) | swap_err[0] | swap_err[1];
      return MORI_OK;
    }
    case MORI_Q_LAST_MODE:
      *value = ctx->last_mode;
      return MORI_OK;
    case MORI_Q_PLAN_EVENT:
      *value = reinterpret_cast<uint64_t>(ctx->ev_plan);
      return MORI_OK;
    case MORI_Q_OUT_EVENT:
      *value = reinterpret_cast<uint64_t>(ctx->ev_out);
      return MORI_OK;
    case MORI_Q_IN_EVENT:
      *value = reinterpret_cast<uint64_t>(ctx->ev_in);
      return MORI_OK;
    default:
      return MORI_EINVAL;
  }
}

extern "C" int mori_evict_workspace(uint32_t num_blocks, uint64_t* bytes) {
  if (!bytes) return MORI_EINVAL;
  *bytes = evict_workspace_bytes(num_blocks);
  return MORI_OK;
}

extern "C" int mori_evict_order(const mori_blocks* b, uint32_t tier, uint64_t need_bytes, void* workspace,
                                uint64_t workspace_bytes, uint32_t* order, uint64_t* prefix, uint32_t* result,
                                void* stream) {
  if (!b || !workspace || !result) return MORI_EINVAL;
  if (tier != MORI_TIER_GPU && tier != MORI_TIER_CPU) return MORI_EINVAL;
  if (reinterpret_cast<uintptr_t>(workspace) & 255u) return MORI_EINVAL;
  if (workspace_bytes < evict_workspace_bytes(b->num_blocks)) return MORI_EINVAL;
  if (b->num_blocks && (!b->type || !b->last_access || !order)) return MORI_EINVAL;
  const hipError_t e = launch_evict(b->num_blocks, b->type, b->last_access, b->size, b->unit_bytes, tier,
                                    need_bytes, workspace, order, prefix, result, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) {
    (void)hipGetLastError();
    return MORI_EHIP;
  }
  return MORI_OK;
}

extern "C" int mori_profile(mori_ctx* ctx, int enable) {
  if (!ctx) return MORI_EINVAL;
  if (enable && ctx->prof_ev[0].empty()) {
    HIP_TRY(ctx, hipSetDevice(ctx->device));
    for (int d = 0; d < 2; ++d) {
      ctx->prof_ev[d].resize(2 * mori_ctx::kProfCap, nullptr);
      for (hipEvent_t& e : ctx->prof_ev[d]) {
        const hipError_t err = hipEventCreate(&e);
        if (err != hipSuccess) {
          e = nullptr;
          ctx->last_hip_error = (int)err;
          (void)hipGetLastError();
          destroy_profile_events(ctx);
          return MORI_EHIP;
        }
      }
    }
  }
  ctx->profiling = enable != 0;
  return MORI_OK;
}

extern "C" int mori_profile_read(mori_ctx* ctx, int direction, uint64_t* launches, uint64_t* payload_bytes,
                                 double* kernel_ms) {
  if (!ctx || !launches || !payload_bytes || !kernel_ms || direction < 0 || direction > 1) return MORI_EINVAL;
  const int d = direction;
  double total = 0.0;
  for (uint32_t i = 0; i < ctx->prof_n[d]; ++i) {
    HIP_TRY(ctx, hipEventSynchronize(ctx->prof_ev[d][2 * i + 1]));
    float ms = 0.f;
    HIP_TRY(ctx, hipEventElapsedTime(&ms, ctx->prof_ev[d][2 * i], ctx->prof_ev[d][2 * i + 1]));
    total += ms;
  }
  if (int rc = fold_direct_bytes(ctx)) return rc;
  *launches = ctx->prof_n[d];
  *payload_bytes = ctx->prof_bytes[d];
  *kernel_ms = total;
  ctx->prof_n[d] = 0;
  ctx->prof_bytes[d] = 0;
  return MORI_OK;
}

extern "C" const char* mori_strerror(int code) {
  switch (code) {
    case MORI_OK: return "ok";
    case MORI_EINVAL: return "invalid argument";
    case MORI_ENOSPC: return "capacity exceeded";
    case MORI_ESTATE: return "call out of order";
    case MORI_EHIP: return "HIP runtime error";
    case MORI_EDEVICE: return "device-side validation failed";
    default: return "unknown error";
  }
}
