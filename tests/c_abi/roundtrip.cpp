// Standalone use of the C ABI: plain pointers and HIP runtime calls only, no
// Python and no torch.  Three rebalances of a seeded pool (boundary policy,
// Sec. 4.3 / Sec. 7.2: drawn windows, the reversed ranking, a smaller GPU
// budget with skip-fit), alternating the copy modes, each compared with the
// CPU oracle bit for bit: the plan (order, prefix, categories, summary), the
// block tables, tiers and free map, every byte of the resident pages and of
// the CPU tier's host buffers.  The swaps' kernel timing records (each
// direction's payload equals the plans' bytes), the typed eviction order of
// random KV blocks on both tiers (Sec. 4.3.2) and the multi-replica admission
// of a random Waiting queue with both rules (Sec. 4.1, Sec. 4.3.1), each
// against the same oracle.
//
//   roundtrip <programs> <seed>      exit status 0 when everything matches
#include <hip/hip_runtime.h>

#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <initializer_list>
#include <utility>
#include <vector>

#include "mori.h"
#include "mori_oracle.h"

namespace {

int failures = 0;

#define EXPECT(cond, ...)                          \
  do {                                             \
    if (!(cond)) {                                 \
      std::fprintf(stderr, "mismatch: " __VA_ARGS__); \
      std::fprintf(stderr, "\n");                  \
      ++failures;                                  \
    }                                              \
  } while (0)

#define HIP_OK(expr)                                                              \
  do {                                                                            \
    hipError_t e_ = (expr);                                                       \
    if (e_ != hipSuccess) {                                                       \
      std::fprintf(stderr, "%s: %s\n", #expr, hipGetErrorString(e_));             \
      std::exit(2);                                                               \
    }                                                                             \
  } while (0)

#define MORI_OK_(expr)                                                            \
  do {                                                                            \
    int rc_ = (expr);                                                             \
    if (rc_ != MORI_OK) {                                                         \
      std::fprintf(stderr, "%s: %s (%d)\n", #expr, mori_strerror(rc_), rc_);      \
      std::exit(2);                                                               \
    }                                                                             \
  } while (0)

// splitmix64: the seeded source of every input
struct Rng {
  uint64_t s;
  uint64_t next() {
    uint64_t z = (s += 0x9E3779B97F4A7C15ull);
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
  }
  uint32_t below(uint32_t n) { return (uint32_t)(next() % n); }
};

template <typename T>
T* dev_copy(const std::vector<T>& v) {
  T* d = nullptr;
  HIP_OK(hipMalloc(&d, v.empty() ? sizeof(T) : v.size() * sizeof(T)));
  if (!v.empty()) HIP_OK(hipMemcpy(d, v.data(), v.size() * sizeof(T), hipMemcpyHostToDevice));
  return d;
}

template <typename T>
std::vector<T> host_copy(const T* d, size_t n) {
  std::vector<T> v(n);
  if (n) HIP_OK(hipMemcpy(v.data(), d, n * sizeof(T), hipMemcpyDeviceToHost));
  return v;
}

}  // namespace

int main(int argc, char** argv) {
  const uint32_t P = argc > 1 ? (uint32_t)std::atoi(argv[1]) : 200;
  Rng rng{argc > 2 ? (uint64_t)std::atoll(argv[2]) : 1};
  const uint32_t L = 2, C = 2, T = 4, ROW = 64, K = 5;
  const uint64_t run = (uint64_t)T * ROW, LC = (uint64_t)L * C, block = LC * run;

  // programs on the GPU (55%) or the CPU tier, up to 24 blocks each
  std::vector<uint32_t> nblk(P), tbl_off(P + 1, 0);
  std::vector<uint8_t> tier(P);
  uint64_t gpu_blocks = 0;
  for (uint32_t p = 0; p < P; ++p) {
    nblk[p] = rng.below(25);
    tier[p] = rng.below(100) < 55 ? ORC_GPU : ORC_CPU;
    tbl_off[p + 1] = tbl_off[p] + nblk[p];
    if (tier[p] == ORC_GPU) gpu_blocks += nblk[p];
  }
  const uint32_t NB = (uint32_t)gpu_blocks + 37 + rng.below(300);
  const uint32_t tbl_len = tbl_off[P];
  // GPU programs own a random permutation's pages, the rest of the pool is free
  std::vector<uint32_t> perm(NB);
  for (uint32_t i = 0; i < NB; ++i) perm[i] = i;
  for (uint32_t i = NB; i > 1; --i) std::swap(perm[i - 1], perm[rng.below(i)]);
  std::vector<uint32_t> tbl(tbl_len, ORC_NONE);
  std::vector<uint8_t> free_map(NB, 1);
  uint32_t used = 0;
  for (uint32_t p = 0; p < P; ++p)
    if (tier[p] == ORC_GPU)
      for (uint32_t i = 0; i < nblk[p]; ++i) {
        tbl[tbl_off[p] + i] = perm[used];
        free_map[perm[used++]] = 0;
      }
  std::vector<uint8_t> pool((uint64_t)NB * block);
  for (auto& b : pool) b = (uint8_t)rng.next();
  // host buffers: one extent per program, [plane][block][run] bytes
  std::vector<uint64_t> ext(P + 1, 0);
  for (uint32_t p = 0; p < P; ++p) ext[p + 1] = ext[p] + ((nblk[p] * block + 255) & ~255ull);
  std::vector<std::vector<uint8_t>> obuf(P);
  for (uint32_t p = 0; p < P; ++p) {
    obuf[p].resize(nblk[p] * block);
    if (tier[p] == ORC_CPU)
      for (auto& b : obuf[p]) b = (uint8_t)rng.next();
  }
  std::printf("programs %u, blocks %u, pages %u, block %llu B\n", P, tbl_len, NB, (unsigned long long)block);

  // ---- the library's side: device state, context, pinned arena ----------
  HIP_OK(hipSetDevice(0));
  uint8_t* d_pool = dev_copy(pool);
  uint32_t* d_off = dev_copy(tbl_off);
  uint32_t* d_tbl = dev_copy(tbl);
  uint8_t* d_tier = dev_copy(tier);
  uint8_t* d_free = dev_copy(free_map);
  float* d_win = nullptr;
  HIP_OK(hipMalloc(&d_win, sizeof(float) * P * K * 2 + 16));
  hipStream_t s_out, s_in;
  HIP_OK(hipStreamCreateWithFlags(&s_out, hipStreamNonBlocking));
  HIP_OK(hipStreamCreateWithFlags(&s_in, hipStreamNonBlocking));
  mori_pool mp{L, C, T, ROW, NB, d_pool};
  mori_ctx* ctx = nullptr;
  // copy streams of its own only when this process has the hardware queues for them
  const char* hwq = std::getenv("GPU_MAX_HW_QUEUES");
  const uint32_t cflags = hwq && std::atoi(hwq) >= 8 ? MORI_CREATE_COPY_STREAMS : 0u;
  MORI_OK_(mori_create(&mp, P, 16 * block, cflags, &ctx));  // small staging: many chunks per direction
  void* arena = nullptr;
  MORI_OK_(mori_host_alloc(ext[P] + 256, &arena));
  MORI_OK_(mori_register(ctx, arena, ext[P] + 256));
  std::vector<uint64_t> host_addr(P);
  for (uint32_t p = 0; p < P; ++p) {
    host_addr[p] = (uint64_t)(uintptr_t)arena + ext[p];
    std::memcpy((void*)(uintptr_t)host_addr[p], obuf[p].data(), obuf[p].size());
  }

  // ---- windows: exact ties from a few dyadic values ----------------------
  const float vals[6] = {0.0f, 0.25f, 0.5f, 1.0f, 2.0f, 4.0f};
  std::vector<float> window((size_t)P * K * 2);
  for (auto& w : window) w = vals[rng.below(6)];
  uint64_t total = 0;
  for (uint32_t p = 0; p < P; ++p) total += nblk[p] * block;

  orc_geometry g{L, C, T, ROW, NB};
  std::vector<uint32_t> o_order(P), o_rank(P);
  std::vector<uint8_t> o_told(P), o_cat(P);
  std::vector<uint64_t> o_prefix(P);
  std::vector<uint8_t*> obuf_ptr(P);
  for (uint32_t p = 0; p < P; ++p) obuf_ptr[p] = obuf[p].data();

  MORI_OK_(mori_profile(ctx, 1));
  uint64_t moved[2] = {0, 0};  // plans' bytes per direction
  for (int step = 0; step < 3; ++step) {
    if (step == 1)  // the reversed ranking: each program's reasoning and tool time swap
      for (size_t i = 0; i < window.size(); i += 2) std::swap(window[i], window[i + 1]);
    const uint64_t gpu_budget = (step == 2 ? (uint64_t)NB * 3 / 10 : (uint64_t)NB / 2) * block;
    const uint32_t flags = step == 2 ? MORI_F_SKIP_FIT : 0u;
    const uint32_t mode = step == 1 ? MORI_COPY_KERNEL : MORI_COPY_CE;

    orc_summary os{};
    const int orc = orc_rebalance(&g, pool.data(), P, K, window.data(), nullptr, nullptr, tbl_off.data(), tbl_len,
                                  tbl.data(), tier.data(), free_map.data(), gpu_budget, total, 0, flags,
                                  obuf_ptr.data(), o_order.data(), o_rank.data(), o_told.data(), o_cat.data(),
                                  o_prefix.data(), &os);
    if (orc != ORC_OK) {
      std::fprintf(stderr, "oracle rejected step %d: %d\n", step, orc);
      return 2;
    }

    HIP_OK(hipMemcpy(d_win, window.data(), sizeof(float) * window.size(), hipMemcpyHostToDevice));
    mori_programs prog{P, K, d_win, nullptr, nullptr, d_off, tbl_len, d_tbl, d_tier, d_free};
    mori_budget budget{gpu_budget, total, flags, 0};
    MORI_OK_(mori_rank_partition(ctx, &prog, &budget, s_out));
    mori_plan plan{};
    MORI_OK_(mori_plan_wait(ctx, &plan));
    EXPECT(plan.m_gpu == os.m_gpu && plan.m_cpu == os.m_cpu, "step %d m_gpu/m_cpu", step);
    EXPECT(plan.n_out == os.n_out && plan.n_in == os.n_in, "step %d n_out/n_in", step);
    EXPECT(plan.bytes_out == os.bytes_out && plan.bytes_in == os.bytes_in, "step %d bytes", step);
    EXPECT(plan.pages_free_before == os.pages_free_before && plan.pages_released == os.pages_released &&
               plan.pages_recycled == os.pages_recycled && plan.pages_free_after == os.pages_free_after &&
               plan.pages_dropped == os.pages_dropped,
           "step %d page counts", step);
    EXPECT(plan.gpu_bytes_after == os.gpu_bytes_after && plan.cpu_bytes_after == os.cpu_bytes_after,
           "step %d tier bytes", step);
    for (uint32_t r = 0; r < P; ++r) {
      EXPECT(plan.order[r] == o_order[r] && plan.prefix[r] == o_prefix[r], "step %d rank %u", step, r);
      EXPECT(plan.category[r] == o_cat[r] && plan.tier_old[r] == o_told[r], "step %d program %u", step, r);
    }
    moved[0] += plan.bytes_out;
    moved[1] += plan.bytes_in;
    // the caller's part: nothing to place, every program keeps its extent
    MORI_OK_(mori_kv_swap_out(ctx, host_addr.data(), mode, s_out));
    MORI_OK_(mori_kv_swap_in(ctx, host_addr.data(), mode, s_in));
    HIP_OK(hipDeviceSynchronize());
    uint64_t dev_err = 1;
    MORI_OK_(mori_query(ctx, MORI_Q_DEVICE_ERROR, &dev_err));
    EXPECT(dev_err == 0, "step %d device error %llx", step, (unsigned long long)dev_err);

    const auto g_tbl = host_copy(d_tbl, tbl_len);
    const auto g_tier = host_copy(d_tier, P);
    const auto g_free = host_copy(d_free, NB);
    EXPECT(g_tbl == tbl, "step %d block tables", step);
    EXPECT(g_tier == tier, "step %d tiers", step);
    EXPECT(g_free == free_map, "step %d free map", step);
    const auto g_pool = host_copy(d_pool, pool.size());
    uint64_t pages = 0;
    for (uint32_t e = 0; e < tbl_len; ++e) {
      if (tbl[e] == ORC_NONE) continue;
      ++pages;
      for (uint64_t q = 0; q < LC; ++q) {
        const uint64_t o = (q * NB + tbl[e]) * run;
        if (std::memcmp(&g_pool[o], &pool[o], run) != 0) {
          EXPECT(false, "step %d page %u plane %llu bytes", step, tbl[e], (unsigned long long)q);
          break;
        }
      }
    }
    uint32_t cpu_programs = 0;
    for (uint32_t p = 0; p < P; ++p)
      if (tier[p] == ORC_CPU) {
        ++cpu_programs;
        EXPECT(std::memcmp((const void*)(uintptr_t)host_addr[p], obuf[p].data(), obuf[p].size()) == 0,
               "step %d host bytes of program %u", step, p);
      }
    std::printf("step %d (%s): out %u in %u, %llu resident pages and %u CPU-tier buffers compared\n", step,
                mode == MORI_COPY_KERNEL ? "kernel" : "copy engine", plan.n_out, plan.n_in,
                (unsigned long long)pages, cpu_programs);
  }

  for (int d = 0; d < 2; ++d) {  // kernel timing: one record per swap launch
    uint64_t launches = 0, payload = 0;
    double ms = -1.0;
    MORI_OK_(mori_profile_read(ctx, d, &launches, &payload, &ms));
    EXPECT(payload == moved[d], "direction %d profiled payload %llu of %llu", d, (unsigned long long)payload,
           (unsigned long long)moved[d]);
    EXPECT((launches > 0) == (moved[d] > 0) && ms >= 0.0, "direction %d launches %llu", d,
           (unsigned long long)launches);
    MORI_OK_(mori_profile_read(ctx, d, &launches, &payload, &ms));  // a read clears the record
    EXPECT(launches == 0 && payload == 0, "direction %d record not cleared", d);
  }
  std::printf("profiling: %llu B out, %llu B in recorded\n", (unsigned long long)moved[0],
              (unsigned long long)moved[1]);
  MORI_OK_(mori_destroy(ctx));

  // ---- typed eviction order of random KV blocks, both tiers ----------------
  {
    const uint32_t N = 3000 + rng.below(5000);
    std::vector<uint8_t> type(N);
    std::vector<uint64_t> last(N);
    std::vector<uint32_t> size(N);
    uint64_t total = 0;
    for (uint32_t i = 0; i < N; ++i) {  // runs of blocks sharing a program's label and, often, its time
      const bool fresh = i == 0 || rng.below(8) == 0;
      type[i] = fresh ? (uint8_t)rng.below(3) : type[i - 1];
      last[i] = fresh || rng.below(2) ? rng.next() >> 24 : last[i - 1];
      size[i] = 1 + rng.below(16);
      total += size[i];
    }
    const uint8_t* d_type = dev_copy(type);
    const uint64_t* d_last = dev_copy(last);
    const uint32_t* d_size = dev_copy(size);
    uint64_t ws_bytes = 0;
    MORI_OK_(mori_evict_workspace(N, &ws_bytes));
    void* ws = nullptr;
    uint32_t *d_order = nullptr, *d_result = nullptr;
    uint64_t* d_prefix = nullptr;
    HIP_OK(hipMalloc(&ws, ws_bytes));
    HIP_OK(hipMalloc(&d_order, 4ull * N));
    HIP_OK(hipMalloc(&d_prefix, 8ull * N));
    HIP_OK(hipMalloc(&d_result, 8));
    const mori_blocks blocks{N, d_type, d_last, d_size, 4096};
    for (uint32_t tier_e : {MORI_TIER_GPU, MORI_TIER_CPU}) {
      const uint64_t need = (uint64_t)rng.below((uint32_t)total + 1) * 4096;
      MORI_OK_(mori_evict_order(&blocks, tier_e, need, ws, ws_bytes, d_order, d_prefix, d_result, s_out));
      HIP_OK(hipStreamSynchronize(s_out));
      std::vector<uint32_t> o_ord(N);
      std::vector<uint64_t> o_pre(N);
      uint32_t o_count = 0;
      EXPECT(orc_evict_order(N, type.data(), last.data(), size.data(), 4096, tier_e, need, o_ord.data(),
                             o_pre.data(), &o_count) == ORC_OK,
             "oracle eviction order");
      const auto g_ord = host_copy(d_order, N);
      const auto g_pre = host_copy(d_prefix, N);
      const auto g_res = host_copy(d_result, 2);
      EXPECT(g_ord == o_ord && g_pre == o_pre, "eviction order tier %u", tier_e);
      EXPECT(g_res[0] == o_count && g_res[1] == 0, "eviction count tier %u: %u vs %u", tier_e, g_res[0], o_count);
      std::printf("eviction order: %u blocks, tier %u, %u evictions free %llu B\n", N, tier_e, g_res[0],
                  (unsigned long long)need);
    }
    for (void* d : {ws, (void*)d_order, (void*)d_prefix, (void*)d_result, (void*)d_type, (void*)d_last,
                    (void*)d_size})
      HIP_OK(hipFree(d));
  }

  // ---- multi-replica admission of a Waiting queue (host memory) -----------
  {
    const uint32_t W = 300, R = 8;
    std::vector<uint64_t> bytes(W), room(R);
    std::vector<float> iota(W);
    std::vector<uint8_t> st(W);
    uint64_t want = 0;
    for (uint32_t p = 0; p < W; ++p) {
      bytes[p] = (uint64_t)(1 + rng.below(64)) << 21;
      iota[p] = (float)rng.below(1001) / 1000.0f;
      st[p] = (uint8_t)rng.below(3);
      want += bytes[p];
    }
    for (uint32_t r = 0; r < R; ++r) room[r] = (uint64_t)rng.below((uint32_t)(want >> 21) / 4 + 1) << 21;
    for (uint32_t flags_a : {0u, (uint32_t)MORI_ADMIT_BEST_FIT}) {
      std::vector<int32_t> rep_g(W), rep_o(W);
      std::vector<uint64_t> after_g(R), after_o(R);
      MORI_OK_(mori_replica_admit(W, bytes.data(), iota.data(), st.data(), R, room.data(), flags_a, rep_g.data(),
                                  after_g.data()));
      EXPECT(orc_replica_admit(W, bytes.data(), iota.data(), st.data(), R, room.data(), flags_a, rep_o.data(),
                               after_o.data()) == ORC_OK,
             "oracle replica admission");
      EXPECT(rep_g == rep_o && after_g == after_o, "replica admission flags %u", flags_a);
      uint32_t admitted = 0;
      for (int32_t r : rep_g) admitted += r >= 0;
      std::printf("replica admission (%s): %u of %u waiting programs placed on %u replicas\n",
                  flags_a ? "best fit" : "most room", admitted, W, R);
    }
  }
  MORI_OK_(mori_host_free(arena));
  HIP_OK(hipStreamDestroy(s_out));
  HIP_OK(hipStreamDestroy(s_in));
  for (void* d : {(void*)d_pool, (void*)d_off, (void*)d_tbl, (void*)d_tier, (void*)d_free, (void*)d_win})
    HIP_OK(hipFree(d));
  std::printf(failures ? "FAILED: %d mismatches\n" : "ok\n", failures);
  return failures ? 1 : 0;
}
