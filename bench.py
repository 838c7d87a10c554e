#!/usr/bin/env python3
"""Benchmark of the KV tier-migration hot path on one MI355X.

One step = one whole rebalance: Eq. 1 idleness -> ranking -> GPU/CPU/Waiting
boundaries -> sticky diff and page allocation -> swap-out (GPU -> pinned host)
concurrently with swap-in (pinned host -> GPU) on two streams.

The headline workload is the compressed-latent (MLA-style) one, the largest
that fits one GPU (256 programs, a 155 GiB pool, 72 KiB runs).  Its schedule
rotates the tiers through idleness windows: every step each program gets
windows of its current tier's set (CPU tier busy, GPU tier middle, Waiting
idle, redrawn per step), so the kernel computes Eq. 1 on the device every
step and the CPU tier comes back while as many bytes leave the GPU.  The
Llama-3-8B workload follows as a second leg (drawn and reversed windows,
alternating).

value = KV migration GB/s = (bytes swapped out + bytes swapped in) / step wall
time, with the pool, tables and windows already resident in HBM and the CPU
tier already in pinned host memory when the timed region starts.  The
host-link peaks (pinned hipMemcpyAsync: D2H, H2D, and both directions at
once as chunk streams, rate over the window where both run) and the HBM copy
peak are measured in the same run.  The roofline object is for the
gather/scatter kernel (HBM-bound), timed per launch with events on its stream.
"""
from __future__ import annotations

import os
import sys

# Hardware queues per process (HIP's default is four): with eight, the two swap
# streams and libmori's two copy streams each get a queue of their own.  Must
# be set before the HIP runtime starts (it overrides the environment's value);
# --hw-queues 4 runs the in-order copy path instead.
_HWQ = "8"
for _i, _a in enumerate(sys.argv[:-1]):
    if _a == "--hw-queues":
        _HWQ = sys.argv[_i + 1]
os.environ["GPU_MAX_HW_QUEUES"] = _HWQ

import argparse
import ctypes as C
import json
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

GIB = 1 << 30
HBM_PEAK_GBPS = 8000.0  # MI355X HBM3E, published


def log(msg: str) -> None:
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=6)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--workload", default="mla")
    ap.add_argument("--scale", type=float, default=None,
                    help="context scale (churn: default 0.32, a ~120 GiB pool; others: 1)")
    ap.add_argument("--schedule", default=None, choices=["reverse", "rotate"],
                    help="reverse: steps alternate drawn and reversed windows; rotate: each step every program "
                         "gets windows of its tier's set (CPU busy, GPU middle, Waiting idle), so both directions "
                         "move every step (default: rotate for mla, reverse otherwise)")
    ap.add_argument("--extra", default="llama3_8b",
                    help="comma-separated workloads timed after the headline one ('' for none)")
    ap.add_argument("--extra-steps", type=int, default=4)
    ap.add_argument("--mode", default="auto", choices=["auto", "kernel", "ce"])
    ap.add_argument("--arena-gib", type=float, default=60.0, help="pinned CPU-tier arena")
    ap.add_argument("--cpu-gib", type=float, default=28.0, help="CPU-tier budget")
    ap.add_argument("--staging-mib", type=int, default=2048, help="per direction, two halves")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-verify", action="store_true")
    ap.add_argument("--no-evict", action="store_true", help="skip the typed eviction-order leg")
    ap.add_argument("--no-plan", action="store_true", help="skip the rank/partition latency leg")
    ap.add_argument("--cpu-seconds", type=float, default=12.0)
    ap.add_argument("--hw-queues", type=int, default=8, help="GPU_MAX_HW_QUEUES for this process (read at start)")
    ap.add_argument("--serial-swaps", action="store_true",
                    help="for kernel traces: the swap-in on the swap-out's stream, so (with --hw-queues 4) every "
                         "kernel and copy runs in order and no kernel shares the GPU with another (not a "
                         "throughput configuration)")
    return ap.parse_args()


# --------------------------------------------------------------------------
# CPU baseline: the oracle, as it stands, on a bounded sample of the workload
# --------------------------------------------------------------------------
# tier -> rotation window set: GPU middle, CPU busy, Waiting (and SSD) idle
ROT_SET_OF_TIER = (1, 0, 2, 2)


def schedule_windows(np, inst, schedule: str, steps: int):
    """Host windows of step t given the tiers before it: 'reverse' alternates
    the drawn and the reversed windows (every program's reasoning and tool
    times swapped); 'rotate' gives each program a window of its tier's set."""
    from workload import rotation_windows

    if schedule == "rotate":
        rot = rotation_windows(inst.seed, inst.P, steps)
        sel = np.array(ROT_SET_OF_TIER)
        ar = np.arange(inst.P)
        return lambda t, tier: np.ascontiguousarray(rot[t % steps][sel[tier], ar])
    wins = (np.ascontiguousarray(inst.window), inst.window[:, :, ::-1].copy())
    return lambda t, tier: wins[t % 2]


def cpu_baseline(cfg, schedule: str, cpu_frac: float, seconds: float, evict_sizes=(), plan_cases=()):
    import numpy as np

    from oracle import oracle
    from workload import budget_bytes, fill_pool_np, make_bank, make_instance

    scale = 1.0 / 32
    inst = make_instance(cfg, scale=scale)
    g = inst.geom
    bank = make_bank(cfg.seed, cfg.dtype, g.run_bytes)
    pool = fill_pool_np(inst, bank)
    bufs = [np.zeros(int(n) * g.block_bytes, np.uint8) for n in inst.nblk]
    tbl, tier, free = inst.copy_state()
    bg = budget_bytes(inst.total_bytes, cfg.gpu_pct)
    bc = int(inst.total_bytes * cpu_frac)
    window_of = schedule_windows(np, inst, schedule, 256)
    moved, spent, steps = 0, 0.0, 0
    t = 0
    while True:
        w = window_of(t, tier)
        t0 = time.perf_counter()
        res = oracle.rebalance(g, window=w, tbl_off=inst.tbl_off, tbl=tbl, tier=tier, free_map=free,
                               gpu_budget=bg, cpu_budget=bc, pool=pool, host_bufs=bufs)
        dt = time.perf_counter() - t0
        assert res.rc == oracle.OK
        if t >= 1:  # the first step only moves out; time the bidirectional ones
            moved += res.summary["bytes_out"] + res.summary["bytes_in"]
            spent += dt
            steps += 1
        t += 1
        if spent >= seconds or t > 200:
            break
    out = {"value": round(moved / spent / 1e9, 3), "unit": "GB/s", "cores": 1, "kind": "oracle",
           "sample": (f"{cfg.name} with contexts scaled by {scale:g} ({inst.P} programs, "
                      f"{inst.total_bytes / GIB:.2f} GiB of KV, same GPU/CPU budget fractions, {schedule} "
                      f"schedule), {steps} bidirectional rebalances, memcpy per run between host buffers, "
                      f"single thread")}
    # the same oracle on all of this process's cores: one thread per core, each
    # rebalancing its own copy of a smaller sample (the C oracle runs outside
    # the GIL and shares no state between calls)
    import threading

    threads = max(1, min(16, len(os.sched_getaffinity(0))))
    small = make_instance(cfg, scale=1.0 / 128)
    sg = small.geom
    sbank = make_bank(cfg.seed, cfg.dtype, sg.run_bytes)
    sbg = budget_bytes(small.total_bytes, cfg.gpu_pct)
    sbc = int(small.total_bytes * cpu_frac)
    swindow_of = schedule_windows(np, small, schedule, 256)
    moved_t = [0] * threads
    stop = threading.Event()

    errors = []

    def worker(w):
        try:
            pool_w = fill_pool_np(small, sbank)
            bufs_w = [np.zeros(int(n) * sg.block_bytes, np.uint8) for n in small.nblk]
            tbl_w, tier_w, free_w = small.copy_state()
            ready.wait(timeout=300)
            t = 0
            while not stop.is_set():
                r = oracle.rebalance(sg, window=swindow_of(t, tier_w), tbl_off=small.tbl_off, tbl=tbl_w, tier=tier_w,
                                     free_map=free_w, gpu_budget=sbg, cpu_budget=sbc, pool=pool_w, host_bufs=bufs_w)
                if t >= 1 and not stop.is_set():
                    moved_t[w] += r.summary["bytes_out"] + r.summary["bytes_in"]
                t += 1
        except Exception as e:  # a failed worker ends the measurement instead of hanging it
            errors.append(repr(e))
            ready.abort()

    ready = threading.Barrier(threads + 1)
    pool_threads = [threading.Thread(target=worker, args=(w,), daemon=True) for w in range(threads)]
    for th in pool_threads:
        th.start()
    try:
        ready.wait(timeout=300)
        t0 = time.perf_counter()
        time.sleep(min(seconds, 8.0))
    except threading.BrokenBarrierError:
        t0 = time.perf_counter()
    stop.set()
    span = time.perf_counter() - t0
    for th in pool_threads:
        th.join()
    model = ""
    try:
        model = next(l.split(":", 1)[1].strip() for l in open("/proc/cpuinfo") if l.startswith("model name"))
    except (OSError, StopIteration):
        pass
    out["value_all_threads"] = None if errors else round(sum(moved_t) / span / 1e9, 3)
    if errors:
        out["all_threads_error"] = errors[0]
    out["threads"] = threads
    out["cpu_model"] = model
    out["sample_all_threads"] = (f"{threads} threads, each rebalancing its own copy of {cfg.name} with contexts "
                                 f"scaled by 1/128 ({small.P} programs, {small.total_bytes / GIB:.2f} GiB of KV) "
                                 f"for {span:.1f} s; steps still running at the end are not counted")
    # the oracle on the inputs of the eviction-order and rank/partition legs
    out["evict_order_us"] = {}
    for N in evict_sizes:
        typ, la, size, need = evict_inputs(np, N)
        t0 = time.perf_counter()
        rc, *_ = oracle.evict_order(typ, la, 0, need, size=size, unit_bytes=4096)
        out["evict_order_us"][str(N)] = round((time.perf_counter() - t0) * 1e6, 1)
        assert rc == oracle.OK
    out["replica_admit_us"] = []
    for P, R in REPLICA_CASES:
        sizes, iota, status, room = replica_inputs(np, P, R)
        for rule, flags in (("most room", 0), ("best fit", oracle.ADMIT_BEST_FIT)):
            t0 = time.perf_counter()
            rc, *_ = oracle.replica_admit(sizes, iota, status, room, flags)
            out["replica_admit_us"].append({"programs": P, "replicas": R, "rule": rule,
                                            "us": round((time.perf_counter() - t0) * 1e6, 1)})
            assert rc == oracle.OK
    out["plan_us"] = []
    for label, geom, src, gb, cb, status, wins in plan_cases:
        for policy, flags, sfrac in POLICIES:
            tbl, tier, free = src.copy_state()
            t0 = time.perf_counter()
            res = oracle.rebalance(geom, window=wins[0], status=status, tbl_off=src.tbl_off, tbl=tbl, tier=tier,
                                   free_map=free, gpu_budget=gb, cpu_budget=cb, flags=flags,
                                   ssd_budget=ssd_budget(src, sfrac))
            out["plan_us"].append({"case": label, "policy": policy,
                                   "us": round((time.perf_counter() - t0) * 1e6, 1)})
            assert res.rc == oracle.OK
    return out


# --------------------------------------------------------------------------
# peaks measured in the same run
# --------------------------------------------------------------------------
def bytes_done_by(ends, w: float, chunk: int) -> float:
    """Bytes a stream of equal chunks, started at time 0 and ending at the
    given times, had moved by time w: the chunks ended by then, plus the
    share of the one under way that its own span puts before w."""
    prev = 0.0
    for c, e in enumerate(ends):
        if e > w:
            return (c + (w - prev) / max(e - prev, 1e-12)) * chunk
        prev = e
    return float(len(ends) * chunk)


# --------------------------------------------------------------------------
# --------------------------------------------------------------------------
def measure_peaks(torch, M, s1, s2):
    # the HIP runtime torch already loaded (a second copy of the runtime must never be loaded)
    hip = C.CDLL("libamdhip64.so.7", mode=os.RTLD_NOLOAD | os.RTLD_GLOBAL)
    hip.hipMemcpyAsync.argtypes = [C.c_void_p, C.c_void_p, C.c_size_t, C.c_int, C.c_void_p]
    H2D, D2H, D2D = 1, 2, 3
    n = 4 * GIB
    dev_a = torch.empty(n, dtype=torch.uint8, device="cuda")
    dev_b = torch.empty(n, dtype=torch.uint8, device="cuda")
    dev_a.fill_(1)
    dev_b.fill_(2)
    rc1, h1 = M.mori_host_alloc(n)
    rc2, h2 = M.mori_host_alloc(n)
    assert rc1 == 0 and rc2 == 0
    C.memset(h1, 3, n)
    C.memset(h2, 4, n)

    def timed(fn, reps=5):
        ts = []
        for _ in range(reps):
            torch.cuda.synchronize()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(s1)
            s2.wait_event(e0)
            fn()
            e2 = torch.cuda.Event()
            e2.record(s2)
            s1.wait_event(e2)
            e1.record(s1)
            e1.synchronize()
            ts.append(e0.elapsed_time(e1) / 1e3)
        return sorted(ts)[len(ts) // 2]

    def cp(dst, src, kind, s):
        assert hip.hipMemcpyAsync(dst, src, n, kind, C.c_void_p(s.cuda_stream)) == 0

    t_d2h = timed(lambda: cp(h1, dev_a.data_ptr(), D2H, s1))
    t_h2d = timed(lambda: cp(dev_b.data_ptr(), h2, H2D, s1))
    t_bi = timed(lambda: (cp(h1, dev_a.data_ptr(), D2H, s1), cp(dev_b.data_ptr(), h2, H2D, s2)))

    # Both directions at once, as streams of copies (D2H on s1, H2D on s2,
    # started together, 16 GiB each way cycling over the 4 GiB buffers), each
    # copy's end recorded by an event on its stream.  The rate is taken over
    # the window in which both directions run: from the start to the end of
    # the direction that finishes first, counting the bytes each direction
    # completed inside it (the copy that straddles the window's end counted
    # pro rata over its own span).  Two copy sizes (the swaps' copies range
    # up to a 1 GiB staging half); the better median is the peak.
    stream_bytes = 4 * n
    steady = {}
    for chunk in (256 << 20, 1 << 30):
        nch = stream_bytes // chunk
        per_buf = n // chunk
        runs = []
        for _ in range(5):
            torch.cuda.synchronize()
            e0 = torch.cuda.Event(enable_timing=True)
            ev_d = [torch.cuda.Event(enable_timing=True) for _ in range(nch)]
            ev_h = [torch.cuda.Event(enable_timing=True) for _ in range(nch)]
            e0.record(s1)
            s2.wait_event(e0)
            for c in range(nch):
                o = (c % per_buf) * chunk
                assert hip.hipMemcpyAsync(h1 + o, dev_a.data_ptr() + o, chunk, D2H, C.c_void_p(s1.cuda_stream)) == 0
                ev_d[c].record(s1)
                assert hip.hipMemcpyAsync(dev_b.data_ptr() + o, h2 + o, chunk, H2D, C.c_void_p(s2.cuda_stream)) == 0
                ev_h[c].record(s2)
            torch.cuda.synchronize()
            td = [e0.elapsed_time(e) / 1e3 for e in ev_d]
            th = [e0.elapsed_time(e) / 1e3 for e in ev_h]
            w = min(td[-1], th[-1])
            bd, bh = bytes_done_by(td, w, chunk), bytes_done_by(th, w, chunk)
            runs.append(((bd + bh) / w, bd / w, bh / w))
        steady[chunk] = sorted(runs)[2]
    best = max(steady, key=lambda k: steady[k][0])
    t_d2d = timed(lambda: cp(dev_b.data_ptr(), dev_a.data_ptr(), D2D, s1))
    torch.cuda.synchronize()
    M.mori_host_free(h1)
    M.mori_host_free(h2)
    del dev_a, dev_b
    torch.cuda.empty_cache()
    return {"d2h_GBps": round(n / t_d2h / 1e9, 2), "h2d_GBps": round(n / t_h2d / 1e9, 2),
            "bidir_pair_GBps": round(2 * n / t_bi / 1e9, 2), "bidir_GBps": round(steady[best][0] / 1e9, 2),
            "bidir_split_GBps": {"d2h": round(steady[best][1] / 1e9, 2), "h2d": round(steady[best][2] / 1e9, 2)},
            "bidir_by_copy_GBps": {f"{k >> 20} MiB": round(v[0] / 1e9, 2) for k, v in steady.items()},
            "d2d_copy_GBps": round(2 * n / t_d2d / 1e9, 1),
            "method": ("pinned hipMemcpyAsync, 4 GiB per direction, median of 5.  bidir_pair: one D2H and one H2D "
                       "copy started together on two streams, 8 GiB over the time both took.  bidir: D2H and H2D "
                       "started together as streams of 16 GiB each in 256 MiB or 1 GiB copies with an event after "
                       "each, bytes both directions completed while both ran over the time until the first of them "
                       "finished, the better copy size (bidir_by_copy; bidir_split: each direction's share)")}


def link_bound_s(out_bytes: int, in_bytes: int, peaks: dict) -> float:
    """Lower bound on the time of one step's D2H and H2D bytes on the measured
    link: neither direction beats its one-direction rate and both together do
    not beat the two-way capacity."""
    return max(out_bytes / (peaks["d2h_GBps"] * 1e9), in_bytes / (peaks["h2d_GBps"] * 1e9),
               (out_bytes + in_bytes) / (peaks["bidir_GBps"] * 1e9))


def split_model_s(out_bytes: int, in_bytes: int, peaks: dict) -> float:
    """Time of one step's copies if both directions start together and run
    flat out: at the two-way split measured in the same run (bidir_split)
    until the smaller direction is done, then the larger one alone at its
    one-direction rate.  A model of two unpaced copy streams, not a bound
    (pacing the smaller direction could beat it when the two differ)."""
    rd, rh = peaks["bidir_split_GBps"]["d2h"] * 1e9, peaks["bidir_split_GBps"]["h2d"] * 1e9
    alone_d, alone_h = peaks["d2h_GBps"] * 1e9, peaks["h2d_GBps"] * 1e9
    if out_bytes == 0 or in_bytes == 0:
        return out_bytes / alone_d + in_bytes / alone_h
    t_d, t_h = out_bytes / rd, in_bytes / rh
    if t_d <= t_h:
        return t_d + (in_bytes - rh * t_d) / alone_h
    return t_h + (out_bytes - rd * t_h) / alone_d


def evict_inputs(np, N):
    """Synthetic block metadata of the eviction-order leg (Sec. 4.3.2): N
    blocks of 1024 programs, half the timestamps tied, variable block sizes,
    a request to free a quarter of the bytes."""
    from workload import eviction_blocks

    rng = np.random.default_rng(N)
    typ, la, size = eviction_blocks(rng, N, programs=1024, tie_frac=0.5, var_size=True)
    need = int(size.astype(np.int64).sum()) * 4096 // 4
    return typ, la, size, need


def evict_leg(torch, np, M, sizes, reps=20):
    """Typed eviction order (Sec. 4.3.2) of the GPU tier: device time per call
    (events on its stream, median of `reps`).  Exact parity with the oracle at
    these sizes is a GPU test; the oracle's time is in the CPU baseline."""
    out = []
    for N in sizes:
        typ, la, size, need = evict_inputs(np, N)
        t = torch.from_numpy(typ).cuda()
        la_d = torch.from_numpy(la.view(np.int64)).cuda()
        sz = torch.from_numpy(size.view(np.int32)).cuda()
        _, wb = M.mori_evict_workspace(N)
        ws = torch.empty(wb, dtype=torch.uint8, device="cuda")
        order = torch.empty(N, dtype=torch.int32, device="cuda")
        prefix = torch.empty(N, dtype=torch.int64, device="cuda")
        res = torch.zeros(2, dtype=torch.int32, device="cuda")
        blk = M.mori_blocks(N, t.data_ptr(), la_d.data_ptr(), sz.data_ptr(), 4096)
        s = torch.cuda.current_stream()
        times = []
        for _ in range(reps + 2):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(s)
            assert M.mori_evict_order(blk, 0, need, ws.data_ptr(), wb, order.data_ptr(), prefix.data_ptr(),
                                      res.data_ptr(), s.cuda_stream) == 0
            e1.record(s)
            e1.synchronize()
            times.append(e0.elapsed_time(e1) * 1e3)
        us = sorted(times[2:])[reps // 2]
        assert int(res[1]) == 0, "eviction order rejected its input"
        out.append({"blocks": N, "us": round(us, 1), "Mblocks_per_s": round(N / us, 1), "evictions": int(res[0])})
    return out


def plan_cases(np, inst, bg, bc):
    """Inputs of the rank/partition leg: the workload's programs, tables and
    pool pages, and 4096 random programs, each with statuses (busy programs
    Reasoning, idle ones Acting, a third of Waiting new arrivals) and the drawn
    and reversed windows.  The step never touches KV bytes, so pages are 16 B."""
    from workload import Geometry, random_instance

    bb = inst.geom.block_bytes
    rng = np.random.default_rng(4096)
    big = random_instance(rng, P=4096, max_blocks=64, geom=Geometry(1, 1, 1, 16, 0), ties=False,
                          tier_p=(0.5, 0.3, 0.2), extra_free=20000)
    cases = []
    for label, geom, src, gb, cb in (
            (f"{inst.name} programs and pages", Geometry(1, 1, 1, 16, inst.geom.num_blocks), inst, bg // bb * 16,
             bc // bb * 16),
            ("4096 programs", big.geom, big, big.total_bytes // 2 // 16 * 16, big.total_bytes // 4 // 16 * 16)):
        status = np.where(src.busy, 0, 1).astype(np.uint8)
        status[(src.tier == 2) & (np.arange(src.P) % 3 == 0)] = 2
        wins = [np.ascontiguousarray(src.window), src.window[:, :, ::-1].copy()]
        cases.append((label, geom, src, gb, cb, status, wins))
    return cases


# (name, flags, SSD budget as a fraction of the case's KV bytes): the boundary
# policy, the incremental policy (MORI_F_INCREMENTAL) and three tiers
# (MORI_F_SSD_TIER, the SSD tier a quarter of the KV bytes)
POLICIES = (("boundary", 0, 0.0), ("incremental", 8, 0.0), ("three-tier", 16, 0.25))


def ssd_budget(src, frac: float) -> int:
    """SSD budget of a plan case, in its 16-byte pages."""
    return int(src.total_bytes // max(src.geom.block_bytes, 1) * frac) * 16


def plan_leg(torch, np, M, cases, reps=30):
    """The rank/partition step alone (Eq. 1, ranking, the boundary policy, the
    incremental policy or three tiers, page allocation, table rewrite), which is
    latency-bound:
    device time of mori_rank_partition (events on its stream, median of `reps`
    calls alternating the two windows, each followed by its plan on the host).
    Exact parity with the oracle on these inputs is a GPU test; the oracle's
    time is in the CPU baseline."""
    from paper_2606_00866_amd.tiering import TierPool

    out = []
    for label, geom, src, gb, cb, status, wins in cases:
        st_d = torch.from_numpy(status).cuda()
        wins_d = [torch.from_numpy(w).cuda() for w in wins]
        for policy, flags, sfrac in POLICIES:
            tp = TierPool(geom, src.tbl_off, src.tbl, src.tier, src.free_map, arena_bytes=64 << 20,
                          max_programs=src.P, staging_bytes=1 << 20)
            sb = ssd_budget(src, sfrac)
            s = torch.cuda.current_stream()
            times = []
            for i in range(reps + 2):
                e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                e0.record(s)
                assert tp.rank_partition(gpu_bytes=gb, cpu_bytes=cb, window=wins_d[i % 2], status=st_d,
                                         flags=flags, stream=s, ssd_bytes=sb) == 0
                e1.record(s)
                rc, p = tp.plan_wait()
                assert rc == 0, (label, policy, rc, p.device_error)
                e1.synchronize()
                times.append(e0.elapsed_time(e1) * 1e3)
            tp.close()
            out.append({"case": label, "programs": src.P, "pages": geom.num_blocks, "policy": policy,
                        "us": round(sorted(times[2:])[reps // 2], 1)})
    return out


REPLICA_CASES = ((4096, 8), (4096, 64))  # (Waiting programs, replicas)


def replica_inputs(np, P: int, R: int):
    """A shared Waiting queue for multi-replica admission: P programs with
    lognormal KV sizes (whole 2 MiB blocks), random idleness, a quarter Acting
    (they stay), a third of the rest new arrivals; R replicas whose free GPU
    room totals about half the queue's bytes."""
    rng = np.random.default_rng(P * 1000 + R)
    blocks = np.clip(np.exp(np.log(2048) + 0.5 * rng.standard_normal(P)), 256, 16384).astype(np.int64)
    sizes = (blocks * (2 << 20)).astype(np.uint64)
    iota = rng.random(P).astype(np.float32)
    status = np.where(rng.random(P) < 0.25, 1, np.where(rng.random(P) < 1 / 3, 2, 0)).astype(np.uint8)
    room = (rng.random(R) * 2 * sizes.sum() * 0.5 / R).astype(np.uint64)
    return sizes, iota, status, room


def replica_leg(np, M, reps=20):
    """Multi-replica admission of the shared Waiting queue (host code behind the
    ABI): median wall time of `reps` calls, both replica rules.  Parity with the
    oracle on these inputs is a CPU test; the oracle's time is in the CPU baseline."""
    out = []
    for P, R in REPLICA_CASES:
        sizes, iota, status, room = replica_inputs(np, P, R)
        for rule, flags in (("most room", 0), ("best fit", M.MORI_ADMIT_BEST_FIT)):
            times = []
            for _ in range(reps):
                t0 = time.perf_counter()
                rc, rep_, after = M.mori_replica_admit(sizes, iota, status, room, flags)
                times.append((time.perf_counter() - t0) * 1e6)
                assert rc == 0
            out.append({"programs": P, "replicas": R, "rule": rule, "admitted": int((rep_ >= 0).sum()),
                        "us": round(sorted(times)[reps // 2], 1)})
    return out


def stored_traffic(workload: str, direction: int):
    """HBM bytes per launch of the swap kernel from the committed counter
    summary, or None when that summary is for another workload or the kernel
    source has changed since the counters were taken."""
    import hashlib

    path = os.path.join(ROOT, "profiles", f"swap_kernel_{workload}_pmc.md")
    if not os.path.exists(path):
        return None
    line = [l for l in open(path) if l.startswith("traffic_json: ")]
    if not line:
        return None
    rec = json.loads(line[0][len("traffic_json: "):])
    src = os.path.join(ROOT, "paper_2606_00866_amd", "csrc", "swap_kernels.hip")
    if hashlib.sha256(open(src, "rb").read()).hexdigest() != rec["kernel_source_sha256"]:
        return None
    return rec["gather" if direction == 0 else "scatter"]["traffic_bytes_per_launch"]


def run_workload(args, name, schedule, steps, warmup, s_out, s_in, peaks, torch, np, M):
    """Times `steps` rebalances of one workload (after `warmup` untimed ones)
    and checks the final state; the pool and the CPU tier are freed before it
    returns."""
    from paper_2606_00866_amd.tiering import TierPool, check
    from workload import CONFIGS, budget_bytes, churn_steps, fill_pool_torch, make_bank, make_instance

    cfg = CONFIGS[name]
    churn = cfg.name == "churn"  # 1024 programs, nothing placed yet, budget swinging, phases flipping
    scale = args.scale if args.scale is not None else (0.32 if churn else 1.0)
    inst = make_instance(cfg, scale=scale, resident="wait" if churn else "gpu")
    g = inst.geom
    total = inst.total_bytes
    bg = budget_bytes(total, cfg.gpu_pct)
    bc = int(args.cpu_gib * GIB)
    # churn: step 0 places the first partition; step t >= 1 takes the t-th budget and windows
    churn_inputs = ([(budget_bytes(total, pct), w) for _, pct, _, w in
                     churn_steps(cfg, inst.busy, steps=warmup + steps)] if churn else None)
    log(f"workload {cfg.name}: P={inst.P} NB={g.num_blocks} block={g.block_bytes} B total={total / GIB:.2f} GiB "
        f"gpu_budget={bg / GIB:.2f} GiB cpu_budget={bc / GIB:.2f} GiB schedule={schedule}")

    free_b, _ = torch.cuda.mem_get_info()
    need = g.pool_bytes + 2 * args.staging_mib * (1 << 20) + (2 << 30)
    if free_b < need:
        raise SystemExit(f"pool needs {need / GIB:.1f} GiB of HBM, {free_b / GIB:.1f} GiB free")
    t0 = time.perf_counter()
    pool = torch.empty(g.pool_bytes, dtype=torch.uint8, device="cuda")
    bank = make_bank(cfg.seed, cfg.dtype, g.run_bytes)
    bank_dev = torch.from_numpy(bank.view(np.int16)).cuda()
    fill_pool_torch(pool, inst, bank_dev)
    torch.cuda.synchronize()
    log(f"pool {g.pool_bytes / GIB:.2f} GiB filled in {time.perf_counter() - t0:.1f} s")
    tp = TierPool(g, inst.tbl_off, inst.tbl, inst.tier, inst.free_map, arena_bytes=int(args.arena_gib * GIB),
                  max_programs=inst.P, staging_bytes=args.staging_mib << 20, pool=pool)
    mode = {"auto": M.MORI_COPY_AUTO, "kernel": M.MORI_COPY_KERNEL, "ce": M.MORI_COPY_CE}[args.mode]
    wins = [torch.from_numpy(inst.window).cuda(), torch.from_numpy(inst.window[:, :, ::-1].copy()).cuda()]
    if schedule == "rotate":
        from workload import rotation_windows

        # every step's three window sets, resident before the timed region
        rot = torch.from_numpy(rotation_windows(cfg.seed, inst.P, warmup + steps)).cuda()
        rot_sel = torch.tensor(ROT_SET_OF_TIER, dtype=torch.int64, device="cuda")
        prog_ids = torch.arange(inst.P, device="cuda")
    if churn:
        churn_inputs = [(b, torch.from_numpy(np.ascontiguousarray(w)).cuda()) for b, w in churn_inputs]
    step_bg = [bg]  # the GPU budget of the last step
    history = []
    valid = np.ones(inst.P, bool)  # programs whose KV bytes are defined (never re-admitted from Waiting)

    span = [0.0, 0.0, 0.0]  # summed device time from the step's start to the end of swap-out / swap-in / plan

    last_w = [None]  # the window tensor of the last step

    def one_step(t, timed=False, budget=None, window=None):
        e0, e_plan, e_out, e_in = (torch.cuda.Event(enable_timing=True) for _ in range(4))
        e0.record(s_out)
        if window is not None:  # an explicit step (the one-way pair after the timed steps)
            check(tp.rank_partition(gpu_bytes=budget, cpu_bytes=bc, window=window, stream=s_out), "rank")
        elif churn:
            bg_t, w_t = (bg, wins[0]) if t == 0 else churn_inputs[t - 1]
            step_bg[0] = bg_t
            check(tp.rank_partition(gpu_bytes=bg_t, cpu_bytes=bc, window=w_t, stream=s_out), "rank")
            last_w[0] = w_t
        elif schedule == "rotate":  # each program's window from its tier's set: Eq. 1 on the device
            with torch.cuda.stream(s_out):
                w_t = rot[t][rot_sel[tp.tier.long()], prog_ids]
            check(tp.rank_partition(gpu_bytes=bg, cpu_bytes=bc, window=w_t, stream=s_out), "rank")
            last_w[0] = w_t
        else:
            check(tp.rank_partition(gpu_bytes=bg, cpu_bytes=bc, window=wins[t % 2], stream=s_out), "rank")
            last_w[0] = wins[t % 2]
        e_plan.record(s_out)
        rc, p = tp.plan_wait()
        if rc != M.MORI_OK:
            raise RuntimeError(f"plan rejected: {rc} {p.device_error:#x}")
        tp.place_host_buffers()
        check(tp.swap_out(mode, s_out), "swap_out")
        e_out.record(s_out)
        check(tp.swap_in(mode, s_in), "swap_in")
        e_in.record(s_in)
        tp.synchronize()
        if timed:
            span[0] += e0.elapsed_time(e_out)
            span[1] += e0.elapsed_time(e_in)
            span[2] += e0.elapsed_time(e_plan)
        cat = tp.plan_arrays(p)["category"]
        valid[cat == M.MORI_CAT_ADMIT_GPU] = False
        valid[cat == M.MORI_CAT_ADMIT_CPU] = False
        history.append({k: getattr(p, k) for k in ("m_gpu", "m_cpu", "n_out", "n_in", "n_drop_gpu", "n_admit_gpu",
                                                   "pages_in", "pages_admit", "pages_free_before", "pages_released",
                                                   "pages_free_after", "pages_recycled", "bytes_out", "bytes_in")})
        return p

    for t in range(warmup):
        p = one_step(t)
        log(f"warmup {t}: out {p.bytes_out / GIB:.2f} GiB in {p.bytes_in / GIB:.2f} GiB")
    _, last_mode = M.mori_query(tp.ctx, M.MORI_Q_LAST_MODE)
    M.mori_profile(tp.ctx, True)
    for d in (0, 1):
        M.mori_profile_read(tp.ctx, d)
    torch.cuda.synchronize()
    moved = 0
    t_start = time.perf_counter()
    for t in range(warmup, warmup + steps):
        p = one_step(t, timed=True)
        moved += p.bytes_out + p.bytes_in
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t_start
    prof = [M.mori_profile_read(tp.ctx, d) for d in (0, 1)]
    M.mori_profile(tp.ctx, False)
    value = moved / elapsed / 1e9
    mix_bound_s = sum(link_bound_s(h["bytes_out"], h["bytes_in"], peaks) for h in history[-steps:])
    split_s = sum(split_model_s(h["bytes_out"], h["bytes_in"], peaks) for h in history[-steps:])
    log(f"timed {steps} steps: {moved / GIB:.2f} GiB in {elapsed:.3f} s -> {value:.2f} GB/s")

    # One way at a time, after the timed steps: every CPU-tier program back to
    # the GPU (a GPU budget of all KV bytes: H2D only), then the last timed
    # step's budgets and windows again, which put the same programs on the CPU
    # tier (D2H only) and so restore its tiers; each over its wall time (plan
    # included), against the same direction's measured peak.
    one_way = None
    if not churn and inst.total_bytes <= g.num_blocks * g.block_bytes:
        one_way = []
        w_keep = last_w[0]
        for label, budget in (("H2D", inst.total_bytes), ("D2H", bg)):
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            p = one_step(warmup + steps, budget=budget, window=w_keep)
            dt = time.perf_counter() - t0
            nb, other = (p.bytes_in, p.bytes_out) if label == "H2D" else (p.bytes_out, p.bytes_in)
            rate = nb / dt / 1e9
            peak = peaks["h2d_GBps"] if label == "H2D" else peaks["d2h_GBps"]
            one_way.append({"direction": label, "bytes": int(nb), "other_direction_bytes": int(other),
                            "ms": round(dt * 1e3, 2), "GBps": round(rate, 2),
                            "frac_of_one_way_peak": round(rate / peak, 4)})
        log(f"one way: {one_way}")

    # dominant kernel: the gather/scatter kernel of the direction on the step's
    # critical path (the direction whose work ends last)
    kern = []
    for d, (rc, n, by, ms) in enumerate(prof):
        kern.append({"kernel": "swap_kernel<out> (gather)" if d == 0 else "swap_kernel<in> (scatter)",
                     "launches": n, "payload_bytes": by, "kernel_ms": round(ms, 3),
                     "avg_launch_ms": round(ms / n, 4) if n else None,
                     "hbm_GBps": round(2 * by / (ms / 1e3) / 1e9, 1) if ms > 0 else None})
    crit = 0 if span[0] >= span[1] else 1

    verify = None
    if not args.no_verify:
        t0 = time.perf_counter()
        verify = verify_state(inst, tp, bank_dev, history, step_bg[0], bc, valid, np)
        log(f"verify ({time.perf_counter() - t0:.1f} s): {verify}")
    desc = (f"{cfg.name}: {inst.P} programs, {cfg.layers} layers x {cfg.planes} planes x {cfg.row_bytes} B rows "
            f"({cfg.dtype}), {cfg.block_tokens}-token blocks ({g.run_bytes // 1024} KiB runs), {g.num_blocks} pages "
            f"= {g.pool_bytes / GIB:.2f} GiB pool, GPU budget {cfg.gpu_pct}% of KV bytes, CPU tier "
            f"{args.cpu_gib:g} GiB in a {args.arena_gib:g} GiB pinned arena; "
            + (f"contexts scaled by {scale:g}, nothing placed before step 0, then per step the GPU budget swings "
               f"{cfg.pct_swing[0]:g}+-{cfg.pct_swing[1]:g}% and {cfg.flip_frac:.0%} of programs flip phase"
               if churn else
               "steps alternate drawn / reversed idleness windows" if schedule == "reverse" else
               "each step every program gets idleness windows of its tier's set (CPU tier busy, GPU tier middle, "
               "Waiting idle; redrawn per step), Eq. 1 computed on the device"))
    out = {"name": cfg.name, "value": value, "elapsed": elapsed, "moved": moved, "kern": kern, "crit": crit,
           "span": span, "verify": verify, "desc": desc, "copy_mode": int(last_mode), "bg": bg, "bc": bc,
           "mix_bound_s": mix_bound_s, "split_s": split_s, "one_way": one_way, "inst": inst}
    tp.close()
    del tp, pool, bank_dev, wins
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    return out


def main() -> int:
    args = parse()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py runs on exactly one GPU: the KV migration path moves one GPU's pool to its own "
              "host memory and has no multi-GPU form here (--gpus 1).", file=sys.stderr)
        return 2

    import numpy as np
    import torch

    # The two swap streams are the process's first streams: HIP maps streams to
    # a small number of hardware queues (4 per process by default) and streams
    # created later share queues, which serialises swap-out with swap-in.
    s_out, s_in = torch.cuda.Stream(), torch.cuda.Stream()

    from paper_2606_00866_amd import mori as M
    from workload import CONFIGS, budget_bytes, make_instance

    cfg = CONFIGS[args.workload]
    schedule = args.schedule or ("rotate" if cfg.name == "mla" else "reverse")
    M.lib()
    assert torch.cuda.is_available(), "bench.py needs the GPU"
    churn = cfg.name == "churn"
    scale = args.scale if args.scale is not None else (0.32 if churn else 1.0)
    inst0 = make_instance(cfg, scale=scale, resident="wait" if churn else "gpu")
    bg0 = budget_bytes(inst0.total_bytes, cfg.gpu_pct)
    bc = int(args.cpu_gib * GIB)
    evict_sizes = () if args.no_evict else (inst0.geom.num_blocks, 1 << 20)
    cases = () if args.no_plan else plan_cases(np, inst0, bg0, bc)
    cpu = None
    if not args.no_cpu_baseline:
        t0 = time.perf_counter()
        cpu = cpu_baseline(cfg, schedule, bc / inst0.total_bytes, args.cpu_seconds, evict_sizes, cases)
        log(f"cpu baseline {cpu['value']} GB/s ({time.perf_counter() - t0:.1f} s)")

    peaks = measure_peaks(torch, M, s_out, s_in)
    log(f"peaks {peaks}")

    head = run_workload(args, cfg.name, schedule, args.steps, args.warmup, s_out, s_out if args.serial_swaps else s_in,
                        peaks, torch, np, M)
    others = {}
    for name in [w for w in args.extra.split(",") if w and w != cfg.name]:
        o = run_workload(args, name, "rotate" if name == "mla" else "reverse", args.extra_steps, args.warmup, s_out,
                         s_in, peaks, torch, np, M)
        k = o["kern"]
        others[name] = {"value": round(o["value"], 3), "unit": "GB/s", "steps": args.extra_steps,
                        "ms_per_step": round(o["elapsed"] / args.extra_steps * 1e3, 3),
                        "bytes_per_step": int(o["moved"] / max(args.extra_steps, 1)), "workload": o["desc"],
                        "frac_of_bidir_peak": round(o["value"] / peaks["bidir_GBps"], 4),
                        "gather_hbm_GBps": k[0]["hbm_GBps"], "scatter_hbm_GBps": k[1]["hbm_GBps"],
                        "gather_frac_of_hbm_peak": round((k[0]["hbm_GBps"] or 0) / HBM_PEAK_GBPS, 4),
                        "scatter_frac_of_hbm_peak": round((k[1]["hbm_GBps"] or 0) / HBM_PEAK_GBPS, 4),
                        "verify": o["verify"]}

    evict = None if args.no_evict else evict_leg(torch, np, M, evict_sizes)
    if evict:
        log(f"evict order: {evict}")
    plan = None if args.no_plan else plan_leg(torch, np, M, cases)
    if plan:
        log(f"plan: {plan}")
    replica = None if args.no_plan else replica_leg(np, M)
    if replica:
        log(f"replica admission: {replica}")

    kern, crit = head["kern"], head["crit"]
    dom = kern[crit]
    achieved = dom["hbm_GBps"] or 0.0
    value = head["value"]
    out = {
        "metric": "KV migration GB/s (D2H+H2D) vs host-link peak; gather/scatter HBM GB/s",
        "value": round(value, 3),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(head["elapsed"] / args.steps * 1e3, 3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "u8",
        "data": "synthetic",
        "config": {
            "workload": head["desc"],
            "copy_mode": {0: "auto", 1: "kernel", 2: "copy-engine"}[head["copy_mode"]],
            "hw_queues": int(os.environ["GPU_MAX_HW_QUEUES"]),
            "gpu_budget_bytes": head["bg"],
            "cpu_budget_bytes": head["bc"],
            "bytes_per_step": int(head["moved"] / max(args.steps, 1)),
        },
        "hostlink": {**peaks, "frac_of_bidir_peak": round(value / peaks["bidir_GBps"], 4),
                     "frac_of_mix_bound": round(head["mix_bound_s"] / head["elapsed"], 4),
                     "mix_bound": ("lower bound on the timed steps' time on this link, per step max(out / d2h, "
                                   "in / h2d, (out + in) / bidir), summed; frac_of_mix_bound = that bound over the "
                                   "measured time (equals frac_of_bidir_peak when every step moves as much each way)"),
                     "one_way_step": head["one_way"],
                     "split_model_over_measured": round(head["split_s"] / head["elapsed"], 4),
                     "split_model": ("per step, both directions started together at the measured two-way split "
                                     "(bidir_split) until the smaller is done, then the larger alone at its "
                                     "one-direction rate, summed; over the measured time (a model of two unpaced "
                                     "copy streams, not a bound: above 1 the steps beat it)")},
        "roofline": {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                     "frac": round(achieved / HBM_PEAK_GBPS, 4), "traffic": stored_traffic(cfg.name, crit),
                     "algorithmic_bytes_per_launch": int(2 * dom["payload_bytes"] / max(dom["launches"], 1)),
                     "kernel": dom["kernel"], "frac_of_measured_copy_peak":
                         round(achieved / peaks["d2d_copy_GBps"], 4)},
        "kernels": kern,
        "paper_context": {
            "end_to_end_throughput_vs_best_offloading_baseline": "+20% to +71%",
            "average_ttft_vs_best_offloading_baseline": "-18% to -43%",
            "hardware": "H200 (capped to 80 GB, and full) and B200 (TP=2), SGLang with HiCache",
            "note": ("whole-system serving gains of the method, context only; the paper reports no KV migration "
                     "or gather/scatter bandwidth, hence vs_baseline null"),
        },
        "direction_ms_per_step": {"swap_out": round(head["span"][0] / args.steps, 2),
                                  "swap_in": round(head["span"][1] / args.steps, 2)},
        "plan_us_in_step": round(head["span"][2] / args.steps * 1e3, 1),
        "other_workloads": others or None,
        "plan": plan,
        "replica_admit": replica,
        "cpu_baseline": cpu,
        "verify": head["verify"],
        "evict_order": evict,
    }
    print(json.dumps(out), flush=True)
    return 0


def verify_state(inst, tp, bank_dev, history, bg, bc, valid, np):
    """Checks of the final state that need no reference implementation (exact
    parity with the oracle at these sizes is a GPU test): every page owned at
    most once and never also free, owned + free pages = the pool, programs off
    the GPU own no page, both budgets respected, each step's page accounting
    consistent, and every byte of every resident run of the programs whose KV
    is defined (all pages of GPU-resident programs, all CPU-tier host buffers)
    equal to its content-addressed value -- the input run of the same program,
    block and plane: the copy rule of a swap."""
    from workload import check_tier_bytes

    g = inst.geom
    tbl, tier, free = tp.state()
    off = inst.tbl_off
    nblk = inst.nblk.astype(np.int64)
    owned = np.concatenate([tbl[off[p]:off[p + 1]] for p in range(inst.P) if tier[p] == 0])
    if (owned >= g.num_blocks).any() or np.unique(owned).size != owned.size or free[owned].any():
        return {"ok": False, "what": "page ownership"}
    if owned.size + int(free.sum()) != g.num_blocks:
        return {"ok": False, "what": "page conservation"}
    if any((tbl[off[p]:off[p + 1]] != 0xFFFFFFFF).any() for p in range(inst.P) if tier[p] != 0):
        return {"ok": False, "what": "non-resident tables"}
    if nblk[tier == 0].sum() * g.block_bytes > bg or nblk[tier == 1].sum() * g.block_bytes > bc:
        return {"ok": False, "what": "budgets"}
    for t, h in enumerate(history):
        if h["pages_free_before"] + h["pages_released"] - h["pages_in"] - h["pages_admit"] != h["pages_free_after"]:
            return {"ok": False, "what": "page accounting", "step": t}
    r = check_tier_bytes(tp.pool, g, off, tbl, tier, bank_dev, tp.host_view, programs=valid)
    if not r["ok"]:
        return {"ok": False, "what": "bytes", **r}
    return {"ok": True, "steps": len(history), "runs_checked": r["gpu_runs"] + r["host_runs"],
            "bytes_checked": r["bytes"], "programs_checked": int((valid & (tier != 2) & (inst.nblk > 0)).sum())}


if __name__ == "__main__":
    sys.exit(main())
