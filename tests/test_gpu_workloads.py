"""The named workloads on the GPU, in the launch configuration bench.py times
(copy-engine swaps, 2 GiB of staging per direction in two halves, one pinned CPU-tier arena).

Full-size Llama-3-8B, Llama-3-70B and MLA pools (136-155 GiB of HBM) and one
rank's share of the Llama-3-70B programs under tensor parallelism of 2 (the
same programs with 1 KiB rows and 16 KiB runs, 76 GiB): three
boundary-policy steps, one incremental-policy step and one three-tier (SSD)
step.  The oracle replays every step's placement; after every step the
summary, block tables, tiers and free map must match it exactly, and every
byte of every resident run -- each page of each GPU-resident program and each
host buffer of the CPU and SSD tiers -- must equal its content-addressed
value (regenerated and compared on the device).

Churn (1024 programs, 100 steps, GPU budget swinging 45-65%, 10% of programs
flipping phase per step), scaled to fit one GPU and the pinned-memory ceiling:
the same checks after every step, in both copy modes.
"""
import numpy as np
import pytest
import torch

from gpu_helpers import log
from oracle import oracle
from paper_2606_00866_amd import mori as M
from paper_2606_00866_amd.tiering import TierPool
from workload import (CHURN, LLAMA3_70B, LLAMA3_70B_TP2, LLAMA3_70B_TP4, LLAMA3_70B_TP8, LLAMA3_8B, MLA, budget_bytes,
                      check_tier_bytes, churn_steps, fill_pool_torch, make_bank, make_instance, program_content_torch)

pytestmark = [pytest.mark.gpu, pytest.mark.slow]
GIB = 1 << 30
SUMMARY = ("m_gpu", "m_cpu", "n_out", "n_in", "n_drop_gpu", "n_drop_cpu", "n_admit_gpu", "n_admit_cpu", "pages_out",
           "pages_in", "pages_admit", "pages_free_before", "pages_released", "pages_recycled", "pages_free_after",
           "bytes_out", "bytes_in", "gpu_bytes_after", "cpu_bytes_after")


class Harness:
    def __init__(self, inst, arena_bytes, staging=2 << 30, fill=True):
        self.inst = inst
        g = inst.geom
        self.g = g
        free, _ = torch.cuda.mem_get_info()
        assert g.pool_bytes + 4 * GIB < free, f"pool {g.pool_bytes / GIB:.1f} GiB > free {free / GIB:.1f} GiB"
        self.bank = make_bank(inst.seed, inst.dtype, g.run_bytes)
        self.bank_dev = torch.from_numpy(self.bank.view(np.int16)).cuda()
        pool = torch.empty(g.pool_bytes, dtype=torch.uint8, device="cuda")
        if fill:
            fill_pool_torch(pool, inst, self.bank_dev)
        self.tp = TierPool(g, inst.tbl_off, inst.tbl, inst.tier, inst.free_map, arena_bytes=arena_bytes,
                           max_programs=inst.P, staging_bytes=staging, pool=pool)
        self.tbl, self.tier, self.free = inst.copy_state()
        self.valid = np.ones(inst.P, bool)
        self.s_out, self.s_in = torch.cuda.Stream(), torch.cuda.Stream()
        self.steps = 0
        self.bytes_checked = 0

    def close(self):
        torch.cuda.synchronize()
        self.tp.close()
        del self.tp.pool
        torch.cuda.empty_cache()

    def step(self, window, bg, bc, mode=M.MORI_COPY_AUTO, iota=None, status=None, flags=0, ssd=0):
        inst = self.inst
        flags |= oracle.F_IDLENESS_GIVEN if iota is not None else 0
        res = oracle.rebalance(self.g, window=window, iota=iota, status=status, tbl_off=inst.tbl_off, tbl=self.tbl,
                               tier=self.tier, free_map=self.free, gpu_budget=bg, cpu_budget=bc, flags=flags,
                               ssd_budget=ssd)
        assert res.rc == oracle.OK
        w = None if window is None else torch.from_numpy(np.ascontiguousarray(window)).cuda()
        it = None if iota is None else torch.from_numpy(np.ascontiguousarray(iota, np.float32)).cuda()
        st = None if status is None else torch.from_numpy(np.ascontiguousarray(status, np.uint8)).cuda()
        plan = self.tp.step(gpu_bytes=bg, cpu_bytes=bc, window=w, idleness=it, status=st, flags=flags, mode=mode,
                            s_out=self.s_out, s_in=self.s_in, ssd_bytes=ssd)
        for k in SUMMARY:
            assert getattr(plan, k) == res.summary[k], (self.steps, k, getattr(plan, k), res.summary[k])
        arr = self.tp.plan_arrays(plan)
        assert (arr["order"] == res.order).all() and (arr["category"] == res.category).all()
        tbl, tier, free = self.tp.state()
        assert (tbl == self.tbl).all() and (tier == self.tier).all() and (free == self.free).all(), self.steps
        self.prefill(res.category)
        self.check_all_bytes()
        self.steps += 1
        return plan

    def prefill(self, cat):
        """Programs admitted from Waiting get their KV recomputed (an engine's
        prefill in a real system); the harness writes the expected content."""
        inst, g = self.inst, self.g
        adm_g = np.flatnonzero((cat == oracle.ADMIT_GPU) & (inst.nblk > 0))
        if adm_g.size:
            op = np.zeros(g.num_blocks, np.int64)
            oi = np.zeros(g.num_blocks, np.int64)
            for p in adm_g:
                pages_p = self.tbl[inst.tbl_off[p]:inst.tbl_off[p + 1]].astype(np.int64)
                op[pages_p] = p
                oi[pages_p] = np.arange(pages_p.size)
            pages = np.concatenate([self.tbl[inst.tbl_off[p]:inst.tbl_off[p + 1]] for p in adm_g]).astype(np.int64)
            fill_pool_torch(self.tp.pool, inst, self.bank_dev, torch.from_numpy(op).cuda(),
                            torch.from_numpy(oi).cuda(), pages=torch.from_numpy(pages).cuda())
        for p in np.flatnonzero(((cat == oracle.ADMIT_CPU) | (cat == oracle.ADMIT_SSD)) & (inst.nblk > 0)):
            dst = torch.from_numpy(self.tp.host_view(int(p)).view(np.int16))
            program_content_torch(inst, self.bank_dev, int(p), out=dst)  # one copy into the pinned tier
        torch.cuda.synchronize()

    def check_all_bytes(self):
        """Every resident run equals its content-addressed value: all pages of
        every GPU-resident program (through the tables) and every CPU/SSD host
        buffer, compared on the device."""
        r = check_tier_bytes(self.tp.pool, self.g, self.inst.tbl_off, self.tbl, self.tier, self.bank_dev,
                             self.tp.host_view)
        assert r["ok"], (self.steps, r)
        self.bytes_checked += r["bytes"]


@pytest.mark.parametrize("cfg", [LLAMA3_8B, LLAMA3_70B, LLAMA3_70B_TP2, LLAMA3_70B_TP4, LLAMA3_70B_TP8, MLA],
                         ids=lambda c: c.name)
def test_full_size_workload(cfg):
    inst = make_instance(cfg)
    total = inst.total_bytes
    bg = budget_bytes(total, cfg.gpu_pct)
    bc = 28 * GIB
    log(f"{cfg.name}: P={inst.P} NB={inst.geom.num_blocks} pool {inst.geom.pool_bytes / GIB:.1f} GiB "
        f"gpu {bg / GIB:.1f} GiB cpu {bc / GIB:.1f} GiB")
    h = Harness(inst, arena_bytes=60 * GIB)
    try:
        wins = (inst.window, inst.window[:, :, ::-1].copy())
        for t in range(3):
            if t < 2:  # drawn windows, then every program's reasoning and tool time swapped
                plan = h.step(wins[t], bg, bc)
            else:  # given idleness: CPU-tier programs busiest, then GPU-tier ones, Waiting last
                iota = np.array([0.5, 0.1, 0.9], np.float32)[h.tier]  # indexed by tier: GPU, CPU, Wait
                plan = h.step(None, bg, bc, iota=iota)
            log(f"  step {t}: out {plan.bytes_out / GIB:.2f} GiB in {plan.bytes_in / GIB:.2f} GiB "
                f"admit {plan.n_admit_gpu} drop {plan.n_drop_gpu} recycled {plan.pages_recycled}")
        assert plan.n_in > 0 and plan.n_out > 0
        # the incremental policy (Sec. 4.3.1) at full size: the GPU budget cut by a tenth forces
        # demotions (Acting first) into CPU room grown by as much; busy programs are Reasoning,
        # a third of the waiting ones new
        status = np.where(inst.busy, 0, 1).astype(np.uint8)
        status[(h.tier == 2) & (np.arange(inst.P) % 3 == 0)] = 2
        plan = h.step(inst.window, bg - bg // 10, bc + bg // 10, status=status, flags=oracle.F_INCREMENTAL)
        log(f"  incremental step: out {plan.bytes_out / GIB:.2f} GiB drop {plan.n_drop_gpu} "
            f"in {plan.n_in} admit {plan.n_admit_gpu}")
        assert plan.n_out > 0
        # the SSD tier (Sec. 7.1): a third run of the ranking, its KV in host buffers here (the CPU
        # room kept below what leaves the GPU, so that the smaller shards also reach the SSD tier)
        plan = h.step(inst.window, bg, min(bc, (total - bg) // 2), flags=oracle.F_SSD_TIER, ssd=8 * GIB)
        log(f"  SSD step: m_ssd {plan.m_ssd} out {plan.n_out} in {plan.n_in}")
        assert plan.m_ssd > 0
        log(f"  bytes compared over {h.steps} steps: {h.bytes_checked / GIB:.1f} GiB")
    finally:
        h.close()


@pytest.mark.parametrize("cfg", [MLA, LLAMA3_70B_TP2], ids=lambda c: c.name)
def test_full_size_kernel_direct(cfg):
    """Kernel-direct swaps at full size: the gather stores into, and the
    scatter loads from, the pinned CPU tier over the host link (two runs per
    workgroup, one vector per thread per round; the swap-in in two launches
    around the swap-out's event).  Drawn windows, then twice given idleness
    that ranks the CPU tier busiest (both directions move); every byte
    compared after each step."""
    inst = make_instance(cfg)
    bg = budget_bytes(inst.total_bytes, cfg.gpu_pct)
    bc = 28 * GIB
    log(f"{cfg.name} kernel-direct: P={inst.P} pool {inst.geom.pool_bytes / GIB:.1f} GiB")
    h = Harness(inst, arena_bytes=60 * GIB)
    try:
        moved_both = 0
        for t in range(3):
            if t == 0:
                plan = h.step(inst.window, bg, bc, mode=M.MORI_COPY_KERNEL)
            else:  # CPU-tier programs busiest, then GPU-tier ones, Waiting last
                iota = np.array([0.5, 0.1, 0.9], np.float32)[h.tier]
                plan = h.step(None, bg, bc, mode=M.MORI_COPY_KERNEL, iota=iota)
            moved_both += plan.n_in > 0 and plan.n_out > 0
            log(f"  step {t}: out {plan.bytes_out / GIB:.2f} GiB in {plan.bytes_in / GIB:.2f} GiB")
        assert moved_both == 2
        assert M.mori_query(h.tp.ctx, M.MORI_Q_LAST_MODE) == (M.MORI_OK, M.MORI_COPY_KERNEL)
    finally:
        h.close()


def test_churn_scaled():
    """Churn at 8% of its context lengths (about 46 GiB of KV, a 30 GiB pool and
    a CPU tier of a quarter of the KV bytes): 100 steps, both directions each step."""
    scale = 0.08
    inst = make_instance(CHURN, scale=scale, resident="wait")
    total = inst.total_bytes
    bc = total // 4
    log(f"churn x{scale}: P={inst.P} NB={inst.geom.num_blocks} total {total / GIB:.1f} GiB cpu {bc / GIB:.1f} GiB")
    h = Harness(inst, arena_bytes=int(2.2 * bc) + GIB, fill=False)
    try:
        h.step(inst.window, budget_bytes(total, CHURN.pct_swing[0]), bc)  # step 0: place everything
        moved, recycled_steps = 0, 0
        for t, pct, busy, window in churn_steps(CHURN, inst.busy):
            mode = M.MORI_COPY_CE if t % 2 else M.MORI_COPY_KERNEL  # both copy modes at scale
            plan = h.step(window, budget_bytes(total, pct), bc, mode=mode)
            moved += plan.bytes_out + plan.bytes_in
            recycled_steps += plan.pages_recycled > 0
            if t % 20 == 0:
                log(f"  step {t}: pct {pct:.1f} out {plan.bytes_out / GIB:.2f} in {plan.bytes_in / GIB:.2f} GiB "
                    f"recycled {plan.pages_recycled}, {h.bytes_checked / GIB:.1f} GiB compared so far")
        assert moved > 0
        assert recycled_steps > 0  # swap-ins onto pages released by the same step's swap-out
    finally:
        h.close()
