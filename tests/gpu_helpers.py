"""Side-by-side driver for the GPU parity tests: the same seeded state is run
through libmori (via the C ABI) and through the CPU oracle, then compared
element by element."""
from __future__ import annotations

import sys

import numpy as np
import torch

from oracle import oracle
from paper_2606_00866_amd import mori as M
from paper_2606_00866_amd.tiering import MoriError, TierPool
from workload import fill_pool_np, make_bank, program_host_content

NONE = 0xFFFFFFFF


def log(msg: str) -> None:
    print(msg, flush=True)
    sys.stdout.flush()


class Pair:
    """GPU state (TierPool) and oracle state (numpy) of one instance."""

    def __init__(self, inst, seed=0, arena_bytes=None, staging_bytes=0, max_programs=None, content=True):
        self.inst = inst
        g = inst.geom
        self.g = g
        self.bank = make_bank(seed, inst.dtype, g.run_bytes)
        self.pool = fill_pool_np(inst, self.bank) if content else np.zeros(g.pool_bytes, np.uint8)
        self.bufs = []
        for p in range(inst.P):
            if inst.tier[p] in (1, 3) and content:  # CPU or SSD tier: KV in the host buffer
                self.bufs.append(program_host_content(inst, self.bank, p).copy())
            else:
                self.bufs.append(np.zeros(int(inst.nblk[p]) * g.block_bytes, np.uint8))
        self.tbl, self.tier, self.free = inst.copy_state()
        arena = arena_bytes if arena_bytes is not None else 2 * inst.total_bytes + 4096 * (inst.P + 1) + (1 << 20)
        self.tp = TierPool(g, inst.tbl_off, inst.tbl, inst.tier, inst.free_map, arena_bytes=arena,
                           max_programs=max_programs or max(inst.P, 1), staging_bytes=staging_bytes)
        if g.pool_bytes:
            self.tp.pool.copy_(torch.from_numpy(self.pool).to(self.tp.device))
        for p in range(inst.P):
            if inst.tier[p] in (1, 3):
                self.tp.give_host_buffer(p)
                if self.bufs[p].size:
                    self.tp.host_view(p)[:] = self.bufs[p]
        self.s_out, self.s_in = torch.cuda.Stream(), torch.cuda.Stream()

    def close(self):
        torch.cuda.synchronize()
        self.tp.close()

    def step(self, *, gpu_bytes, cpu_bytes, window=None, iota=None, status=None, flags=0,
             mode=M.MORI_COPY_AUTO, compare_bytes=True, ssd_bytes=0):
        inst, g = self.inst, self.g
        res = oracle.rebalance(g, window=window, iota=iota, status=status, tbl_off=inst.tbl_off, tbl=self.tbl,
                               tier=self.tier, free_map=self.free, gpu_budget=gpu_bytes, cpu_budget=cpu_bytes,
                               flags=flags, pool=self.pool, host_bufs=self.bufs, ssd_budget=ssd_bytes)
        dev = lambda a, dt: None if a is None else torch.from_numpy(np.ascontiguousarray(a, dt)).to(self.tp.device)
        w, it, st = dev(window, np.float32), dev(iota, np.float32), dev(status, np.uint8)
        if res.rc != oracle.OK:
            return res, None
        plan = self.tp.step(gpu_bytes=gpu_bytes, cpu_bytes=cpu_bytes, window=w, idleness=it, status=st,
                            flags=flags, mode=mode, s_out=self.s_out, s_in=self.s_in, ssd_bytes=ssd_bytes)
        self.compare(res, plan, compare_bytes)
        self.prefill(res)
        return res, plan

    def prefill(self, res):
        """Programs admitted from Waiting get their KV recomputed (by the engine in
        a real system): write the same content on both sides."""
        inst, g = self.inst, self.g
        for p in np.flatnonzero(res.category == oracle.ADMIT_GPU):
            n = int(inst.nblk[p])
            if n == 0:
                continue
            content = program_host_content(inst, self.bank, int(p)).reshape(g.nplanes, n, g.run_bytes)
            pages = self.tbl[inst.tbl_off[p]:inst.tbl_off[p + 1]].astype(np.int64)
            self.pool.reshape(g.nplanes, g.num_blocks, g.run_bytes)[:, pages] = content
            dpool = self.tp.pool.view(g.nplanes, g.num_blocks, g.run_bytes)
            dpool[:, torch.from_numpy(pages).to(self.tp.device)] = torch.from_numpy(content).to(self.tp.device)
        for p in np.flatnonzero((res.category == oracle.ADMIT_CPU) | (res.category == oracle.ADMIT_SSD)):
            if inst.nblk[p]:
                c = program_host_content(inst, self.bank, int(p))
                self.bufs[p][:] = c
                self.tp.host_view(int(p))[:] = c
        torch.cuda.synchronize()

    def compare(self, res, plan, compare_bytes=True):
        tp, g, inst = self.tp, self.g, self.inst
        arr = tp.plan_arrays(plan)
        assert plan.device_error == 0
        assert (arr["order"] == res.order).all(), "rank order"
        assert (arr["prefix"] == res.prefix).all(), "byte prefix"
        assert (arr["tier_old"] == res.tier_old).all(), "old tiers"
        assert (arr["category"] == res.category).all(), "categories"
        for k, v in res.summary.items():
            assert getattr(plan, k) == v, f"summary field {k}: gpu {getattr(plan, k)} oracle {v}"
        assert (arr["out_programs"] == res.order[res.category[res.order] == oracle.OUT]).all()
        assert (arr["in_programs"] == res.order[res.category[res.order] == oracle.IN]).all()
        tbl, tier, free = tp.state()
        assert (tier == self.tier).all(), "tiers"
        assert (tbl == self.tbl).all(), "block tables"
        assert (free == self.free).all(), "free map"
        if not compare_bytes:
            return
        if g.pool_bytes:
            dpool = tp.pool.cpu().numpy().reshape(g.nplanes, g.num_blocks, g.run_bytes)
            opool = self.pool.reshape(g.nplanes, g.num_blocks, g.run_bytes)
            owned = self.tbl[self.tbl != NONE].astype(np.int64)
            assert np.array_equal(dpool[:, owned], opool[:, owned]), "pool bytes of resident pages"
        for p in np.flatnonzero((self.tier == 1) | (self.tier == 3)):
            if res.category[p] in (oracle.ADMIT_CPU, oracle.ADMIT_SSD):
                continue
            assert np.array_equal(tp.host_view(int(p)), self.bufs[p]), f"host bytes of program {p}"


def instance_from_blocks(blocks, tier, gpu_budget_blocks, status=None, extra_free=3, seed=0):
    """A consistent pool holding programs of the given block counts and tiers,
    one block = 16 bytes, with room for the GPU budget (hand-derived fixtures)."""
    from workload import Geometry, random_instance

    P = len(blocks)
    rng = np.random.default_rng(seed)
    inst = random_instance(rng, P=P, geom=Geometry(1, 1, 1, 16, 0), extra_free=0)
    nblk = np.array(blocks, np.uint32)
    tier = np.array(tier, np.uint8)
    NB = max(int(nblk[tier == 0].sum()) + extra_free, gpu_budget_blocks)
    off = np.zeros(P + 1, np.uint32)
    off[1:] = np.cumsum(nblk)
    tbl = np.full(int(off[-1]), NONE, np.uint32)
    perm = rng.permutation(NB).astype(np.uint32)
    used = 0
    for p in range(P):
        if tier[p] == 0:
            tbl[off[p]:off[p + 1]] = perm[used:used + nblk[p]]
            used += int(nblk[p])
    free = np.zeros(NB, np.uint8)
    free[perm[used:]] = 1
    inst.geom = Geometry(1, 1, 1, 16, NB)
    inst.nblk, inst.tbl_off, inst.tbl, inst.tier, inst.free_map = nblk, off, tbl, tier, free
    inst.ctx = nblk.astype(np.int64)
    if status is not None:
        inst.status = np.array(status, np.uint8)
    return inst


__all__ = ["Pair", "log", "MoriError", "NONE", "instance_from_blocks"]
