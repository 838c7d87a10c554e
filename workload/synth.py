"""Seeded synthetic inputs shared by the oracle and the HIP path.

This module draws inputs only -- program sizes, idleness windows, block tables,
pool occupancy, budgets and KV bytes -- and holds none of
the placement method's arithmetic (no idleness, ranking, boundary, page
allocation or copying).  Every draw is reproducible from the config's seed:
``SeedSequence(seed).spawn`` gives one independent stream per draw kind, taken
in the fixed order contexts -> phases -> windows -> fragmentation -> KV bank ->
per-step draws.

KV bytes are content-addressed: the run of program ``p``, logical block ``i``,
plane ``q`` (= layer * planes + k/v) holds a window of a seeded bank of normal
values (fp16 or bf16) starting at ``run_offset(p, i, q)``, and its first four
bytes are overwritten by ``run_tag(p, i, q)``.  Any run can therefore be
regenerated on its own, so placement errors are caught without a full mirror.
"""
from __future__ import annotations

import math
from dataclasses import dataclass

import numpy as np

from .configs import (A_BUSY_MEDIAN, A_IDLE_MEDIAN, A_SIGMA, FRAG_MEAN_CHUNK, R_MEDIAN, R_SIGMA, SIGMA_CTX,
                      WINDOW_K, KVConfig)

NO_PAGE = 0xFFFFFFFF
TIER_GPU, TIER_CPU, TIER_WAIT = 0, 1, 2
BANK_BITS = 22
BANK = 1 << BANK_BITS
FREE_OWNER = 0x7FF  # owner id used to fill pages that belong to no program


# --------------------------------------------------------------------------
# geometry and instance
# --------------------------------------------------------------------------
@dataclass
class Geometry:
    layers: int
    planes: int
    block_tokens: int
    row_bytes: int
    num_blocks: int

    @property
    def nplanes(self) -> int:
        return self.layers * self.planes

    @property
    def run_bytes(self) -> int:
        return self.block_tokens * self.row_bytes

    @property
    def block_bytes(self) -> int:
        return self.nplanes * self.run_bytes

    @property
    def pool_bytes(self) -> int:
        return self.nplanes * self.num_blocks * self.run_bytes


@dataclass
class Instance:
    name: str
    geom: Geometry
    dtype: str
    ctx: np.ndarray        # int64 [P] tokens
    nblk: np.ndarray       # uint32 [P]
    busy: np.ndarray       # bool [P]
    window: np.ndarray     # float32 [P][k][2] (reasoning s, acting s), oldest first
    status: np.ndarray     # uint8 [P] 0 reasoning, 1 acting
    tbl_off: np.ndarray    # uint32 [P+1]
    tbl: np.ndarray        # uint32 [sum nblk]
    tier: np.ndarray       # uint8 [P]
    free_map: np.ndarray   # uint8 [NB]
    seed: int
    scale: float = 1.0

    @property
    def P(self) -> int:
        return int(self.nblk.size)

    @property
    def total_bytes(self) -> int:
        return int(self.nblk.astype(np.uint64).sum()) * self.geom.block_bytes

    def copy_state(self):
        return self.tbl.copy(), self.tier.copy(), self.free_map.copy()


def _streams(seed: int, n: int = 6):
    return [np.random.Generator(np.random.PCG64(s)) for s in np.random.SeedSequence(seed).spawn(n)]


def budget_bytes(total: int, pct: float) -> int:
    """floor(total * pct / 100) with pct taken to 1/100 of a percent, in integers."""
    bp = int(round(pct * 100))
    return total * bp // 10000


# --------------------------------------------------------------------------
# draws
# --------------------------------------------------------------------------
def draw_contexts(rng, cfg: KVConfig, scale: float = 1.0) -> np.ndarray:
    P = cfg.programs
    if cfg.ctx_kind == "uniform":
        ctx = rng.integers(cfg.ctx_lo, cfg.ctx_hi + 1, size=P).astype(np.float64) * scale
    else:
        z = rng.standard_normal(P)
        ctx = np.exp(math.log(cfg.ctx_median * scale) + SIGMA_CTX * z)
        ctx = np.clip(ctx, cfg.ctx_lo * scale, cfg.ctx_hi * scale)
    return np.floor(ctx).astype(np.int64)


def draw_phases(rng, P: int, busy_frac: float) -> np.ndarray:
    busy = np.zeros(P, bool)
    busy[rng.permutation(P)[: int(round(busy_frac * P))]] = True
    return busy


def draw_windows(rng, busy: np.ndarray, k: int = WINDOW_K) -> np.ndarray:
    """[P][k][2] float32 seconds: reasoning ~ lognormal(2 s, 0.5); tool call ~
    lognormal(1 s busy / 60 s idle, 1.0); the newest tool call is still running,
    so only a uniform fraction of it has elapsed."""
    P = busy.size
    r = np.exp(math.log(R_MEDIAN) + R_SIGMA * rng.standard_normal((P, k)))
    med = np.where(busy, A_BUSY_MEDIAN, A_IDLE_MEDIAN)[:, None]
    a = np.exp(np.log(med) + A_SIGMA * rng.standard_normal((P, k)))
    a[:, -1] *= rng.random(P)
    return np.stack([r, a], axis=2).astype(np.float32)


def page_permutation(rng, NB: int, frag: str) -> np.ndarray:
    """Initial page order dealt to programs: a uniform permutation ('shuffled') or
    a shuffle of contiguous chunks with geometric lengths of mean 4 ('chunked')."""
    if frag == "shuffled":
        return rng.permutation(NB).astype(np.uint32)
    lens = []
    tot = 0
    while tot < NB:
        n = int(rng.geometric(1.0 / FRAG_MEAN_CHUNK))
        n = min(n, NB - tot)
        lens.append(n)
        tot += n
    starts = np.concatenate([[0], np.cumsum(lens)[:-1]]).astype(np.int64)
    chunks = [np.arange(s, s + n, dtype=np.uint32) for s, n in zip(starts, lens)]
    order = rng.permutation(len(chunks))
    return np.concatenate([chunks[j] for j in order]) if chunks else np.zeros(0, np.uint32)


def make_instance(cfg: KVConfig, scale: float = 1.0, resident: str = "gpu") -> Instance:
    """Build the workload's initial state.  resident='gpu': every program holds
    its pages (pool = max(min_blocks, total blocks)); resident='wait': nothing is
    placed yet and the pool has ceil(0.65 * total blocks) free pages."""
    g_ctx, g_phase, g_win, g_frag, _g_bank, _g_steps = _streams(cfg.seed)
    ctx = draw_contexts(g_ctx, cfg, scale)
    nblk = ((ctx + cfg.block_tokens - 1) // cfg.block_tokens).astype(np.uint32)
    busy = draw_phases(g_phase, cfg.programs, cfg.busy_frac)
    window = draw_windows(g_win, busy)
    total_blocks = int(nblk.astype(np.int64).sum())
    tbl_off = np.zeros(cfg.programs + 1, np.uint32)
    tbl_off[1:] = np.cumsum(nblk.astype(np.int64))
    if resident == "gpu":
        NB = max(cfg.min_blocks, total_blocks)
        perm = page_permutation(g_frag, NB, cfg.frag)
        tbl = perm[:total_blocks].copy()
        free_map = np.zeros(NB, np.uint8)
        free_map[perm[total_blocks:]] = 1
        tier = np.zeros(cfg.programs, np.uint8)
    else:
        NB = int(math.ceil(0.65 * total_blocks))
        tbl = np.full(total_blocks, NO_PAGE, np.uint32)
        free_map = np.ones(NB, np.uint8)
        tier = np.full(cfg.programs, TIER_WAIT, np.uint8)
    geom = Geometry(cfg.layers, cfg.planes, cfg.block_tokens, cfg.row_bytes, NB)
    status = np.ones(cfg.programs, np.uint8)  # every program is in a tool call at the tick
    return Instance(cfg.name, geom, cfg.dtype, ctx, nblk, busy, window, status, tbl_off, tbl, tier, free_map,
                    cfg.seed, scale)


def churn_steps(cfg: KVConfig, busy0: np.ndarray, steps: int | None = None):
    """Per-step inputs of the churn workload: (t, gpu_pct, busy, window).
    The GPU budget swings as centre + amplitude * sin(2 pi t / 20); exactly
    round(flip_frac * P) programs flip phase each step; all windows are redrawn."""
    rng = _streams(cfg.seed)[5]
    busy = busy0.copy()
    P = busy.size
    n_flip = int(round(cfg.flip_frac * P))
    centre, amp = cfg.pct_swing
    for t in range(1, (steps if steps is not None else cfg.steps) + 1):
        pct = centre + amp * math.sin(2 * math.pi * t / 20.0)
        flip = rng.choice(P, size=n_flip, replace=False)
        busy[flip] = ~busy[flip]
        yield t, pct, busy.copy(), draw_windows(rng, busy)


# Window sets of the rotation schedule: (reasoning, tool-call) seconds drawn
# uniformly per cycle.  The three sets never interleave in idleness: over k
# cycles the busy set's tool time is at most 0.3k s against at least 1.5k s of
# reasoning (idleness below 0.3 / 1.8 = 0.17), the middle set's lies in
# [2k, 4k] against [1.5k, 2.5k] (idleness in [2 / 4.5, 4 / 5.5] = [0.44, 0.73])
# and the idle set's in [40k, 80k] (idleness above 40 / 42.5 = 0.94).
ROTATION_SETS = ((1.5, 2.5, 0.0, 0.3), (1.5, 2.5, 2.0, 4.0), (1.5, 2.5, 40.0, 80.0))


def rotation_windows(seed: int, P: int, steps: int, k: int = WINDOW_K) -> np.ndarray:
    """float32 [steps][3][P][k][2] windows, redrawn every step: set 0 busy
    (tool calls that have just ended), set 1 middle, set 2 idle (long tool
    calls).  A schedule that gives each program the set of its current tier
    (CPU tier busy, GPU tier middle, Waiting idle) makes the CPU tier the
    busiest every step, so every step moves KV both ways; within a set the
    drawn windows order the programs."""
    rng = _streams(seed, 7)[6]
    out = np.empty((steps, 3, P, k, 2), np.float32)
    for j, (r_lo, r_hi, a_lo, a_hi) in enumerate(ROTATION_SETS):
        out[:, j, :, :, 0] = rng.uniform(r_lo, r_hi, size=(steps, P, k))
        out[:, j, :, :, 1] = rng.uniform(a_lo, a_hi, size=(steps, P, k))
    return out


# --------------------------------------------------------------------------
# random small instances (parity and property tests)
# --------------------------------------------------------------------------
def random_instance(rng, P: int | None = None, max_blocks: int = 12, geom: Geometry | None = None,
                    tier_p=(0.5, 0.3, 0.2), extra_free: int | None = None, ties: bool = True) -> Instance:
    """A random, consistent pool state: GPU programs own distinct pages, the
    rest of the pool is free, CPU/Waiting programs own none."""
    if P is None:
        P = int(rng.integers(0, 24))
    if geom is None:
        geom = Geometry(int(rng.integers(1, 4)), int(rng.integers(1, 3)), int(rng.choice([1, 2, 4, 16])),
                        int(rng.choice([16, 32, 48, 512, 1152])), 0)
    nblk = rng.integers(0, max_blocks + 1, size=P).astype(np.uint32)
    tier = rng.choice(len(tier_p), size=P, p=list(tier_p)).astype(np.uint8)  # a 4th entry: SSD tier (3)
    gpu_blocks = int(nblk[tier == TIER_GPU].astype(np.int64).sum())
    if extra_free is None:
        extra_free = int(rng.integers(0, 2 * max_blocks + 1))
    NB = gpu_blocks + extra_free
    geom = Geometry(geom.layers, geom.planes, geom.block_tokens, geom.row_bytes, NB)
    tbl_off = np.zeros(P + 1, np.uint32)
    tbl_off[1:] = np.cumsum(nblk.astype(np.int64))
    tbl = np.full(int(tbl_off[-1]), NO_PAGE, np.uint32)
    perm = rng.permutation(NB).astype(np.uint32)
    used = 0
    for p in range(P):
        if tier[p] == TIER_GPU:
            n = int(nblk[p])
            tbl[tbl_off[p]:tbl_off[p] + n] = perm[used:used + n]
            used += n
    free_map = np.zeros(NB, np.uint8)
    free_map[perm[used:]] = 1
    busy = rng.random(P) < 0.5
    if ties:
        # windows from a small set of dyadic values: exact ties between programs
        vals = np.array([0.0, 0.25, 0.5, 1.0, 2.0, 4.0], np.float32)
        window = vals[rng.integers(0, vals.size, size=(P, WINDOW_K, 2))]
    else:
        window = draw_windows(rng, busy)
    status = rng.integers(0, 2, size=P).astype(np.uint8)
    ctx = nblk.astype(np.int64) * geom.block_tokens
    return Instance("random", geom, "fp16", ctx, nblk, busy, window, status, tbl_off, tbl, tier, free_map, 0)


# --------------------------------------------------------------------------
# content-addressed KV bytes
# --------------------------------------------------------------------------
def run_offset(p, i, q):
    """Bank offset of run (p, i, q); integer mixing on non-negative int64 only
    (identical on numpy arrays and torch int64 tensors)."""
    x = p * 0x9E3779B1 + i * 0x85EBCA77 + q * 0xC2B2AE3D + 0x27D4EB2F
    x = (x ^ (x >> 31)) & 0x7FFFFFFF
    x = x ^ (x >> 16)
    x = (x * 0x045D9F3B) & 0x7FFFFFFF
    x = x ^ (x >> 16)
    x = (x * 0x045D9F3B) & 0x7FFFFFFF
    x = x ^ (x >> 16)
    return x & (BANK - 1)


def run_tag(p, i, q):
    """32-bit tag written over the first four bytes of run (p, i, q)."""
    return ((p & 0x7FF) << 21) | ((i & 0x1FFF) << 8) | (q & 0xFF)


def make_bank(cfg_seed: int, dtype: str, run_bytes: int) -> np.ndarray:
    """uint16 bank of 2^22 N(0,1) values rounded to fp16/bf16 (round to nearest
    even), extended by one run so every window is a plain slice."""
    rng = _streams(cfg_seed)[4]
    v = rng.standard_normal(BANK).astype(np.float32)
    if dtype == "fp16":
        bits = v.astype(np.float16).view(np.uint16)
    else:
        u = v.view(np.uint32).astype(np.uint64)
        bits = ((u + 0x7FFF + ((u >> 16) & 1)) >> 16).astype(np.uint16)
    e = run_bytes // 2
    return np.concatenate([bits, bits[:e]])


def run_content(bank: np.ndarray, run_bytes: int, p, i, q) -> np.ndarray:
    """Expected bytes of runs (p, i, q) (scalars or equal-length arrays) -> uint8 [n][run_bytes]."""
    p = np.atleast_1d(np.asarray(p, np.int64))
    i = np.atleast_1d(np.asarray(i, np.int64))
    q = np.atleast_1d(np.asarray(q, np.int64))
    e = run_bytes // 2
    win = np.lib.stride_tricks.sliding_window_view(bank, e)
    out = win[run_offset(p, i, q)].copy()
    tag = run_tag(p, i, q).astype(np.uint32)
    out[:, 0] = (tag & 0xFFFF).astype(np.uint16)
    out[:, 1] = (tag >> 16).astype(np.uint16)
    return out.view(np.uint8).reshape(len(p), run_bytes)


def page_owners(inst: Instance):
    """(owner program, logical block) of every page, FREE_OWNER/page id for free pages."""
    NB = inst.geom.num_blocks
    owner_p = np.full(NB, FREE_OWNER, np.int64)
    owner_i = np.arange(NB, dtype=np.int64)
    for p in range(inst.P):
        if inst.tier[p] == TIER_GPU:
            pages = inst.tbl[inst.tbl_off[p]:inst.tbl_off[p + 1]].astype(np.int64)
            owner_p[pages] = p
            owner_i[pages] = np.arange(pages.size)
    return owner_p, owner_i


def fill_pool_np(inst: Instance, bank: np.ndarray) -> np.ndarray:
    """Host mirror of the pool, [planes][NB][run] bytes, holding each resident run's content."""
    g = inst.geom
    owner_p, owner_i = page_owners(inst)
    pool = np.empty(g.pool_bytes, np.uint8)
    view = pool.reshape(g.nplanes, g.num_blocks, g.run_bytes)
    for q in range(g.nplanes):
        if g.num_blocks:
            view[q] = run_content(bank, g.run_bytes, owner_p, owner_i, np.full(g.num_blocks, q))
    return pool


def program_host_content(inst: Instance, bank: np.ndarray, p: int) -> np.ndarray:
    """Program p's KV in the host layout [planes][nblk][run] bytes."""
    g = inst.geom
    n = int(inst.nblk[p])
    qq, ii = np.meshgrid(np.arange(g.nplanes), np.arange(n), indexing="ij")
    if n == 0:
        return np.zeros(0, np.uint8)
    return run_content(bank, g.run_bytes, np.full(qq.size, p), ii.ravel(), qq.ravel()).reshape(-1)


def fill_pool_torch(pool, inst: Instance, bank_dev, owner_p=None, owner_i=None, pages=None):
    """Device fill of the pool tensor (uint8, [planes][NB][run]) with content.
    ``pages`` restricts the fill to those page ids (int64 tensor on the device)."""
    import torch

    g = inst.geom
    e = g.run_bytes // 2
    if owner_p is None:
        op, oi = page_owners(inst)
        owner_p = torch.from_numpy(op).to(pool.device)
        owner_i = torch.from_numpy(oi).to(pool.device)
    win = torch.as_strided(bank_dev, (BANK, e), (1, 1))
    planes = pool.view(g.nplanes, g.num_blocks, g.run_bytes)
    for q in range(g.nplanes):
        dst = planes[q].view(torch.int16)
        if pages is None:
            offs = run_offset(owner_p, owner_i, q)
            torch.index_select(win, 0, offs, out=dst)
            tags = run_tag(owner_p, owner_i, q)
            dst.view(torch.int32)[:, 0] = torch.where(tags >= 2**31, tags - 2**32, tags).to(torch.int32)
        else:
            pp, ii = owner_p[pages], owner_i[pages]
            vals = torch.index_select(win, 0, run_offset(pp, ii, q))
            tags = run_tag(pp, ii, q)
            vals.view(torch.int32)[:, 0] = torch.where(tags >= 2**31, tags - 2**32, tags).to(torch.int32)
            dst[pages] = vals


def runs_torch(bank_dev, run_bytes: int, p, i, q):
    """Expected bytes of runs (p, i, q), generated on the device: p, i, q are
    int64 tensors of equal length (or Python ints for q) on bank_dev's device;
    returns int16 [n][run_bytes / 2]."""
    import torch

    e = run_bytes // 2
    win = torch.as_strided(bank_dev, (BANK, e), (1, 1))
    vals = torch.index_select(win, 0, run_offset(p, i, q))
    tags = run_tag(p, i, q)
    vals.view(torch.int32)[:, 0] = torch.where(tags >= 2**31, tags - 2**32, tags).to(torch.int32)
    return vals


def program_content_torch(inst: Instance, bank_dev, p: int, out=None):
    """Program p's KV in the host layout [planes][nblk][run], generated on the
    device (int16 tensor of nblk * block / 2 elements, written into ``out`` when given)."""
    import torch

    g = inst.geom
    n = int(inst.nblk[p])
    e = g.run_bytes // 2
    dev = bank_dev.device
    q = torch.arange(g.nplanes, device=dev, dtype=torch.int64).repeat_interleave(n)
    i = torch.arange(n, device=dev, dtype=torch.int64).repeat(g.nplanes)
    pp = torch.full_like(q, p)
    win = torch.as_strided(bank_dev, (BANK, e), (1, 1))
    vals = torch.index_select(win, 0, run_offset(pp, i, q))
    tags = run_tag(pp, i, q)
    vals.view(torch.int32)[:, 0] = torch.where(tags >= 2**31, tags - 2**32, tags).to(torch.int32)
    vals = vals.reshape(-1)
    if out is not None:
        out.copy_(vals)
        return out
    return vals


def eviction_blocks(rng, N: int, programs: int = 256, type_p=(0.5, 0.3, 0.2), tie_frac: float = 0.5,
                    horizon: int = 1 << 40, var_size: bool = False):
    """KV blocks for the typed eviction order: N blocks dealt to programs in
    contiguous runs; each program draws a type label (busy / idle / inactive
    with probabilities type_p) and a last-activity time in [0, horizon) us.
    A fraction tie_frac of programs stamp every block with that time (their
    whole prefix is touched by each request, so ties are common); the others'
    blocks are older by a random step per block.  Sizes: one unit per block,
    or 1..16 units (radix-tree nodes of varying token counts)."""
    programs = max(1, min(programs, max(N, 1)))
    cuts = np.sort(rng.choice(np.arange(1, max(N, 2)), size=min(programs - 1, max(N - 1, 0)), replace=False)) \
        if N > 1 else np.zeros(0, np.int64)
    owner = np.zeros(N, np.int64)
    if N:
        owner[cuts] = 1
        owner = np.cumsum(owner)
    P = int(owner[-1]) + 1 if N else 0
    ptype = rng.choice(3, size=P, p=list(type_p)).astype(np.uint8)
    ptime = rng.integers(0, horizon, size=P, dtype=np.int64)
    tied = rng.random(P) < tie_frac
    steps = rng.integers(1, 1 << 20, size=N, dtype=np.int64)
    t = ptime[owner] - np.where(tied[owner], 0, steps)
    t = np.clip(t, 0, None).astype(np.uint64)
    size = rng.integers(1, 17, size=N).astype(np.uint32) if var_size else None
    return ptype[owner], t, size
