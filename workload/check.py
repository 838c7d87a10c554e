"""Exact check of a tier state against the content-addressed KV values.

Every run of the workload holds a value that can be regenerated on its own
from (program, block, plane) (``synth.run_content``), so the bytes a
rebalance leaves behind can be compared in full with what they must be,
without a mirror of the pool: every page of every GPU-resident program (found
through its block table) and every host buffer of a CPU- or SSD-tier program
(layout [plane][block][run]).  The expected runs are generated on the device
and compared there, chunk by chunk; nothing here belongs to the placement
method.
"""
from __future__ import annotations

import numpy as np

from .synth import runs_torch

NO_PAGE = 0xFFFFFFFF


def check_tier_bytes(pool, geom, tbl_off, tbl, tier, bank_dev, host_view, programs=None,
                     chunk_bytes: int = 1 << 29) -> dict:
    """Compares every resident run with its content-addressed value.

    pool: uint8 device tensor [planes][num_blocks][run]; tbl_off, tbl, tier:
    numpy state after the step (tables of non-GPU programs hold no page);
    host_view(p): uint8 numpy view of program p's host buffer; programs: bool
    mask of the programs whose KV is defined (all when None).  Returns
    {"ok": True, ...counts} or {"ok": False, "where": ...} at the first
    mismatch."""
    import torch

    dev = pool.device
    P = int(tier.size)
    nblk = np.diff(np.asarray(tbl_off, np.int64))
    mask = np.ones(P, bool) if programs is None else np.asarray(programs, bool)
    e = geom.run_bytes // 2
    planes = pool.view(geom.nplanes, geom.num_blocks, geom.run_bytes).view(torch.int16)
    per_chunk = max(1, chunk_bytes // geom.run_bytes)

    # GPU tier: every page of every resident program, plane by plane
    gpu = np.flatnonzero((tier == 0) & (nblk > 0) & mask)
    gpu_runs = 0
    if gpu.size:
        owner = np.concatenate([np.full(nblk[p], p, np.int64) for p in gpu])
        block = np.concatenate([np.arange(nblk[p], dtype=np.int64) for p in gpu])
        pages = np.concatenate([tbl[tbl_off[p]:tbl_off[p + 1]] for p in gpu]).astype(np.int64)
        if (pages >= geom.num_blocks).any():
            return {"ok": False, "where": "a resident program's table holds no valid page"}
        o_d, b_d, g_d = (torch.from_numpy(a).to(dev) for a in (owner, block, pages))
        for q in range(geom.nplanes):
            for a in range(0, pages.size, per_chunk):
                sl = slice(a, a + per_chunk)
                want = runs_torch(bank_dev, geom.run_bytes, o_d[sl], b_d[sl], q)
                got = planes[q].index_select(0, g_d[sl])
                if not torch.equal(got, want):
                    bad = int((got != want).any(dim=1).nonzero()[0, 0]) + a
                    return {"ok": False, "where": "pool page", "program": int(owner[bad]),
                            "block": int(block[bad]), "plane": q, "page": int(pages[bad])}
            gpu_runs += pages.size

    # CPU and SSD tiers: every host buffer, a few planes at a time
    host = np.flatnonzero(((tier == 1) | (tier == 3)) & (nblk > 0) & mask)
    host_runs = 0
    for p in host:
        n = int(nblk[p])
        view = host_view(int(p))
        if view.size != n * geom.block_bytes:
            return {"ok": False, "where": "host buffer size", "program": int(p)}
        qs = max(1, per_chunk // n)
        for q0 in range(0, geom.nplanes, qs):
            q1 = min(geom.nplanes, q0 + qs)
            got = torch.from_numpy(view[q0 * n * geom.run_bytes:q1 * n * geom.run_bytes]).to(dev)
            got = got.view(torch.int16).view((q1 - q0) * n, e)
            qq = torch.arange(q0, q1, device=dev, dtype=torch.int64).repeat_interleave(n)
            ii = torch.arange(n, device=dev, dtype=torch.int64).repeat(q1 - q0)
            want = runs_torch(bank_dev, geom.run_bytes, torch.full_like(qq, int(p)), ii, qq)
            if not torch.equal(got, want):
                bad = int((got != want).any(dim=1).nonzero()[0, 0])
                return {"ok": False, "where": "host buffer", "program": int(p), "block": bad % n,
                        "plane": q0 + bad // n}
        host_runs += n * geom.nplanes
    return {"ok": True, "gpu_runs": gpu_runs, "host_runs": host_runs,
            "bytes": (gpu_runs + host_runs) * geom.run_bytes}
