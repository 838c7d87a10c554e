"""The exact content check used after every full-size and churn step
(workload/check.py), pinned on the CPU: it passes on a correct tier state and
names the first wrong run for a corrupted page, a corrupted host buffer, two
swapped table entries and a host buffer of the wrong program."""
import numpy as np
import torch

from workload import (Geometry, check_tier_bytes, fill_pool_torch, make_bank, program_host_content, random_instance,
                      run_content)


def _state(seed=3):
    rng = np.random.default_rng(seed)
    geom = Geometry(layers=2, planes=2, block_tokens=4, row_bytes=64, num_blocks=0)
    while True:
        inst = random_instance(rng, P=10, max_blocks=6, geom=geom, tier_p=(0.5, 0.3, 0.1, 0.1), extra_free=3)
        if (((inst.tier == 0) & (inst.nblk > 1)).sum() >= 2 and
                ((inst.tier == 1) & (inst.nblk > 0)).any()):
            break
    g = inst.geom
    bank = make_bank(11, "bf16", g.run_bytes)
    bank_dev = torch.from_numpy(bank.view(np.int16))
    pool = torch.zeros(g.pool_bytes, dtype=torch.uint8)
    fill_pool_torch(pool, inst, bank_dev)
    host = {p: program_host_content(inst, bank, p).copy() for p in range(inst.P) if inst.tier[p] in (1, 3)}
    return inst, bank, bank_dev, pool, host


def _check(inst, pool, bank_dev, host, tbl=None):
    return check_tier_bytes(pool, inst.geom, inst.tbl_off, inst.tbl if tbl is None else tbl, inst.tier, bank_dev,
                            lambda p: host[p], chunk_bytes=3 * inst.geom.run_bytes)


def test_correct_state_passes_and_counts_every_run():
    inst, bank, bank_dev, pool, host = _state()
    r = _check(inst, pool, bank_dev, host)
    g = inst.geom
    res = inst.nblk[(inst.tier == 0)].sum() + inst.nblk[(inst.tier == 1) | (inst.tier == 3)].sum()
    assert r["ok"] and r["gpu_runs"] + r["host_runs"] == int(res) * g.nplanes
    # the fill really is the content-addressed value
    p = int(np.flatnonzero((inst.tier == 0) & (inst.nblk > 0))[0])
    page = int(inst.tbl[inst.tbl_off[p]])
    got = pool.numpy().reshape(g.nplanes, g.num_blocks, g.run_bytes)[1, page]
    assert np.array_equal(got, run_content(bank, g.run_bytes, p, 0, 1)[0])


def test_corrupted_pool_byte_is_found():
    inst, bank, bank_dev, pool, host = _state()
    g = inst.geom
    p = int(np.flatnonzero((inst.tier == 0) & (inst.nblk > 1))[0])
    page = int(inst.tbl[inst.tbl_off[p] + 1])
    view = pool.view(g.nplanes, g.num_blocks, g.run_bytes)
    view[g.nplanes - 1, page, g.run_bytes - 1] ^= 1  # last byte of the last plane: past the tag
    r = _check(inst, pool, bank_dev, host)
    assert not r["ok"] and r["where"] == "pool page"
    assert (r["program"], r["block"], r["plane"], r["page"]) == (p, 1, g.nplanes - 1, page)


def test_swapped_table_entries_are_found():
    inst, bank, bank_dev, pool, host = _state()
    gpu = np.flatnonzero((inst.tier == 0) & (inst.nblk > 1))
    tbl = inst.tbl.copy()
    a, b = int(inst.tbl_off[gpu[0]]), int(inst.tbl_off[gpu[1]])
    tbl[a], tbl[b] = tbl[b], tbl[a]
    r = _check(inst, pool, bank_dev, host, tbl=tbl)
    assert not r["ok"] and r["where"] == "pool page" and r["program"] == gpu[0] and r["block"] == 0


def test_corrupted_host_byte_and_wrong_buffer_are_found():
    inst, bank, bank_dev, pool, host = _state()
    g = inst.geom
    p = int(np.flatnonzero((inst.tier == 1) & (inst.nblk > 0))[0])
    n = int(inst.nblk[p])
    bad = {k: v.copy() for k, v in host.items()}
    bad[p][((g.nplanes - 1) * n + n - 1) * g.run_bytes + 7] ^= 0x80
    r = _check(inst, pool, bank_dev, bad)
    assert not r["ok"] and (r["where"], r["program"], r["block"], r["plane"]) == ("host buffer", p, n - 1,
                                                                                g.nplanes - 1)
    # another program's bytes in the buffer (same size): the tags differ
    q = p + 1 if p + 1 < inst.P else p - 1
    inst.nblk[q] = n
    other = program_host_content(inst, bank, q)
    bad = {k: v.copy() for k, v in host.items()}
    bad[p][:] = other
    assert not _check(inst, pool, bank_dev, bad)["ok"]
