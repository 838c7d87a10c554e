"""Readers for the hand-derived fixtures under tests/golden/."""
import os
from fractions import Fraction

import numpy as np

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")
NONE = 0xFFFFFFFF


def idleness_cases():
    cases = []
    for line in open(os.path.join(GOLDEN, "idleness_eq1.txt")):
        line = line.strip()
        if not line or line.startswith("#"):
            continue
        r, a, exact = [s.split() for s in line.split("|")]
        cases.append((np.array([float(x) for x in r], np.float32), np.array([float(x) for x in a], np.float32),
                      Fraction(exact[0])))
    return cases


def _kv_blocks(path):
    sections, cur = {}, {}
    for line in open(path):
        line = line.strip()
        if not line or line.startswith("#"):
            continue
        if line.startswith("[") and line.endswith("]"):
            cur = sections.setdefault(line[1:-1], {})
            continue
        k, v = line.split(":", 1)
        cur[k.strip()] = v.strip()
    return sections, cur


def boundary_case():
    _, kv = _kv_blocks(os.path.join(GOLDEN, "boundary_worked.txt"))
    return kv


def _tables(s):
    out = []
    for grp in s.split("|"):
        out.append([NONE if t == "-" else int(t) for t in grp.split()])
    return out


def plan_cases():
    sections, _ = _kv_blocks(os.path.join(GOLDEN, "plan_worked.txt"))
    res = {}
    for name, kv in sections.items():
        d = dict(kv)
        d["blocks"] = [int(x) for x in kv["blocks"].split()]
        d["tier"] = [int(x) for x in kv["tier"].split()]
        d["new_tier"] = [int(x) for x in kv["new_tier"].split()]
        d["tables"] = _tables(kv["tables"])
        d["new_tables"] = _tables(kv["new_tables"])
        d["free"] = [int(x) for x in kv["free"].split()]
        d["status"] = [STATUS[x] for x in kv["status"].split()] if "status" in kv else None
        d["flags"] = kv.get("flags", "").split()
        d["new_free"] = [int(x) for x in kv["new_free"].split()]
        d["idleness"] = [float(x) for x in kv["idleness"].split()]
        d["summary"] = {k: int(v) for k, v in (t.split("=") for t in kv["summary"].split())}
        for key in ("num_blocks", "gpu_budget", "cpu_budget"):
            d[key] = int(kv[key])
        res[name] = d
    return res


def round_to_f32(fr: Fraction) -> np.float32:
    """Correctly rounded (nearest, ties to even) binary32 value of an exact rational."""
    x = np.float32(float(fr))
    cands = [np.nextafter(x, np.float32(-np.inf)), x, np.nextafter(x, np.float32(np.inf))]
    return min(cands, key=lambda c: (abs(Fraction(float(c)) - fr), int(np.float32(c).view(np.uint32)) & 1))


STATUS = {"R": 0, "A": 1, "N": 2}


def incremental_cases():
    sections, _ = _kv_blocks(os.path.join(GOLDEN, "incremental_worked.txt"))
    res = {}
    for name, kv in sections.items():
        d = {k: [int(x) for x in kv[k].split()] for k in ("blocks", "tier", "new_tier", "order")}
        d["status"] = [STATUS[x] for x in kv["status"].split()]
        d["idleness"] = [float(x) for x in kv["idleness"].split()]
        for key in ("gpu_budget", "cpu_budget", "skip_fit", "m_gpu", "m_cpu"):
            d[key] = int(kv[key])
        res[name] = d
    return res


def ssd_cases():
    sections, _ = _kv_blocks(os.path.join(GOLDEN, "ssd_worked.txt"))
    res = {}
    for name, kv in sections.items():
        d = {k: [int(x) for x in kv[k].split()] for k in ("blocks", "tier", "new_tier", "category", "m")}
        d["idleness"] = [float(x) for x in kv["idleness"].split()]
        for key in ("gpu_budget", "cpu_budget", "ssd_budget", "skip_fit"):
            d[key] = int(kv[key])
        res[name] = d
    return res


def replica_cases():
    sections, _ = _kv_blocks(os.path.join(GOLDEN, "replica_worked.txt"))
    res = {}
    for name, kv in sections.items():
        d = {k: [int(x) for x in kv[k].split()] for k in ("bytes", "room", "replica", "room_after")}
        d["status"] = [STATUS[x] for x in kv["status"].split()]
        d["idleness"] = [float(x) for x in kv["idleness"].split()]
        d["best_fit"] = int(kv["best_fit"])
        res[name] = d
    return res
