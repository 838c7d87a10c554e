"""The C ABI used from C: tests/c_abi/roundtrip drives libmori with plain
pointers and HIP runtime calls (no Python, no torch) through three rebalances,
the kernel timing records, a typed eviction order on both tiers and a
multi-replica admission with both rules, and compares every result with the C
oracle bit for bit.  Run as a child process, one per program count, covering
the rank kernel's three shapes."""
import os
import subprocess

import pytest

pytestmark = pytest.mark.gpu

BIN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "c_abi", "roundtrip")


@pytest.mark.parametrize("programs,seed", [(200, 1), (700, 2), (3000, 3)])
def test_c_program_matches_oracle(programs, seed):
    assert os.path.exists(BIN), "tests/c_abi/roundtrip is not built: run __graft_entry__.build()"
    print(f"roundtrip programs={programs} seed={seed}", flush=True)
    res = subprocess.run([BIN, str(programs), str(seed)], capture_output=True, text=True, timeout=120)
    print(res.stdout, res.stderr, flush=True)
    assert res.returncode == 0, res.stderr[-2000:]
    assert res.stdout.strip().endswith("ok")
