"""bench.py's command-line contract on the CPU: it runs on exactly one GPU and
says so for any other count, before touching torch or the GPU."""
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_is_refused_with_a_message():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
    assert r.stdout == ""


def test_help_lists_the_driver_flags():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--help"], capture_output=True, text=True,
                       timeout=120)
    assert r.returncode == 0
    for flag in ("--gpus", "--steps", "--warmup", "--workload", "--schedule"):
        assert flag in r.stdout


def test_link_bound_is_a_lower_bound_per_step():
    """The per-step link bound: each direction alone at its one-way rate, both
    within the two-way capacity; the largest of the three is the bound."""
    sys.path.insert(0, ROOT)
    import bench

    pk = {"d2h_GBps": 50.0, "h2d_GBps": 60.0, "bidir_GBps": 100.0}
    assert bench.link_bound_s(0, 0, pk) == 0.0
    assert bench.link_bound_s(10e9, 0, pk) == 10e9 / 50e9               # one-way D2H
    assert bench.link_bound_s(0, 12e9, pk) == 12e9 / 60e9               # one-way H2D
    assert bench.link_bound_s(20e9, 20e9, pk) == 40e9 / 100e9           # balanced: the two-way capacity
    assert bench.link_bound_s(30e9, 1e9, pk) == 30e9 / 50e9             # D2H-heavy: its own rate
    # never below any of the three single limits
    for o, i in ((1e9, 2e9), (7e9, 3e9), (5e9, 5e9)):
        t = bench.link_bound_s(o, i, pk)
        assert t >= o / 50e9 and t >= i / 60e9 and t >= (o + i) / 100e9


def test_split_model_of_two_unpaced_copy_streams():
    """Both directions at the measured two-way split until the smaller is
    done, then the larger alone: worked by hand."""
    sys.path.insert(0, ROOT)
    import bench

    pk = {"d2h_GBps": 60.0, "h2d_GBps": 60.0, "bidir_split_GBps": {"d2h": 40.0, "h2d": 50.0}}
    assert bench.split_model_s(0, 0, pk) == 0.0
    assert bench.split_model_s(12e9, 0, pk) == 12e9 / 60e9              # one direction: its own rate
    assert bench.split_model_s(0, 6e9, pk) == 6e9 / 60e9
    # D2H 8 GB, H2D 5 GB: H2D done at 0.1 s (D2H has moved 4 GB), 4 GB left at 60 GB/s
    assert abs(bench.split_model_s(8e9, 5e9, pk) - (0.1 + 4e9 / 60e9)) < 1e-12
    # D2H 2 GB, H2D 10 GB: D2H done at 0.05 s (H2D has moved 2.5 GB), 7.5 GB left at 60 GB/s
    assert abs(bench.split_model_s(2e9, 10e9, pk) - (0.05 + 7.5e9 / 60e9)) < 1e-12
    # never below the link bound built from the same figures
    pk2 = dict(pk, bidir_GBps=90.0)
    for o, i in ((1e9, 2e9), (7e9, 3e9), (5e9, 5e9)):
        assert bench.split_model_s(o, i, pk) >= bench.link_bound_s(o, i, pk2) - 1e-12


def test_steady_two_way_window_counts_bytes_done():
    sys.path.insert(0, ROOT)
    import bench

    ends = [1.0, 2.0, 3.0, 4.0]  # four chunks of 10 bytes, one per second
    assert bench.bytes_done_by(ends, 4.0, 10) == 40.0
    assert bench.bytes_done_by(ends, 2.0, 10) == 20.0
    assert bench.bytes_done_by(ends, 2.5, 10) == 25.0
    assert bench.bytes_done_by(ends, 0.5, 10) == 5.0
    assert bench.bytes_done_by([1.0, 3.0], 2.0, 10) == 15.0  # the straddling chunk's own span
    assert bench.bytes_done_by(ends, 9.0, 10) == 40.0


def test_rotation_schedule_gives_each_tier_its_set():
    import numpy as np

    sys.path.insert(0, ROOT)
    import bench
    from oracle import oracle
    from workload import MLA, make_instance, rotation_windows

    inst = make_instance(MLA, scale=1 / 64)
    window_of = bench.schedule_windows(np, inst, "rotate", 4)
    rot = rotation_windows(MLA.seed, inst.P, 4)
    tier = np.arange(inst.P, dtype=np.uint8) % 3
    w = window_of(2, tier)
    for p in (0, 1, 2, 7):
        assert np.array_equal(w[p], rot[2, bench.ROT_SET_OF_TIER[tier[p]], p])
    # CPU tier busiest, then GPU, then Waiting, by Eq. 1
    rc, iota = oracle.idleness(w)
    assert rc == oracle.OK
    assert iota[tier == 1].max() < iota[tier == 0].min() and iota[tier == 0].max() < iota[tier == 2].min()
    rev = bench.schedule_windows(np, inst, "reverse", 4)
    assert np.array_equal(rev(1, tier), inst.window[:, :, ::-1])
