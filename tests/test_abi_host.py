"""CPU-only checks of the C ABI: the library loads, exports every function the
header declares, and rejects bad arguments on the host before touching HIP."""
import ctypes as C
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def M():
    from paper_2606_00866_amd import build, mori
    if not os.path.exists(mori.LIB_PATH):
        build.build()
    mori.lib()
    return mori


def header_functions():
    text = open(os.path.join(ROOT, "include", "mori.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(mori_[a-z_]+)\s*\(", text)))


def test_exports_every_declared_function(M):
    declared = header_functions()
    assert set(declared) == set(M.EXPORTS), declared
    for name in declared:
        assert hasattr(M.lib(), name), name


def test_header_constants_match_binding(M):
    text = open(os.path.join(ROOT, "include", "mori.h")).read()
    for name, val in re.findall(r"#define (MORI_[A-Z0-9_]+) \(?(-?(?:0x)?[0-9A-Fa-f]+)u?\)?", text):
        if hasattr(M, name):
            assert getattr(M, name) == int(val, 0), name


def test_strerror(M):
    assert M.mori_strerror(0) == "ok"
    assert M.mori_strerror(M.MORI_EDEVICE) == "device-side validation failed"
    assert M.mori_strerror(12345) == "unknown error"


def test_create_rejects_bad_pools_on_host(M):
    ok = dict(layers=2, planes=2, block_tokens=16, row_bytes=512, num_blocks=8, base=0x100000)
    for bad in (dict(base=0), dict(base=0x100010), dict(row_bytes=24), dict(row_bytes=0), dict(layers=0),
                dict(planes=0), dict(block_tokens=0), dict(num_blocks=0), dict(num_blocks=0xFFFFFFFF)):
        rc, ctx = M.mori_create(M.mori_pool(**{**ok, **bad}), 8)
        assert rc == M.MORI_EINVAL and not ctx.value, bad
    for mp in (0, M.MORI_MAX_PROGRAMS + 1):
        rc, _ = M.mori_create(M.mori_pool(**ok), mp)
        assert rc == M.MORI_EINVAL
    assert M.lib().mori_create(None, 8, 0, 0, C.byref(C.c_void_p())) == M.MORI_EINVAL


def test_create_flags_checked_on_host(M):
    """The copy-stream choice is the caller's explicit flag: any other bit is
    rejected before the HIP runtime is touched."""
    ok = dict(layers=2, planes=2, block_tokens=16, row_bytes=512, num_blocks=8, base=0x100000)
    for flags in (2, 4, 0x80000000, M.MORI_CREATE_COPY_STREAMS | 2):
        rc, ctx = M.mori_create(M.mori_pool(**ok), 8, 0, flags)
        assert rc == M.MORI_EINVAL and not ctx.value, flags


def test_tierpool_copy_stream_choice(monkeypatch):
    from paper_2606_00866_amd import tiering

    for env, want in (("8", 8), ("32", 32), ("4", 4), ("", 4), ("x", 4), ("0", 4)):
        monkeypatch.setenv("GPU_MAX_HW_QUEUES", env)
        assert tiering.hw_queues() == want
    monkeypatch.delenv("GPU_MAX_HW_QUEUES")
    assert tiering.hw_queues() == 4


def test_null_context_calls(M):
    assert M.mori_rank_partition(None, M.mori_programs(), M.mori_budget()) == M.MORI_EINVAL
    assert M.mori_plan_wait(None)[0] == M.MORI_EINVAL
    assert M.mori_kv_swap_out(None, 0) == M.MORI_EINVAL
    assert M.mori_kv_swap_in(None, 0) == M.MORI_EINVAL
    assert M.mori_query(None, M.MORI_Q_LAST_MODE)[0] == M.MORI_EINVAL
    assert M.mori_register(None, 0, 0) == M.MORI_EINVAL
    assert M.mori_destroy(None) == M.MORI_OK
    assert M.mori_host_alloc(0)[0] == M.MORI_EINVAL
    assert M.mori_host_free(0) == M.MORI_OK
