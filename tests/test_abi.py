"""C-ABI boundary checks that need no GPU: the library loads, exports every
entry point include/dps.h declares, and rejects bad arguments on the host
before launching anything."""
import ctypes
import os
import re

import pytest

from paper_2609_34380_amd import dps

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "dps.h")


def _declared():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(dps_[a-z0-9_]+)\s*\(", text)))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(dps.LIB_PATH):
        import __graft_entry__
        __graft_entry__.build()
    return dps.load_library()


def test_header_declares_the_boundary():
    names = _declared()
    for expected in ("dps_select_enc", "dps_split", "dps_merge", "dps_restore", "dps_backup",
                     "dps_linear",
                     "dps_linear_grouped", "dps_quant_rows_e4m3", "dps_workspace_bytes",
                     "dps_status_str", "dps_last_error"):
        assert expected in names


def test_every_declared_symbol_is_exported(lib):
    for name in _declared():
        assert hasattr(lib, name), name
    assert set(_declared()) == set(dps.EXPORTED)


def test_status_strings(lib):
    for code in range(8):
        assert lib.dps_status_str(code) != b"unknown status"
    assert lib.dps_status_str(0) == b"ok"
    assert lib.dps_status_str(7) == b"timed out"
    assert lib.dps_status_str(8) == b"unknown status"


def _weight(n=64, k=64, experts=1, enc=0, hi=0x1000, pool=0x2000, slots=0x3000,
            pool_bytes=1 << 16, n_chunks=1, log2=16):
    res = dps.CResidual(pool, pool_bytes, slots, n_chunks, log2)
    return dps.CWeight(hi, res, experts, n, k, enc)


def _linear(lib, mode=0, flags=0, x=0x4000, m=4, w=None, y=0x5000, ws=None, ws_bytes=0):
    w = w if w is not None else _weight()
    return lib.dps_linear(mode, flags, x, m, ctypes.byref(w), y, ws, ws_bytes, None)


@pytest.mark.parametrize("kwargs,status", [
    (dict(mode=7), 1),
    (dict(flags=9), 1),
    (dict(mode=0, flags=1), 1),                      # FP8 activations need fast mode
    (dict(w=_weight(k=40)), 1),                      # k % 16 != 0
    (dict(w=_weight(k=(1 << 30) + 16)), 1),          # k above 2^30
    (dict(w=_weight(n=1 << 31)), 1),                 # n above 2^31-1
    (dict(w=_weight(n=0)), 1),
    (dict(w=_weight(enc=2)), 1),                     # unknown nested encoding
    (dict(w=_weight(experts=2)), 1),                 # dense call with stacked experts
    (dict(w=_weight(hi=0x1001)), 2),                 # misaligned plane
    (dict(x=0x4008), 2),
    (dict(w=_weight(pool=0)), 1),                    # full mode needs a pool
    (dict(w=_weight(slots=0)), 1),
    (dict(w=_weight(log2=3)), 1),
    (dict(w=_weight(pool_bytes=100)), 1),            # smaller than one chunk
    (dict(w=_weight(n=1024, k=1024, n_chunks=1, log2=16)), 1),  # table too short
    (dict(m=-1), 1),
    (dict(x=0), 1),
])
def test_linear_rejects_bad_arguments(lib, kwargs, status):
    assert _linear(lib, **kwargs) == status
    assert lib.dps_last_error()


def test_linear_zero_rows_is_a_noop(lib):
    assert _linear(lib, m=0) == 0


def test_fast_mode_ignores_residual_descriptor(lib):
    # a fast-mode call with an empty residual fails only later (x is NULL here)
    w = _weight(pool=0, slots=0, pool_bytes=0, n_chunks=0, log2=0)
    assert _linear(lib, mode=1, x=0, w=w) == 1
    assert b"x or y" in lib.dps_last_error()


def test_grouped_rejects_bad_arguments(lib):
    w = _weight(experts=4)
    args = lambda **kw: (kw.get("mode", 1), kw.get("flags", 0), kw.get("x", 0x4000),
                         kw.get("off", 0x6000), kw.get("rows", 8), ctypes.byref(w),
                         kw.get("y", 0x5000), None, 0, None)
    assert lib.dps_linear_grouped(*args(flags=2)) == 1            # unknown flags
    assert lib.dps_linear_grouped(*args(mode=0, flags=1)) == 1    # FP8 needs fast mode
    assert lib.dps_linear_grouped(*args(flags=1)) == 4            # FP8 staging: no workspace
    assert lib.dps_linear_grouped(*args(off=0)) == 1
    assert lib.dps_linear_grouped(*args(off=0x6002)) == 2
    assert lib.dps_linear_grouped(*args(rows=-3)) == 1
    assert lib.dps_linear_grouped(*args(rows=0)) == 0


def test_split_merge_reject_bad_arguments(lib):
    # every call here fails validation (or is empty) before any launch
    res = dps.CResidual(0x2000, 1 << 8, 0x3000, 4, 8)
    bad = dps.CResidual(0x2000, 1 << 8, 0x3000, 3, 8)   # 3 chunks of 256 < 1024 bytes
    for enc in (0, 1):
        assert lib.dps_split(enc, 0x1000, 1024, 0x4000, ctypes.byref(bad), None) == 1
        assert lib.dps_split(enc, 0x1000, -1, 0x4000, ctypes.byref(res), None) == 1
        assert lib.dps_split(enc, 0x1000, 0, 0x4000, ctypes.byref(res), None) == 0
        assert lib.dps_split(enc, 0x1004, 1024, 0x4000, ctypes.byref(res), None) == 2
        assert lib.dps_merge(enc, 0x4000, None, 1024, 0x1000, None) == 1
        assert lib.dps_merge(enc, 0x4000, ctypes.byref(bad), 1024, 0x1000, None) == 1
    assert lib.dps_split(2, 0x1000, 1024, 0x4000, ctypes.byref(res), None) == 1
    assert lib.dps_merge(-1, 0x4000, ctypes.byref(res), 1024, 0x1000, None) == 1
    assert lib.dps_select_enc(0x1000, -1, 0x2000, None) == 1
    assert lib.dps_select_enc(0x1000, 64, 0, None) == 1
    assert lib.dps_select_enc(0x1000, 64, 0x2002, None) == 2
    assert lib.dps_select_enc(0x1008, 64, 0x2000, None) == 2
    assert lib.dps_select_enc(0, 64, 0x2000, None) == 1
    assert lib.dps_quant_rows_e4m3(0x1000, 4, 24, 0x2000, 0x3000, None) == 1
    assert lib.dps_quant_rows_e4m3(0x1000, 0, 32, 0x2000, 0x3000, None) == 0
    assert lib.dps_quant_rows_e4m3(0x1000, 4, (1 << 30) + 16, 0x2000, 0x3000, None) == 1


def test_restore_backup_reject_bad_arguments(lib):
    # every call here fails validation (or is empty) before any copy is enqueued
    res = dps.CResidual(0x2000, 4 << 8, 0x3000, 4, 8)   # 4 pool slots of 256 bytes
    good = (ctypes.c_int32 * 4)(3, 0, 2, 1)
    outside = (ctypes.c_int32 * 4)(3, 0, 4, 1)          # slot 4 is past the pool
    negative = (ctypes.c_int32 * 4)(3, -1, 2, 1)
    bk = 0x10000
    P = ctypes.c_void_p
    def restore(backup=bk, numel=1000, r=res, slots=good, c0=0, c1=4, copy=4096):
        return lib.dps_restore(backup, numel, ctypes.byref(r) if r is not None else None,
                               ctypes.cast(slots, P) if slots is not None else None,
                               c0, c1, copy, None)
    assert restore(numel=-1) == 1
    assert restore(copy=0) == 1
    assert restore(r=None) == 1
    assert restore(c0=-1) == 1
    assert restore(c0=3, c1=2) == 1
    assert restore(c1=5) == 1                           # ceil(1000 / 256) = 4 chunks
    assert restore(backup=0) == 1
    assert restore(slots=None) == 1
    assert restore(slots=outside) == 1
    assert restore(slots=negative, c0=0, c1=4) == 1
    assert restore(c0=2, c1=2) == 0                     # empty range: nothing to do
    assert restore(numel=2000) == 1                     # 8 chunks > n_chunks 4
    assert lib.dps_backup(ctypes.byref(res), ctypes.cast(good, P), -1, bk, 4096, None) == 1
    assert lib.dps_backup(ctypes.byref(res), ctypes.cast(good, P), 1000, bk, 0, None) == 1
    assert lib.dps_backup(ctypes.byref(res), ctypes.cast(outside, P), 1000, bk, 4096, None) == 1
    assert lib.dps_backup(ctypes.byref(res), None, 1000, bk, 4096, None) == 1
    assert lib.dps_backup(ctypes.byref(res), ctypes.cast(good, P), 1000, None, 4096, None) == 1
    assert lib.dps_backup(ctypes.byref(res), ctypes.cast(good, P), 0, None, 4096, None) == 0


def test_workspace_query(lib):
    assert lib.dps_workspace_bytes(0, 0, 0, 64, 64, 1) == 0
    # FP8 activations always need room for the quantized copy
    assert lib.dps_workspace_bytes(1, 1, 2048, 4096, 4096, 1) >= 2048 * 4096


@pytest.mark.parametrize("mode", [0, 1], ids=["full", "fast"])
def test_planner_whole_rows_up_to_16_tokens(lib, mode):
    """Dense calls of up to 16 tokens run on whole-row kernels (row GEMV or
    the 16-row-group MFMA kernel): K is never split, so no workspace.  The
    hidden-4096 layers and awkward shapes alike."""
    for m, n, k in ((1, 4096, 4096), (2, 28672, 4096), (3, 28672, 4096), (4, 4096, 14336),
                    (8, 6144, 4096), (8, 28672, 4096), (16, 4096, 14336), (16, 33000, 1040),
                    (1, 64, 33024)):
        assert lib.dps_workspace_bytes(mode, 0, m, n, k, 1) == 0, (m, n, k)


@pytest.mark.parametrize("mode", [0, 1], ids=["full", "fast"])
def test_planner_splits_k_for_narrow_layers_beyond_16_tokens(lib, mode):
    """From 17 tokens on, the 4096 x 4096 layer has too few 128-row weight
    tiles to fill the chip, so K is split and the fp32 partials [splits][m][n]
    need workspace; the plan does not depend on the mode."""
    for m in (17, 32, 128):
        ws = lib.dps_workspace_bytes(mode, 0, m, 4096, 4096, 1)
        assert ws >= 2 * m * 4096 * 4, (m, ws)
        assert ws == lib.dps_workspace_bytes(1 - mode, 0, m, 4096, 4096, 1)


def test_plan_info_names_the_kernel_of_each_shape_class(lib):
    """The planner's choice, read through dps_plan_info, for one shape of each
    kernel family (on a 256-CU part, or when no device is visible)."""
    from paper_2609_34380_amd import dps as d
    assert d.plan_info(0, "fp16", 1, 4096, 4096)["kernel"] == "gemv"
    assert d.plan_info(1, "fp16", 8, 6144, 4096)["kernel"] == "rows"
    p = d.plan_info(1, "fp16", 8, 4096, 4096, experts=8)
    assert p["kernel"] == "decode"
    p = d.plan_info(0, "fp16", 256, 28672, 4096)
    assert (p["kernel"], p["tile_rows"], p["tile_tokens"], p["splits"]) == ("gemm_f16", 128, 128, 1)
    p = d.plan_info(0, "fp16", 2048, 6144, 4096)       # 192 large tiles: the 128 x 128 tile
    assert (p["kernel"], p["tile_rows"], p["tile_tokens"], p["splits"]) == ("gemm_f16", 128, 128, 1)
    p = d.plan_info(0, "fp16", 2048, 28672, 4096)      # 896 large tiles fill the chip
    assert (p["kernel"], p["tile_rows"], p["tile_tokens"], p["splits"]) == ("gemm_f16", 256, 256, 1)
    p = d.plan_info(1, "fp16", 2048, 4096, 14336)      # 128 tiles, two K ranges
    assert (p["kernel"], p["tile_rows"], p["tile_tokens"], p["splits"]) == ("gemm_f16", 256, 256, 2)
    p = d.plan_info(1, "fp16", 512, 4096, 14336)       # 32 tiles would need 8 ranges
    assert (p["kernel"], p["tile_rows"]) == ("gemm_f16", 128)
    p = d.plan_info(1, "fp16", 4096, 4096, 4096, experts=2)   # grouped calls keep 128 rows
    assert (p["kernel"], p["tile_rows"]) == ("gemm_f16", 128)
    p = d.plan_info(1, "fp8", 4096, 4096, 1024)
    assert (p["kernel"], p["tile_rows"], p["tile_tokens"]) == ("gemm_fp8", 256, 256)
    p = d.plan_info(1, "fp8", 2048, 6144, 4096)
    assert (p["kernel"], p["tile_rows"], p["tile_tokens"]) == ("gemm_fp8", 256, 128)
    p = d.plan_info(1, "fp8", 8192, 28672, 4096, experts=8)   # grouped: 128-token tiles
    assert (p["kernel"], p["tile_rows"], p["tile_tokens"]) == ("gemm_fp8", 256, 128)
    assert d.workspace_bytes(1, 1, 1024, 4096, 14336, 8) >= 1024 * 14336 + 1024 * 4
    # the workspace query follows the same plan
    for mode, act, m, n, k in ((0, "fp16", 128, 4096, 4096), (1, "fp8", 512, 4096, 4096)):
        p = d.plan_info(mode, act, m, n, k)
        ws = d.workspace_bytes(mode, d._act_flag(act), m, n, k)
        assert (p["splits"] > 1) == (ws >= p["splits"] * m * n * 4 > 0), (m, n, k, p, ws)


def test_plan_info_rejects_bad_arguments(lib):
    info = (ctypes.c_int64 * 5)()
    assert lib.dps_plan_info(3, 0, 8, 64, 64, 1, 21, info) == 1
    assert lib.dps_plan_info(0, 0, 0, 64, 64, 1, 21, info) == 1
    assert lib.dps_plan_info(0, 0, 8, 64, 64, 1, 3, info) == 1
    assert lib.dps_plan_info(0, 0, 8, 64, 64, 1, 21, None) == 1


def test_grouped_grid_limit_uses_the_planned_token_tile(lib):
    """60000 experts of 10 rows each plan 32-token tiles: 18750 token tiles
    plus one per expert exceed the 65535 blocks of grid.y, so the call is
    refused on the host (it fitted the old 128-token estimate and would have
    failed at launch)."""
    experts, rows = 60000, 600000
    w = _weight(n=64, k=64, experts=experts, n_chunks=experts, log2=12,
                pool_bytes=experts << 12)
    st = lib.dps_linear_grouped(1, 0, 0x4000, 0x6000, rows, ctypes.byref(w), 0x5000, None, 0,
                                None)
    assert st == 3, st
    assert b"too many rows" in lib.dps_last_error()


def test_probe_library_exports_its_header():
    """libdps_probe.so (the ceiling probes the benchmark states fractions
    against) exports exactly what include/dps_probe.h declares, and rejects
    bad arguments on the host with nothing enqueued."""
    from paper_2609_34380_amd import probe

    text = open(os.path.join(ROOT, "include", "dps_probe.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    declared = set(re.findall(r"\b(dps_probe_[a-z0-9_]+)\s*\(", text))
    assert declared == set(probe.EXPORTED)
    if not os.path.exists(probe.LIB_PATH):
        import __graft_entry__
        __graft_entry__.build()
    plib = probe.load_library()
    for name in declared:
        assert hasattr(plib, name), name
    # NULL buffer, misaligned size, zero blocks: status 1
    assert plib.dps_probe_stream_read(None, 1024, 0, 0x1000, 4, None) == 1
    assert plib.dps_probe_stream_read(0x1000, 1000, 0, 0x2000, 4, None) == 1
    assert plib.dps_probe_stream_read(0x1000, 1024, 0, 0x2000, 0, None) == 1
    assert plib.dps_probe_mfma(0, 0, 4, 0x1000, None) == 1
    assert plib.dps_probe_mfma(1, 8, 0, 0x1000, None) == 1
    assert plib.dps_probe_mfma(0, 8, 4, None, None) == 1
    # window under 1 MiB or not whole 4 KiB rows, loader count not 4/8/16
    assert plib.dps_probe_lds_fill(0x1000, 1 << 19, 8, 4, 4, 0x2000, None) == 1
    assert plib.dps_probe_lds_fill(0x1000, (1 << 20) + 16, 8, 4, 4, 0x2000, None) == 1
    assert plib.dps_probe_lds_fill(0x1000, 1 << 20, 6, 4, 4, 0x2000, None) == 1
    assert plib.dps_probe_lds_fill(0x1000, 1 << 20, 8, 0, 4, 0x2000, None) == 1
    assert plib.dps_probe_mfma_lds(2, 0, 1, 8, 4, 0x1000, None) == 1     # no such shape
    assert plib.dps_probe_mfma_lds(0, 0, 1, 0, 4, 0x1000, None) == 1
    assert plib.dps_probe_mfma_lds(0, 0, 1, 8, 4, None, None) == 1


def test_dense_grid_limit_is_refused_on_the_host(lib):
    """A dense call whose GEMM grid would exceed 2^32 threads (here 2^30 - 16
    weight rows at 8192 tokens: 8.4 M tiles of 128 x 128 on 768-thread blocks)
    is refused before anything is enqueued."""
    n, k, rows = (1 << 30) - 16, 16, 8192
    w = _weight(n=n, k=k, n_chunks=1 << 20, log2=30, pool_bytes=1 << 30)
    st = lib.dps_linear(1, 0, 0x4000, rows, ctypes.byref(w), 0x5000, None, 0, None)
    assert st == 3, st
    assert b"too large for one grid" in lib.dps_last_error()


def test_vmm_rejects_bad_arguments_on_the_host(lib):
    """The shared-region calls check their arguments before any HIP call."""
    out = ctypes.c_void_p()
    assert lib.dps_vmm_create(0, 1 << 21, ctypes.byref(out)) == 1          # no units
    assert lib.dps_vmm_create(4, 3 << 20, ctypes.byref(out)) == 1          # not a power of two
    assert b"power of two" in lib.dps_vmm_last_error()
    assert lib.dps_vmm_create(4, 2048, ctypes.byref(out)) == 1             # under 4 KiB
    assert lib.dps_vmm_create(4, 1 << 21, None) == 1
    units = (ctypes.c_int32 * 2)(0, 1)
    assert lib.dps_vmm_map_residual(None, units, 2, ctypes.byref(out)) == 1
    assert lib.dps_vmm_remap(None, 0x1000, 0, 0) == 1
    assert lib.dps_vmm_unmap_residual(None, 0x1000) == 1
    assert lib.dps_vmm_kv_view(None) is None
    assert lib.dps_vmm_unit_bytes(None) == 0
    lib.dps_vmm_destroy(None)


def test_restore_worker_rejects_bad_arguments_on_the_host(lib):
    """Worker creation checks the manager, the targets and the sizes before it
    touches the device; the other calls refuse NULL."""
    sm = dps.SumManager(4, 8, 2)
    res = dps.CResidual(0x2000, 8 << 21, 0x3000, 8, 21)
    good = dps.CRestoreTarget(0x9000, 8 << 21, res)
    arr = (dps.CRestoreTarget * 2)(good, good)
    out = ctypes.c_void_p()
    create = lib.dps_restore_worker_create
    assert create(None, arr, 2, 8, 4 << 20, ctypes.byref(out)) == 1
    assert create(sm._h, None, 2, 8, 4 << 20, ctypes.byref(out)) == 1
    assert create(sm._h, arr, 0, 8, 4 << 20, ctypes.byref(out)) == 1
    assert create(sm._h, arr, 2, 4, 4 << 20, ctypes.byref(out)) == 1      # 8 chunks > 4 per unit
    assert create(sm._h, arr, 2, 8, 0, ctypes.byref(out)) == 1
    big = dps.CRestoreTarget(0x9000, (8 << 21) + 1, res)                   # beyond its chunks
    assert create(sm._h, (dps.CRestoreTarget * 1)(big), 1, 8, 4 << 20, ctypes.byref(out)) == 1
    assert b"target 0" in lib.dps_restore_worker_last_error()
    assert lib.dps_restore_worker_kick(None) == 1
    assert lib.dps_restore_worker_wait_idle(None, 10) == 1
    assert lib.dps_restore_worker_restored(None) == -1
    lib.dps_restore_worker_destroy(None)
    sm.close()
