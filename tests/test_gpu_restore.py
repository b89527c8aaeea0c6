"""Residual backup and restore (Sec. IV-B "Residual Backup"; Sec. IV-C,
restoration paragraph) against the CPU oracle, bit for bit.

The backup is checked against the oracle's read of the same residual
stream; restores of chunk ranges into pools overwritten with KV-like filler
are checked byte for byte over the whole pool (restored chunks and every
untouched byte).  The decode scenario evicts part of a layer's residual,
keeps serving it in fast mode while the restore runs on its own stream, and
then requires the full-mode output to be bit-identical to the one before
the eviction.
"""
import numpy as np
import pytest
import torch

import oracle
from gpu_helpers import DEV, Nested
from paper_2609_34380_amd import dps, workloads

pytestmark = pytest.mark.gpu

FAST, FULL = dps.MODE_FAST, dps.MODE_FULL


@pytest.mark.parametrize("numel,log2c,n_slots,copy", [
    (1_000_003, 12, 400, 4 << 20),      # scattered 4 KiB chunks: one copy per chunk
    (1_000_003, 12, None, 64 << 10),    # identity table: chunks joined, cut into 64 KiB copies
    (8192 * 8192, 21, 64, 4 << 20),     # 2 MiB chunks among KV slots, the paper's 4 MiB copies
    (8192 * 8192, 21, 64, 1 << 20),     # copies smaller than a chunk
    (17, 4, 8, 4 << 20),                # ragged last chunk
])
def test_backup_restore_roundtrip(numel, log2c, n_slots, copy):
    w = workloads.weight_fp16(1, numel, seed=numel % 1000).reshape(-1)
    scattered = n_slots is not None
    nst = Nested(w, log2c, n_slots=n_slots, slot_seed=5 if scattered else None,
                 filler_seed=6 if scattered else None)
    bk = dps.backup(nst.res, numel, copy_bytes=copy)
    torch.cuda.synchronize()
    assert bk.is_pinned()
    bk_ref = oracle.backup(nst.res_ref, numel)
    assert np.array_equal(bk.numpy()[:numel], bk_ref)

    # evict: every pool slot now holds KV-like filler
    n_pool = nst.res.pool.numel() >> log2c
    filler = workloads.kv_filler_pool(n_pool, log2c, seed=7).numpy().copy()
    nst.res.pool.copy_(torch.from_numpy(filler).to(DEV))
    ref = oracle.Residual(filler.copy(), nst.res_ref.slots, log2c)
    used = -(-numel // (1 << log2c))
    for c0, c1 in ((used // 3, used // 2), (0, used // 3), (used // 2, used)):
        dps.restore(bk, nst.res, chunk_begin=c0, chunk_end=c1, copy_bytes=copy)
        oracle.restore(bk_ref, ref, c0, c1)
        torch.cuda.synchronize()
        assert np.array_equal(nst.res.pool.cpu().numpy(), ref.pool), (c0, c1)


def test_restore_from_pageable_memory():
    """A backup in ordinary (pageable) host memory restores the same bytes."""
    numel, log2c = 300_000, 12
    w = workloads.weight_fp16(1, numel, seed=8).reshape(-1)
    nst = Nested(w, log2c, n_slots=200, slot_seed=9, filler_seed=10)
    bk = torch.empty(numel, dtype=torch.uint8)
    dps.backup(nst.res, numel, out=bk)
    torch.cuda.synchronize()
    assert np.array_equal(bk.numpy(), oracle.backup(nst.res_ref, numel))
    want = nst.res.pool.cpu().numpy()
    nst.res.pool.fill_(0x5A)
    dps.restore(bk, nst.res)
    torch.cuda.synchronize()
    slots = nst.res_ref.slots
    c = 1 << log2c
    got = nst.res.pool.cpu().numpy().reshape(-1, c)
    assert np.array_equal(got[slots].reshape(-1)[:numel], want.reshape(-1, c)[slots]
                          .reshape(-1)[:numel])


@pytest.mark.parametrize("enc", [dps.ENC_E5M2, dps.ENC_E4M3], ids=["e5m2", "e4m3"])
def test_evict_serve_fast_restore_full(enc):
    """Hidden-8192 O layer, 2 MiB chunks at random slots among KV blocks, 64
    tokens.  Half the residual chunks are overwritten by KV data; fast mode
    keeps its output bit for bit; the restore runs on a copy stream while fast
    passes run on the compute stream; after the compute stream waits for the
    restore, full mode is bit-identical to the pass before the eviction."""
    n = k = 8192
    log2c = 21
    w = workloads.weight_fp16(n, k, seed=11)
    n_chunks = -(-n * k // (1 << log2c))
    nst = Nested(w, log2c, n_slots=2 * n_chunks, slot_seed=12, filler_seed=13, enc=enc)
    x = workloads.activations_fp16(64, k, seed=14).to(DEV)
    compute = torch.cuda.current_stream()
    copy = torch.cuda.Stream()
    y_full = dps.linear(x, nst.nw, FULL)
    y_fast = dps.linear(x, nst.nw, FAST)
    bk = dps.backup(nst.res, n * k)
    torch.cuda.synchronize()

    evicted = np.arange(0, n_chunks, 2)
    kv = workloads.kv_filler_pool(1, log2c, seed=15).to(DEV)
    for c in evicted:
        s = int(nst.res_ref.slots[c])
        nst.res.pool[s << log2c:(s + 1) << log2c].copy_(kv)
    y_full_bad = dps.linear(x, nst.nw, FULL)
    torch.cuda.synchronize()
    assert not torch.equal(y_full_bad.view(torch.int16), y_full.view(torch.int16))

    copy.wait_stream(compute)
    with torch.cuda.stream(copy):
        for c in evicted:
            dps.restore(bk, nst.res, chunk_begin=int(c), chunk_end=int(c) + 1)
        done = torch.cuda.Event()
        done.record(copy)
    fast_outs = [dps.linear(x, nst.nw, FAST) for _ in range(8)]
    compute.wait_event(done)
    y_full_back = dps.linear(x, nst.nw, FULL)
    torch.cuda.synchronize()
    for y in fast_outs:
        assert torch.equal(y.view(torch.int16), y_fast.view(torch.int16))
    assert torch.equal(y_full_back.view(torch.int16), y_full.view(torch.int16))


def test_sum_managed_eviction_and_restore():
    """Three 4096x4096 layers whose residuals (8 chunks of 2 MiB) each fill one
    16 MiB unit of a 6-unit shared pool that KV blocks of 64 KiB also use.
    The native SUM manager hands out KV blocks (their bytes are then written
    with KV data) until two residuals are evicted; fast mode keeps every
    output bit for bit.  Freeing the blocks wakes the restore: each evicted
    residual is bound to a free unit (possibly not its old one), its device
    slot table is rewritten and its bytes copied back from the pinned backup
    on a copy stream.  Full mode is then bit-identical to the start."""
    n = k = 4096
    log2c = 21
    chunks_per_unit = 8
    unit_bytes = chunks_per_unit << log2c
    kv_bytes = 64 << 10
    n_units, n_res = 6, 3
    sum_mgr = dps.SumManager(n_units, unit_bytes // kv_bytes, n_res)
    pool = torch.zeros(n_units * unit_bytes, dtype=torch.uint8, device=DEV)
    x = workloads.activations_fp16(64, k, seed=20).to(DEV)
    layers, y_full, y_fast, backups = [], [], [], []
    for r in range(n_res):
        slots = sum_mgr.slots(r, chunks_per_unit, chunks_per_unit)
        res = dps.Residual(pool, slots.to(DEV), log2c)
        nw = dps.split(workloads.weight_fp16(n, k, seed=21 + r).to(DEV), res)
        layers.append(nw)
        y_full.append(dps.linear(x, nw, FULL))
        y_fast.append(dps.linear(x, nw, FAST))
        backups.append(dps.backup(res, n * k, slots_host=slots))
    torch.cuda.synchronize()

    gen = torch.Generator(device=DEV)
    gen.manual_seed(22)
    held = []
    while sum_mgr.counts()["evicted"] < 2:
        blocks = sum_mgr.alloc(100)
        for b in blocks:          # the serving system writes KV into the new blocks
            pool[b * kv_bytes:(b + 1) * kv_bytes] = torch.randint(
                0, 256, (kv_bytes,), dtype=torch.uint8, device=DEV, generator=gen)
        held += blocks
    assert sum_mgr.mode == dps.MODE_FAST
    for nw, want in zip(layers, y_fast):
        assert torch.equal(dps.linear(x, nw, FAST).view(torch.int16), want.view(torch.int16))

    # unit 0 (the first evicted) keeps its KV blocks, so both residuals move
    bpu = unit_bytes // kv_bytes
    assert sum_mgr.free([b for b in held if b // bpu != 0])
    compute = torch.cuda.current_stream()
    copy = torch.cuda.Stream()
    copy.wait_stream(compute)
    moved = []
    while True:
        step = sum_mgr.restore_begin()
        if step is None:
            break
        r, u = step
        slots = sum_mgr.slots(r, chunks_per_unit, chunks_per_unit)
        moved.append((r, u))
        with torch.cuda.stream(copy):
            layers[r].residual.slots.copy_(slots, non_blocking=True)
            dps.restore(backups[r], layers[r].residual, slots_host=slots)
        copy.synchronize()
        sum_mgr.restore_done(r)
    assert moved == [(0, 1), (1, 3)] and sum_mgr.mode == dps.MODE_FULL
    compute.wait_stream(copy)
    for nw, want in zip(layers, y_full):
        assert torch.equal(dps.linear(x, nw, FULL).view(torch.int16), want.view(torch.int16))


def test_restore_worker_thread_restores_evicted_residuals():
    """The same eviction as above, restored by the native restore worker: a
    host thread that, once kicked, rewrites each evicted residual's device
    chunk table to the unit the manager gives it and copies the backup in on
    its own stream, while fast-mode passes keep running on the compute
    stream with unchanged bits.  When it is idle the mode is full and full
    mode gives its first bits again."""
    n = k = 4096
    log2c = 21
    chunks_per_unit = 8
    unit_bytes = chunks_per_unit << log2c
    kv_bytes = 64 << 10
    n_units, n_res = 6, 3
    sum_mgr = dps.SumManager(n_units, unit_bytes // kv_bytes, n_res)
    pool = torch.zeros(n_units * unit_bytes, dtype=torch.uint8, device=DEV)
    x = workloads.activations_fp16(64, k, seed=30).to(DEV)
    layers, y_full, y_fast, backups = [], [], [], []
    for r in range(n_res):
        slots = sum_mgr.slots(r, chunks_per_unit, chunks_per_unit)
        res = dps.Residual(pool, slots.to(DEV), log2c)
        nw = dps.split(workloads.weight_fp16(n, k, seed=31 + r).to(DEV), res)
        layers.append(nw)
        y_full.append(dps.linear(x, nw, FULL))
        y_fast.append(dps.linear(x, nw, FAST))
        backups.append(dps.backup(res, n * k, slots_host=slots))
    torch.cuda.synchronize()
    worker = dps.RestoreWorker(sum_mgr, [(backups[r], n * k, layers[r].residual)
                                         for r in range(n_res)], chunks_per_unit)

    gen = torch.Generator(device=DEV)
    gen.manual_seed(32)
    held = []
    while sum_mgr.counts()["evicted"] < 2:
        blocks = sum_mgr.alloc(100)
        for b in blocks:
            pool[b * kv_bytes:(b + 1) * kv_bytes] = torch.randint(
                0, 256, (kv_bytes,), dtype=torch.uint8, device=DEV, generator=gen)
        held += blocks
    torch.cuda.synchronize()
    assert sum_mgr.mode == dps.MODE_FAST
    worker.kick()                      # nothing to restore yet: no unit is free
    worker.wait_idle(10000)
    assert worker.restored == 0 and sum_mgr.mode == dps.MODE_FAST

    bpu = unit_bytes // kv_bytes
    assert sum_mgr.free([b for b in held if b // bpu != 0])
    worker.kick()
    passes = 0
    while sum_mgr.mode == dps.MODE_FAST and passes < 2000:   # fast passes meanwhile
        for nw, want in zip(layers, y_fast):
            assert torch.equal(dps.linear(x, nw, FAST).view(torch.int16), want.view(torch.int16))
        passes += 1
    worker.wait_idle(60000)
    assert worker.restored == 2 and sum_mgr.mode == dps.MODE_FULL
    assert [sum_mgr.unit_of(r) for r in range(n_res)] == [1, 3, 2]
    for nw, want in zip(layers, y_full):
        assert torch.equal(dps.linear(x, nw, FULL).view(torch.int16), want.view(torch.int16))
    worker.close()
