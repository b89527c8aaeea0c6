"""Full-size workloads on the GPU, checked on sampled outputs.

The HIP path runs each workload at its real shape through the same entry
points and launch plans the benchmark times; the oracle computes a few
seeded output rows of each call one by one (all N outputs of each sampled
row), plus the bit-exact planes of every weight tensor.
  - hidden-4096 decode layer set, M in {1, 8, 32, 128, 256}, fast and full;
  - the same set as prefill, M in {2048, 8192}, 1% outlier channels x20,
    fast mode on FP8 matrix cores, full mode on FP16 matrix cores;
  - MoE: 8 experts, hidden 4096, ffn 14336, 512 tokens routed top-2;
  - hidden-8192 decode set, M = 64, residual in 2 MiB chunks at random slots
    of a pool whose other slots hold 16-token FP16 KV blocks, modes
    alternating call to call.
"""
import numpy as np
import pytest
import torch

import oracle
from gpu_helpers import DEV, Nested, assert_close, u16
from paper_2609_34380_amd import dps, workloads

pytestmark = [pytest.mark.gpu, pytest.mark.timeout(900)]

FAST, FULL = dps.MODE_FAST, dps.MODE_FULL
LOG2C = 21


def _sample_rows(m, seed, count=3):
    rng = np.random.default_rng(seed)
    rows = {0, m - 1}
    while len(rows) < min(count, m):
        rows.add(int(rng.integers(m)))
    return np.array(sorted(rows), dtype=np.int64)


@pytest.fixture(scope="module")
def h4096_set():
    out = []
    for li, (name, n, k) in enumerate(workloads.H4096_SET):
        w = workloads.weight_fp16(n, k, seed=500 + li)
        nst = Nested(w, LOG2C)
        nst.check_planes()
        del w
        out.append((name, n, k, nst))
    return out


@pytest.mark.parametrize("mode", [FAST, FULL], ids=["fast", "full"])
def test_decode_h4096(h4096_set, mode):
    for name, n, k, nst in h4096_set:
        xs_rows = []
        got_rows = []
        for m in workloads.DECODE_M:
            x = workloads.activations_fp16(m, k, seed=600 + m)
            y = dps.linear(x.to(DEV), nst.nw, mode)
            rows = _sample_rows(m, seed=m + n)
            got_rows.append(y[torch.from_numpy(rows).to(DEV)].cpu())
            xs_rows.append(x[torch.from_numpy(rows)])
        xs = torch.cat(xs_rows)
        ref = oracle.linear_rows(oracle.FAST if mode == FAST else oracle.FULL, u16(xs),
                                 np.arange(xs.shape[0]), nst.hi_ref,
                                 nst.res_ref if mode == FULL else None)
        assert_close(torch.cat(got_rows), ref, name)


@pytest.mark.parametrize("m", workloads.PREFILL_M)
@pytest.mark.parametrize("mode", [FAST, FULL], ids=["fast_fp8", "full_f16"])
def test_prefill_h4096(h4096_set, m, mode):
    for name, n, k, nst in h4096_set:
        x = workloads.activations_fp16(m, k, seed=700 + m + k, outlier_frac=0.01,
                                       outlier_scale=20.0)
        act = "fp8" if mode == FAST else "fp16"
        y = dps.linear(x.to(DEV), nst.nw, mode, act=act)
        rows = _sample_rows(m, seed=m * 3 + n)
        got = y[torch.from_numpy(rows).to(DEV)].cpu()
        xr = x[torch.from_numpy(rows)]
        if mode == FAST:
            xq, s = oracle.act_quant(u16(xr))
            ref = oracle.linear_fp8(xq, s, nst.hi_ref)
        else:
            ref = oracle.linear_rows(oracle.FULL, u16(xr), np.arange(len(rows)), nst.hi_ref,
                                     nst.res_ref)
        assert_close(got, ref, "%s m=%d" % (name, m))


@pytest.mark.parametrize("m", [512, 1024, 3072, 4096])
@pytest.mark.parametrize("mode", [FAST, FULL], ids=["fast_fp8", "full_f16"])
def test_prefill_h4096_tile_rule_sizes(h4096_set, m, mode):
    """Token counts where the planner's tile and split rules change branch:
    FP8 256 x 256 tiles with exactly one block per CU (down and O at 4096
    tokens) and 256 x 128 tiles with a nearly empty last round of big tiles
    (QKV at 3072), FP8 calls without a K split (512, 1024), and the O layer
    on 128-token FP16 tiles from 512 tokens on."""
    for name, n, k, nst in h4096_set:
        x = workloads.activations_fp16(m, k, seed=730 + m + k, outlier_frac=0.01,
                                       outlier_scale=20.0)
        act = "fp8" if mode == FAST else "fp16"
        y = dps.linear(x.to(DEV), nst.nw, mode, act=act)
        rows = _sample_rows(m, seed=m * 5 + n)
        got = y[torch.from_numpy(rows).to(DEV)].cpu()
        xr = x[torch.from_numpy(rows)]
        if mode == FAST:
            xq, s = oracle.act_quant(u16(xr))
            ref = oracle.linear_fp8(xq, s, nst.hi_ref)
        else:
            ref = oracle.linear_rows(oracle.FULL, u16(xr), np.arange(len(rows)), nst.hi_ref,
                                     nst.res_ref)
        assert_close(got, ref, "%s m=%d" % (name, m))


def test_prefill_fp8_quantization_full_size():
    """The E4M3 row quantization at the prefill size, bit-exact on every row."""
    x = workloads.activations_fp16(2048, 14336, seed=710, outlier_frac=0.01, outlier_scale=20.0)
    xq, s = dps.quant_rows_e4m3(x.to(DEV))
    torch.cuda.synchronize()
    xq_ref, s_ref = oracle.act_quant(u16(x))
    assert np.array_equal(s.cpu().numpy().astype(np.float64), s_ref)
    assert np.array_equal(xq.cpu().numpy(), xq_ref)


@pytest.fixture(scope="module")
def moe():
    experts, tokens, topk = 8, 512, 2
    token_of_row, offsets = workloads.moe_routing(tokens, experts, topk, seed=801)
    layers = []
    for li, (name, n, k) in enumerate(workloads.MOE_SHAPES):
        w = workloads.weight_fp16(n, k, seed=810 + li, experts=experts)
        nst = Nested(w, LOG2C)
        nst.check_planes()
        del w
        x_tok = workloads.activations_fp16(tokens, k, seed=820 + li)
        layers.append((name, n, k, nst, x_tok[token_of_row].contiguous()))
    return offsets, layers


@pytest.mark.parametrize("mode", [FAST, FULL], ids=["fast", "full"])
def test_moe_grouped(moe, mode):
    offsets, layers = moe
    off_dev = torch.from_numpy(offsets.numpy().astype(np.int32)).to(DEV)
    for name, n, k, nst, xs in layers:
        y = dps.linear_grouped(xs.to(DEV), off_dev, nst.nw, mode)
        torch.cuda.synchronize()
        per_expert = n * k
        assert per_expert % (1 << LOG2C) == 0
        chunks = per_expert >> LOG2C
        for e in (0, 3, 7):
            r0, r1 = int(offsets[e]), int(offsets[e + 1])
            rows = np.unique(np.array([r0, (r0 + r1) // 2, r1 - 1]))
            hi_e = nst.hi_ref[e]
            res_e = oracle.Residual(nst.res_ref.pool, nst.res_ref.slots[e * chunks:(e + 1) * chunks],
                                    LOG2C)
            ref = oracle.linear_rows(oracle.FAST if mode == FAST else oracle.FULL,
                                     u16(xs), rows, hi_e, res_e if mode == FULL else None)
            assert_close(y[torch.from_numpy(rows).to(DEV)], ref, "%s expert %d" % (name, e))


def test_h8192_scattered_alternating_modes():
    """Residual chunks of the hidden-8192 set at random slots of a 1024-slot
    (2 GiB) pool; every other slot holds KV blocks.  Calls alternate fast and
    full mode over the whole set, twice."""
    n_slots = 1024
    pool_np = workloads.kv_filler_pool(n_slots, LOG2C, seed=901).numpy().copy()
    kv_before = pool_np.copy()
    # place each tensor's chunks at distinct random slots
    perm = torch.randperm(n_slots, generator=torch.Generator().manual_seed(902)).numpy()
    cursor = 0
    pool_dev = torch.from_numpy(pool_np).to(DEV)
    used = []
    tensors = []
    m = 64
    for li, (name, n, k) in enumerate(workloads.H8192_SET):
        numel = n * k
        n_chunks = -(-numel // (1 << LOG2C))
        slots = perm[cursor:cursor + n_chunks].astype(np.int32)
        cursor += n_chunks
        used.extend(slots.tolist())
        w = workloads.weight_fp16(n, k, seed=910 + li)
        res_ref = oracle.Residual(pool_np, slots, LOG2C)     # shared host pool
        hi_ref = oracle.split(u16(w).reshape(n, k), res_ref)
        res = dps.Residual(pool_dev, torch.from_numpy(slots).to(DEV), LOG2C)
        nw = dps.split(w.to(DEV), res)
        del w
        tensors.append((name, n, k, nw, hi_ref, res_ref))
    torch.cuda.synchronize()
    got_pool = pool_dev.cpu().numpy()
    assert np.array_equal(got_pool, pool_np)
    free = np.setdiff1d(np.arange(n_slots), np.array(used))
    c = 1 << LOG2C
    assert np.array_equal(got_pool.reshape(n_slots, c)[free], kv_before.reshape(n_slots, c)[free])
    for name, n, k, nw, hi_ref, _ in tensors:
        assert np.array_equal(nw.hi.cpu().numpy(), hi_ref)

    for step in range(4):
        mode = FAST if step % 2 == 0 else FULL
        for name, n, k, nw, hi_ref, res_ref in tensors:
            x = workloads.activations_fp16(m, k, seed=920 + step)
            y = dps.linear(x.to(DEV), nw, mode)
            rows = _sample_rows(m, seed=step * 11 + n, count=2)
            ref = oracle.linear_rows(oracle.FAST if mode == FAST else oracle.FULL, u16(x), rows,
                                     hi_ref, res_ref if mode == FULL else None)
            assert_close(y[torch.from_numpy(rows).to(DEV)], ref, "%s step %d" % (name, step))
