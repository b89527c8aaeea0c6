"""Full-size workloads on the GPU, in both nestings (E5M2 and E4M3).

The HIP path runs each workload at its real shape through the same entry
points and launch plans the benchmark times; the oracle computes whole output
rows (all N outputs of each checked row), plus the bit-exact planes of every
weight tensor.  Which rows are checked follows the call's launch plan
(dps_plan_info gives the token tile):
  - prefill (M in {2048, 8192}, 1% outlier channels x20; fast mode on FP8
    matrix cores with E4M3 activations, full mode on FP16 matrix cores):
    every row of the first and of the last token tile of each call;
  - decode (hidden-4096 set, M in {1, 8, 32, 128, 256}): every row up to
    32 tokens, else two seeded rows of every 16-row sub-tile of the first
    and the last token tile;
  - MoE (8 experts, hidden 4096, ffn 14336, 512 tokens routed top-2), both
    modes and fast mode with FP8 activations: one seeded row of every 16-row
    sub-tile of every expert's rows;
  - hidden-8192 decode set at M = 64 with residual chunks at random slots of
    a pool whose other slots hold 16-token FP16 KV blocks, modes alternating
    call to call.
"""
import numpy as np
import pytest
import torch

import oracle
from gpu_helpers import DEV, Nested, assert_close, u16
from paper_2609_34380_amd import dps, workloads

pytestmark = [pytest.mark.gpu, pytest.mark.timeout(900)]

FAST, FULL = dps.MODE_FAST, dps.MODE_FULL
ENCS = (dps.ENC_E5M2, dps.ENC_E4M3)
ENC_IDS = ("e5m2", "e4m3")
LOG2C = 21


def _omode(mode):
    return oracle.FAST if mode == FAST else oracle.FULL


def _tile_ends(m, tile):
    """Every row of the first and of the last token tile."""
    last0 = (m - 1) // tile * tile
    return np.unique(np.concatenate([np.arange(min(tile, m)), np.arange(last0, m)]))


def _subtile_rows(m, tile, seed, per=2):
    """All rows up to 32 tokens; else `per` seeded rows of every 16-row
    sub-tile of the first and the last token tile."""
    if m <= 32:
        return np.arange(m)
    rng = np.random.default_rng(seed)
    rows = set()
    for r0 in _tile_ends(m, tile)[::16]:
        r1 = min(r0 + 16, m)
        rows.update(int(v) for v in rng.choice(np.arange(r0, r1), size=min(per, r1 - r0),
                                               replace=False))
    return np.array(sorted(rows), dtype=np.int64)


def _ref_rows(mode, act, x_rows, nst):
    """Oracle outputs for the given activation rows (a torch FP16 tensor)."""
    if act == "fp8":
        xq, s = oracle.act_quant(u16(x_rows))
        return oracle.linear_fp8(xq, s, nst.hi_ref, enc=nst.enc)
    return oracle.linear_rows(_omode(mode), u16(x_rows), np.arange(x_rows.shape[0]), nst.hi_ref,
                              nst.res_ref if mode == FULL else None, enc=nst.enc)


@pytest.fixture(scope="module", params=ENCS, ids=ENC_IDS)
def h4096_set(request):
    enc = request.param
    out = []
    for li, (name, n, k) in enumerate(workloads.H4096_SET):
        w = workloads.weight_fp16(n, k, seed=500 + li)
        nst = Nested(w, LOG2C, enc=enc)
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
            tile = dps.plan_info(mode, "fp16", m, n, k)["tile_tokens"]
            rows = _subtile_rows(m, tile, seed=m + n)
            got_rows.append(y[torch.from_numpy(rows).to(DEV)].cpu())
            xs_rows.append(x[torch.from_numpy(rows)])
        ref = _ref_rows(mode, "fp16", torch.cat(xs_rows), nst)
        assert_close(torch.cat(got_rows), ref, name)


@pytest.mark.parametrize("m", workloads.PREFILL_M)
@pytest.mark.parametrize("mode", [FAST, FULL], ids=["fast_fp8", "full_f16"])
def test_prefill_h4096(h4096_set, m, mode):
    act = "fp8" if mode == FAST else "fp16"
    for name, n, k, nst in h4096_set:
        x = workloads.activations_fp16(m, k, seed=700 + m + k, outlier_frac=0.01,
                                       outlier_scale=20.0)
        y = dps.linear(x.to(DEV), nst.nw, mode, act=act)
        tile = dps.plan_info(mode, act, m, n, k)["tile_tokens"]
        rows = _tile_ends(m, tile)
        got = y[torch.from_numpy(rows).to(DEV)].cpu()
        del y
        assert_close(got, _ref_rows(mode, act, x[torch.from_numpy(rows)], nst),
                     "%s m=%d tile=%d" % (name, m, tile))


@pytest.mark.parametrize("m", [512, 1024, 3072, 4096])
@pytest.mark.parametrize("mode", [FAST, FULL], ids=["fast_fp8", "full_f16"])
def test_prefill_h4096_tile_rule_sizes(h4096_set, m, mode):
    """Token counts where the planner's tile and split rules change branch:
    FP8 256 x 256 tiles with exactly one block per CU (down and O at 4096
    tokens) and 256 x 128 tiles with a nearly empty last round of big tiles
    (QKV at 3072), FP8 calls without a K split (512, 1024), and the O layer
    on 128-token FP16 tiles from 512 tokens on."""
    act = "fp8" if mode == FAST else "fp16"
    for name, n, k, nst in h4096_set:
        x = workloads.activations_fp16(m, k, seed=730 + m + k, outlier_frac=0.01,
                                       outlier_scale=20.0)
        y = dps.linear(x.to(DEV), nst.nw, mode, act=act)
        tile = dps.plan_info(mode, act, m, n, k)["tile_tokens"]
        rows = _subtile_rows(m, tile, seed=m * 5 + n, per=1)
        got = y[torch.from_numpy(rows).to(DEV)].cpu()
        assert_close(got, _ref_rows(mode, act, x[torch.from_numpy(rows)], nst),
                     "%s m=%d" % (name, m))


def test_prefill_fp8_quantization_full_size():
    """The E4M3 row quantization at the prefill size, bit-exact on every row."""
    x = workloads.activations_fp16(2048, 14336, seed=710, outlier_frac=0.01, outlier_scale=20.0)
    xq, s = dps.quant_rows_e4m3(x.to(DEV))
    torch.cuda.synchronize()
    xq_ref, s_ref = oracle.act_quant(u16(x))
    assert np.array_equal(s.cpu().numpy().astype(np.float64), s_ref)
    assert np.array_equal(xq.cpu().numpy(), xq_ref)


@pytest.fixture(scope="module", params=ENCS, ids=ENC_IDS)
def moe(request):
    enc = request.param
    experts, tokens, topk = 8, 512, 2
    token_of_row, offsets = workloads.moe_routing(tokens, experts, topk, seed=801)
    layers = []
    for li, (name, n, k) in enumerate(workloads.MOE_SHAPES):
        w = workloads.weight_fp16(n, k, seed=810 + li, experts=experts)
        nst = Nested(w, LOG2C, enc=enc)
        nst.check_planes()
        del w
        x_tok = workloads.activations_fp16(tokens, k, seed=820 + li)
        layers.append((name, n, k, nst, x_tok[token_of_row].contiguous()))
    return offsets, layers


@pytest.mark.parametrize("mode", [FAST, FULL], ids=["fast", "full"])
def test_moe_grouped(moe, mode):
    offsets, layers = moe
    off_dev = torch.from_numpy(offsets.numpy().astype(np.int32)).to(DEV)
    experts = len(offsets) - 1
    rng = np.random.default_rng(830 + mode)
    for name, n, k, nst, xs in layers:
        y = dps.linear_grouped(xs.to(DEV), off_dev, nst.nw, mode)
        torch.cuda.synchronize()
        per_expert = n * k
        assert per_expert % (1 << LOG2C) == 0
        chunks = per_expert >> LOG2C
        for e in range(experts):
            r0, r1 = int(offsets[e]), int(offsets[e + 1])
            rows = np.array([int(rng.integers(s0, min(s0 + 16, r1))) for s0 in range(r0, r1, 16)],
                            dtype=np.int64)
            res_e = oracle.Residual(nst.res_ref.pool, nst.res_ref.slots[e * chunks:(e + 1) * chunks],
                                    LOG2C)
            ref = oracle.linear_rows(_omode(mode), u16(xs), rows, nst.hi_ref[e],
                                     res_e if mode == FULL else None, enc=nst.enc)
            assert_close(y[torch.from_numpy(rows).to(DEV)], ref, "%s expert %d" % (name, e))


def test_moe_grouped_fp8(moe):
    """The MoE layers in fast mode with FP8 activations: every routed row
    quantized on its own, each expert's rows on the FP8 matrix cores."""
    offsets, layers = moe
    off_dev = torch.from_numpy(offsets.numpy().astype(np.int32)).to(DEV)
    experts = len(offsets) - 1
    rng = np.random.default_rng(840)
    for name, n, k, nst, xs in layers:
        y = dps.linear_grouped(xs.to(DEV), off_dev, nst.nw, FAST, act="fp8")
        torch.cuda.synchronize()
        xq, sc = oracle.act_quant(u16(xs))
        for e in range(experts):
            r0, r1 = int(offsets[e]), int(offsets[e + 1])
            rows = np.array([int(rng.integers(s0, min(s0 + 16, r1))) for s0 in range(r0, r1, 16)],
                            dtype=np.int64)
            ref = oracle.linear_fp8(xq[rows], sc[rows], nst.hi_ref[e], enc=nst.enc)
            assert_close(y[torch.from_numpy(rows).to(DEV)], ref, "%s expert %d" % (name, e))


@pytest.mark.parametrize("enc", ENCS, ids=ENC_IDS)
def test_h8192_scattered_alternating_modes(enc):
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
        hi_ref = oracle.split(u16(w).reshape(n, k), res_ref, enc=enc)
        res = dps.Residual(pool_dev, torch.from_numpy(slots).to(DEV), LOG2C)
        nw = dps.split(w.to(DEV), res, enc=enc)
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
            tile = dps.plan_info(mode, "fp16", m, n, k)["tile_tokens"]
            rows = _subtile_rows(m, tile, seed=step * 11 + n, per=1)
            ref = oracle.linear_rows(_omode(mode), u16(x), rows, hi_ref,
                                     res_ref if mode == FULL else None, enc=enc)
            assert_close(y[torch.from_numpy(rows).to(DEV)], ref, "%s step %d" % (name, step))
