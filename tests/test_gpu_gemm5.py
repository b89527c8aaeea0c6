"""The 256 x 256 FP16 GEMM (eight waves of 128 x 64 wave tiles, 64-element
stages) in both modes and both nestings against the oracle (Sec. IV-C
"Overall concept": full mode rebuilds FP16 during the product, fast mode
uses the upper byte alone; Sec. IV-B "Persistent Region" for the nestings).

The planner takes this tile for dense calls of at least 512 tokens whose
tiles fill the chip, or fill it with two K ranges when K reaches 8192
(asserted through dps_plan_info).  The shapes cut the last weight tile, the
last token tile and the last K stage short, split K in two, and read the
residual through two-chunk row ranges (chunks at least as long as a K range)
as well as through per-vector table lookups (chunks shorter than a range),
over pools whose other slots hold KV-cache filler.  Every row of the first
and of the last token tile is compared (all eight waves of two tiles, each
wave's four 16-token sub-tiles), all N outputs of each."""
import numpy as np
import pytest
import torch

import oracle
from gpu_helpers import DEV, Nested, assert_close, u16
from paper_2609_34380_amd import dps, workloads

pytestmark = [pytest.mark.gpu, pytest.mark.timeout(600)]

FAST, FULL = dps.MODE_FAST, dps.MODE_FULL
E5M2, E4M3 = dps.ENC_E5M2, dps.ENC_E4M3

# (m, n, k, log2c, enc, splits)
CASES = [
    (2000, 8200, 1040, 10, E5M2, 1),   # 33 x 8 tiles (264 blocks), a 16-element K tail,
    (2000, 8200, 1040, 21, E4M3, 1),   # last token tile 208 rows, last weight tile 8 rows;
                                       # 1 KiB chunks shorter than the K range: table lookups
    (1800, 3856, 8208, 12, E5M2, 2),   # 16 x 8 tiles, K in two ranges of 4160 over 4 KiB
    (1800, 3856, 8208, 16, E4M3, 2),   # chunks (lookups) and 64 KiB chunks (two-chunk ranges);
                                       # last token tile 8 rows, last weight tile 16 rows
]


def _id(c):
    return "m%d_n%d_k%d_c%d_%s" % (c[0], c[1], c[2], c[3], "e4m3" if c[4] == E4M3 else "e5m2")


@pytest.fixture(scope="module", params=CASES, ids=_id)
def case(request):
    m, n, k, log2c, enc, splits = request.param
    w = workloads.weight_fp16(n, k, seed=300 + n + k)
    x = workloads.activations_fp16(m, k, seed=400 + m)
    n_chunks = -(-n * k // (1 << log2c))
    nst = Nested(w, log2c, n_slots=2 * n_chunks + 5, slot_seed=n + 3 * k, filler_seed=m, enc=enc)
    return m, n, k, log2c, enc, splits, x, nst


def _rows(m):
    last0 = (m - 1) // 256 * 256
    return np.concatenate([np.arange(256), np.arange(last0, m)])


def test_planner_picks_the_256x256_tile(case):
    m, n, k, log2c, enc, splits, x, nst = case
    for mode in (FAST, FULL):
        plan = dps.plan_info(mode, "fp16", m, n, k, log2_chunk=log2c)
        assert (plan["kernel"], plan["tile_rows"], plan["tile_tokens"], plan["splits"]) == \
            ("gemm_f16", 256, 256, splits)


@pytest.mark.parametrize("mode", [FAST, FULL], ids=["fast", "full"])
def test_gemm5_matches_oracle(case, mode):
    m, n, k, log2c, enc, splits, x, nst = case
    y = dps.linear(x.to(DEV), nst.nw, mode)
    torch.cuda.synchronize()
    rows = _rows(m)
    got = y[torch.from_numpy(rows).to(DEV)].cpu()
    ref = oracle.linear_rows(oracle.FAST if mode == FAST else oracle.FULL, u16(x), rows,
                             nst.hi_ref, nst.res_ref if mode == FULL else None, enc=enc)
    # per wave of the tile (64 tokens) and 16-token sub-tile, so that a wrong
    # wave or sub-tile shows by name
    for wave in range(4):
        for sub in range(4):
            sel = np.nonzero(((rows % 256) // 64 == wave) & ((rows % 64) // 16 == sub))[0]
            if sel.size:
                assert_close(got[sel], ref[sel], "mode=%d wave %d sub-tile %d" % (mode, wave, sub))
    assert_close(got, ref, "mode=%d" % mode)


def test_gemm5_fast_equals_full_with_zero_residual(case):
    m, n, k, log2c, enc, splits, x, nst = case
    zero_res = dps.Residual(torch.zeros_like(nst.res.pool), nst.res.slots, nst.res.log2_chunk)
    nw0 = dps.NestedWeight(nst.nw.hi, zero_res, enc=enc)
    xd = x.to(DEV)
    y_fast = dps.linear(xd, nst.nw, FAST)
    y_full0 = dps.linear(xd, nw0, FULL)
    torch.cuda.synchronize()
    assert torch.equal(y_fast.view(torch.int16), y_full0.view(torch.int16))
