"""The FP8 prefill GEMM on its 256 x 256 tile, in both nestings (E5M2 and
E4M3 upper bytes against E4M3 activations; Sec. IV-B "Persistent Region",
Sec. IV-C "Dual-mode serving").

The tile runs four token-waves of 64 rows, each over four 16-row MFMA
sub-tiles, and two weight-waves of 128 rows.  Every row of the first and of
the last token tile is compared, all N outputs of each, so every token-wave,
sub-tile and weight-wave of two tiles meets the oracle; the ragged case cuts
both the last token tile and the last weight tile short.  The planner's
choice of the tile is asserted through dps_plan_info."""
import numpy as np
import pytest
import torch

import oracle
from gpu_helpers import DEV, Nested, assert_close, u16
from paper_2609_34380_amd import dps, workloads

pytestmark = [pytest.mark.gpu, pytest.mark.timeout(600)]

ENCS = (dps.ENC_E5M2, dps.ENC_E4M3)


@pytest.mark.parametrize("enc", ENCS, ids=("e5m2", "e4m3"))
@pytest.mark.parametrize("m,n,k", [(4096, 4096, 1024), (4000, 4000, 1024), (4096, 4096, 4096)])
def test_fp8_256x256_tile_every_wave(enc, m, n, k):
    plan = dps.plan_info(dps.MODE_FAST, "fp8", m, n, k)
    assert (plan["kernel"], plan["tile_rows"], plan["tile_tokens"]) == ("gemm_fp8", 256, 256)
    nst = Nested(workloads.weight_fp16(n, k, seed=k + n + 3), 21, enc=enc)
    x = workloads.activations_fp16(m, k, seed=m + k + enc, outlier_frac=0.01,
                                   outlier_scale=20.0)
    y = dps.linear(x.to(DEV), nst.nw, dps.MODE_FAST, act="fp8")
    last0 = (m - 1) // 256 * 256
    rows = np.concatenate([np.arange(256), np.arange(last0, m)])
    got = y[torch.from_numpy(rows).to(DEV)].cpu()
    xq, s = oracle.act_quant(u16(x[torch.from_numpy(rows)]))
    ref = oracle.linear_fp8(xq, s, nst.hi_ref, enc=enc)
    for wave in range(4):     # report per token-wave of the tile
        sel = np.nonzero((rows % 256) // 64 == wave)[0]
        assert_close(got[sel], ref[sel], "token-wave %d" % wave)
