"""dps_linear_static, the variant of dps_linear that allocates nothing: its
split-K partials and FP8 activation staging live in the library's static
device scratch.  Its outputs must equal dps_linear's (same plan, same
kernels) bit for bit and meet the oracle's tolerance, on consecutive calls
that share the scratch -- the second with a smaller input -- and inside a
captured HIP graph.  A call that needs more scratch than the static array
holds is refused on the host with DPS_ERR_WORKSPACE."""
import numpy as np
import pytest
import torch

import oracle
from gpu_helpers import DEV, Nested, assert_close, u16
from paper_2609_34380_amd import dps, workloads

pytestmark = pytest.mark.gpu

FAST, FULL = dps.MODE_FAST, dps.MODE_FULL


def _nested(n, k, seed, log2c=21):
    return Nested(workloads.weight_fp16(n, k, seed=seed), log2c)


def _check_against_oracle(y, x, nst, mode, act, rows):
    xr = x[torch.from_numpy(rows)]
    if act == "fp8":
        xq, s = oracle.act_quant(u16(xr))
        ref = oracle.linear_fp8(xq, s, nst.hi_ref)
    else:
        ref = oracle.linear_rows(oracle.FAST if mode == FAST else oracle.FULL, u16(xr),
                                 np.arange(len(rows)), nst.hi_ref,
                                 nst.res_ref if mode == FULL else None)
    assert_close(y[torch.from_numpy(rows).to(DEV)], ref)


# (n, k, m, mode, act): the first call of each pair needs more scratch than
# the second, so the second runs over the first one's leftovers
PAIRS = [
    ((6144, 4096, 128, FULL, "fp16"), (4096, 4096, 32, FULL, "fp16")),
    ((6144, 4096, 128, FAST, "fp16"), (6144, 4096, 17, FAST, "fp16")),
    ((4096, 14336, 256, FAST, "fp8"), (4096, 4096, 200, FAST, "fp8")),
    ((4096, 14336, 128, FULL, "fp16"), (4096, 14336, 33, FULL, "fp16")),
]


@pytest.mark.parametrize("first,second", PAIRS, ids=[str(i) for i in range(len(PAIRS))])
def test_static_matches_workspace_variant(first, second):
    calls = []
    for i, (n, k, m, mode, act) in enumerate((first, second)):
        flag = dps.ACT_FP8_ROWSCALE if act == "fp8" else dps.ACT_FP16
        need = dps.workspace_bytes(mode, flag, m, n, k)
        assert 0 < need <= dps.STATIC_SCRATCH_BYTES, need   # the call uses scratch
        nst = _nested(n, k, seed=40 + i)
        x = workloads.activations_fp16(m, k, seed=50 + i, outlier_frac=0.01 if act == "fp8"
                                       else 0.0)
        calls.append((nst, x, x.to(DEV), mode, act, need))
    assert calls[1][5] < calls[0][5]
    outs = []
    for nst, x, xd, mode, act, _ in calls:
        outs.append(dps.linear_static(xd, nst.nw, mode, act=act))
    torch.cuda.synchronize()
    for (nst, x, xd, mode, act, _), y in zip(calls, outs):
        want = dps.linear(xd, nst.nw, mode, act=act)
        torch.cuda.synchronize()
        assert torch.equal(y.view(torch.int16), want.view(torch.int16))
        m = x.shape[0]
        rows = np.unique(np.array([0, m // 3, m // 2, m - 1], dtype=np.int64))
        _check_against_oracle(y, x, nst, mode, act, rows)


def test_static_in_captured_graph():
    """The caller this variant is for: a captured pass with no workspace.
    Every replay (eager work and synchronizations between replays) equals the
    eager workspace variant."""
    n, k, m = 6144, 4096, 128
    nst = _nested(n, k, seed=60)
    x = workloads.activations_fp16(m, k, seed=61).to(DEV)
    y = torch.empty((m, n), dtype=torch.float16, device=DEV)
    want = {mode: dps.linear(x, nst.nw, mode) for mode in (FAST, FULL)}
    stream = torch.cuda.Stream()
    with torch.cuda.stream(stream):
        dps.linear_static(x, nst.nw, FULL, out=y)      # first call on the device: set-up
    stream.synchronize()
    graphs = {}
    for mode in (FAST, FULL):
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=stream):
            dps.linear_static(x, nst.nw, mode, out=y)
        graphs[mode] = g
    torch.cuda.synchronize()
    for it in range(4):
        mode = FAST if it % 2 == 0 else FULL
        y.fill_(0)
        torch.cuda.synchronize()
        with torch.cuda.stream(stream):
            graphs[mode].replay()
        torch.cuda.synchronize()
        assert torch.equal(y.view(torch.int16), want[mode].view(torch.int16)), (it, mode)


def test_static_refuses_calls_beyond_its_scratch():
    n, k, m = 4096, 14336, 8192
    need = dps.workspace_bytes(FAST, dps.ACT_FP8_ROWSCALE, m, n, k)
    assert need > dps.STATIC_SCRATCH_BYTES
    hi = torch.zeros((n, k), dtype=torch.uint8, device=DEV)
    nw = dps.NestedWeight(hi, None)
    x = torch.zeros((m, k), dtype=torch.float16, device=DEV)
    y = torch.full((m, n), 7.0, dtype=torch.float16, device=DEV)
    with pytest.raises(dps.DpsError) as ei:
        dps.linear_static(x, nw, FAST, act="fp8", out=y)
    assert ei.value.status == 4 and "static scratch" in str(ei.value)
    torch.cuda.synchronize()
    assert bool((y == 7.0).all())       # nothing was enqueued
