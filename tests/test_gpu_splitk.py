"""Split-K FP16 GEMM calls leave fp32 partials in the workspace, one plane
per K range, and a second launch sums them in K-range order and rounds to
FP16.  These tests read the partials a call left behind and redo that sum
on the host (float32 adds in the same order, then round-to-nearest-even to
FP16): Y must match it bit for bit, on dense and grouped calls of every FP16
tile family that splits K (the 32-token, 128-token and 256 x 256 tiles, N
not a multiple of 4), and on repeated calls over two workspaces."""
import numpy as np
import pytest
import torch

from gpu_helpers import DEV, Nested
from paper_2609_34380_amd import dps, workloads

pytestmark = pytest.mark.gpu

FAST, FULL = dps.MODE_FAST, dps.MODE_FULL


def _host_sum(ws, splits, rows, n):
    p = ws[:splits * rows * n * 4].view(torch.float32).view(splits, rows, n).cpu().numpy()
    acc = p[0].copy()
    for s in range(1, splits):
        acc = acc + p[s]
    return acc.astype(np.float16)


def _check(x, nst, mode, offsets=None, ws=None):
    rows = x.shape[0]
    experts = nst.nw.experts
    p = dps.plan_info(mode, "fp16", rows, nst.nw.n, nst.nw.k, experts=experts)
    assert p["kernel"] == "gemm_f16" and p["splits"] > 1, p
    need = dps.workspace_bytes(mode, 0, rows, nst.nw.n, nst.nw.k, experts)
    if ws is None:
        ws = torch.empty(need, dtype=torch.uint8, device=DEV)
    y = torch.full((rows, nst.nw.n), float("nan"), dtype=torch.float16, device=DEV)
    if offsets is None:
        dps.linear(x, nst.nw, mode, out=y, workspace=ws)
    else:
        dps.linear_grouped(x, offsets, nst.nw, mode, out=y, workspace=ws)
    torch.cuda.synchronize()
    ref = _host_sum(ws, p["splits"], rows, nst.nw.n)
    got = y.cpu().numpy()
    assert np.array_equal(got.view(np.uint16), ref.view(np.uint16)), p
    return y


@pytest.mark.parametrize("m,n,k,mode", [
    (64, 4096, 4096, FAST),      # 32-token tiles, K in 4 ranges
    (128, 4096, 4096, FULL),     # 32-token tiles
    (100, 1000, 6144, FULL),     # ragged weight and token tiles
    (256, 4096, 14336, FAST),    # 128-token tiles with DMA waves
    (96, 2050, 3008, FULL),      # N not a multiple of 4: scalar completion
    (2048, 4096, 14336, FULL),   # 256 x 256 tiles, two K ranges
])
def test_reduction_in_gemm_equals_partial_sum(m, n, k, mode):
    w = workloads.weight_fp16(n, k, seed=1201)
    x = workloads.activations_fp16(m, k, seed=1202).to(DEV)
    nst = Nested(w, 21)
    _check(x, nst, mode)


def test_grouped_reduction_in_gemm_equals_partial_sum():
    counts = (40, 0, 70, 3, 33)
    e, n, k = len(counts), 256, 6144
    w = workloads.weight_fp16(n, k, seed=1211, experts=e)
    x = workloads.activations_fp16(sum(counts), k, seed=1212).to(DEV)
    nst = Nested(w, 21)
    off = torch.tensor(np.concatenate([[0], np.cumsum(counts)]).astype(np.int32), device=DEV)
    for mode in (FAST, FULL):
        _check(x, nst, mode, offsets=off)


def test_repeated_calls_and_workspaces_agree():
    """A call repeated on the same workspace, and on a second one, fills
    every output (Y starts as NaN) with the same bits."""
    m, n, k = 64, 4096, 4096
    w = workloads.weight_fp16(n, k, seed=1221)
    x = workloads.activations_fp16(m, k, seed=1222).to(DEV)
    nst = Nested(w, 21)
    need = dps.workspace_bytes(FULL, 0, m, n, k)
    ws1 = torch.empty(need, dtype=torch.uint8, device=DEV)
    ws2 = torch.empty(need, dtype=torch.uint8, device=DEV)
    first = _check(x, nst, FULL, ws=ws1)
    for ws in (ws1, ws1, ws2, ws1):
        y = _check(x, nst, FULL, ws=ws)
        assert torch.equal(y.view(torch.int16), first.view(torch.int16))
