"""The shared region through the HIP virtual memory API (dps_vmm_*): physical
units mapped into the KV view and, per residual tensor, into a contiguous
residual view (paper Sec. IV-B "Shared Region", dual-mapping property).

A weight is split with its residual written through a view of scattered
units: the view holds the oracle's residual bytes, the KV view shows the
same bytes at those units, and full mode through the view's identity table
matches the oracle.  Then a unit is taken for KV blocks (written through the
KV view): the residual goes stale exactly there; the piece is remapped to a
free unit and restored from the host backup through the view, and full mode
gives its earlier bits again while the KV blocks stay intact."""
import numpy as np
import pytest
import torch

import oracle
from gpu_helpers import DEV, assert_close, u16
from paper_2609_34380_amd import dps, workloads

pytestmark = pytest.mark.gpu

FULL = dps.MODE_FULL


def _unit_bytes():
    g = dps.vmm_granularity()
    u = 1 << 21
    while u % g:
        u <<= 1
    return u


@pytest.fixture
def region():
    U = _unit_bytes()
    r = dps.VmmRegion(16, U, device=DEV)
    yield r
    torch.cuda.synchronize()
    r.close()


def test_kv_view_spans_the_units(region):
    U = region.unit_bytes
    assert region.kv.numel() == 16 * U and region.kv.is_cuda
    for u in range(16):
        region.kv[u * U:(u + 1) * U].fill_(u + 1)
    torch.cuda.synchronize()
    view = region.map_residual([3, 3, 15, 0])
    got = view.view(4, U)[:, :4096].cpu().numpy()
    assert np.array_equal(got[:, 0], np.array([4, 4, 16, 1], dtype=np.uint8))
    assert (got == got[:, :1]).all()
    del view


@pytest.mark.parametrize("enc", [dps.ENC_E5M2, dps.ENC_E4M3], ids=["e5m2", "e4m3"])
def test_residual_view_split_linear_evict_restore(region, enc):
    U = region.unit_bytes
    k = 2048
    n = 5 * U // (2 * k)                   # 2.5 units of weights: the last unit partial
    numel = n * k
    units = [5, 2, 9]
    assert -(-numel // U) == len(units)
    w = workloads.weight_fp16(n, k, seed=1301)
    view = region.map_residual(units)
    res = region.residual(view)
    nw = dps.split(w.to(DEV), res, enc=enc)
    torch.cuda.synchronize()

    # the view holds the oracle's residual stream; the KV view shows it at the units
    pool_ref = np.zeros(len(units) * U, dtype=np.uint8)
    res_ref = oracle.Residual(pool_ref, np.arange(len(units), dtype=np.int32),
                              region.log2_unit)
    hi_ref = oracle.split(u16(w), res_ref, enc=enc)
    assert np.array_equal(nw.hi.cpu().numpy(), hi_ref)
    assert np.array_equal(view[:numel].cpu().numpy(), pool_ref[:numel])
    for i, u in enumerate(units):
        assert torch.equal(region.kv[u * U:(u + 1) * U], view[i * U:(i + 1) * U]), (i, u)

    x = workloads.activations_fp16(64, k, seed=1302).to(DEV)
    y0 = dps.linear(x, nw, FULL)
    torch.cuda.synchronize()
    assert_close(y0, oracle.linear(oracle.FULL, u16(x.cpu()), hi_ref, res_ref, enc=enc))

    # back the residual up, then hand unit 2 (piece 1) to KV blocks
    bk = dps.backup(res, numel)
    torch.cuda.synchronize()
    region.kv[2 * U:3 * U].fill_(0x77)
    torch.cuda.synchronize()
    assert bool((view[U:2 * U] == 0x77).all())     # the residual is stale exactly there
    y_stale = dps.linear(x, nw, FULL)
    torch.cuda.synchronize()
    assert not torch.equal(y_stale.view(torch.int16), y0.view(torch.int16))

    # restore chunk 1 into free unit 11: remap the piece, copy the backup through the view
    region.remap(view, 1, 11)
    dps.restore(bk, res, numel=numel, chunk_begin=1, chunk_end=2)
    torch.cuda.synchronize()
    assert torch.equal(region.kv[11 * U:12 * U], view[U:2 * U])
    assert bool((region.kv[2 * U:3 * U] == 0x77).all())   # the KV blocks are intact
    assert np.array_equal(view[:numel].cpu().numpy(), pool_ref[:numel])
    y1 = dps.linear(x, nw, FULL)
    torch.cuda.synchronize()
    assert torch.equal(y1.view(torch.int16), y0.view(torch.int16))
    del nw, res
    region.unmap(view)
    del view


def test_bad_unit_index_is_refused(region):
    with pytest.raises(dps.DpsError):
        region.map_residual([0, 16])
    view = region.map_residual([1])
    with pytest.raises(dps.DpsError):
        region.remap(view, 1, 0)          # piece outside the view
    with pytest.raises(dps.DpsError):
        region.remap(view, 0, -1)
    region.unmap(view)
    with pytest.raises(dps.DpsError):
        region.unmap(view)                # already unmapped
