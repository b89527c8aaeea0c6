"""Graph pair per batch size (Sec. IV-C, "Granularity of the precision
switch"): every replay of a captured fast or full decode pass is
bit-identical to the same pass run eagerly, with eager work and
synchronizations between replays and the mode switching from pass to pass
as a SUM manager dictates."""
import pytest
import torch

from gpu_helpers import DEV
from paper_2609_34380_amd import dps, graphs, workloads

pytestmark = pytest.mark.gpu

LAYERS = (("qkv", 6144, 4096), ("o", 4096, 4096), ("down", 4096, 14336))
BATCHES = (1, 8, 32, 128)
MODES = graphs.ModeGraphs.MODES


def test_graph_pair_replays_match_eager():
    nws = []
    for li, (name, n, k) in enumerate(LAYERS):
        res = dps.make_residual(n * k, 21, DEV)
        nws.append(dps.split(workloads.weight_fp16(n, k, seed=90 + li).to(DEV), res))
    xs = {(m, k): workloads.activations_fp16(m, k, seed=m + k).to(DEV)
          for m in BATCHES for _, _, k in LAYERS}
    ys = {(m, mode, li): torch.empty((m, n), dtype=torch.float16, device=DEV)
          for m in BATCHES for mode in MODES for li, (_, n, _) in enumerate(LAYERS)}
    need = max(dps.workspace_bytes(mode, 0, m, n, k) for m in BATCHES
               for mode in MODES for _, n, k in LAYERS)
    ws = torch.empty(max(need, 256), dtype=torch.uint8, device=DEV)

    def step(m, mode):
        for li, (name, n, k) in enumerate(LAYERS):
            dps.linear(xs[(m, k)], nws[li], mode, out=ys[(m, mode, li)], workspace=ws)

    # eager references
    want = {}
    for m in BATCHES:
        for mode in MODES:
            step(m, mode)
            torch.cuda.synchronize()
            for li in range(len(LAYERS)):
                want[(m, mode, li)] = ys[(m, mode, li)].clone()

    mg = graphs.ModeGraphs(step, BATCHES).capture()
    sum_mgr = dps.SumManager(4, 8, 2)
    held = []
    for it in range(12):
        # the serving loop: KV pressure comes and goes, the mode follows
        if it % 4 == 1:
            held += sum_mgr.alloc(20)        # evicts a residual -> fast
        if it % 4 == 3:
            sum_mgr.free(held)
            held = []
            while (step_r := sum_mgr.restore_begin()) is not None:
                sum_mgr.restore_done(step_r[0])
        mode = sum_mgr.mode
        for m in BATCHES:
            for li in range(len(LAYERS)):
                ys[(m, mode, li)].fill_(0)   # eager work between replays
            mg.replay(m, mode)
            torch.cuda.synchronize()
            for li in range(len(LAYERS)):
                got = ys[(m, mode, li)]
                assert torch.equal(got.view(torch.int16), want[(m, mode, li)].view(torch.int16)), \
                    (it, m, mode, li)
    with pytest.raises(KeyError):
        mg.replay(3, dps.MODE_FAST)
