"""Graph pair per batch size (Sec. IV-C, "Granularity of the precision
switch"): every replay of a captured fast or full decode pass is
bit-identical to the same pass run eagerly and within tolerance of the CPU
oracle (every row up to 32 tokens, two seeded rows of every 16-row sub-tile
beyond), with eager work and synchronizations between replays and the mode
switching from pass to pass as a SUM manager dictates."""
import numpy as np
import pytest
import torch

import oracle
from gpu_helpers import DEV, Nested, assert_close, u16
from paper_2609_34380_amd import dps, graphs, workloads

pytestmark = pytest.mark.gpu

LAYERS = (("qkv", 6144, 4096), ("o", 4096, 4096), ("down", 4096, 14336))
BATCHES = (1, 8, 32, 128)
MODES = graphs.ModeGraphs.MODES


def test_graph_pair_replays_match_eager():
    nsts = [Nested(workloads.weight_fp16(n, k, seed=90 + li), 21)
            for li, (name, n, k) in enumerate(LAYERS)]
    nws = [nst.nw for nst in nsts]
    xs_host = {(m, k): workloads.activations_fp16(m, k, seed=m + k)
               for m in BATCHES for _, _, k in LAYERS}
    xs = {key: x.to(DEV) for key, x in xs_host.items()}
    ys = {(m, mode, li): torch.empty((m, n), dtype=torch.float16, device=DEV)
          for m in BATCHES for mode in MODES for li, (_, n, _) in enumerate(LAYERS)}
    need = max(dps.workspace_bytes(mode, 0, m, n, k) for m in BATCHES
               for mode in MODES for _, n, k in LAYERS)
    ws = torch.empty(max(need, 256), dtype=torch.uint8, device=DEV)

    def step(m, mode):
        for li, (name, n, k) in enumerate(LAYERS):
            dps.linear(xs[(m, k)], nws[li], mode, out=ys[(m, mode, li)], workspace=ws)

    # eager references, and the oracle on the checked rows
    want = {}
    ref = {}
    rng = np.random.default_rng(91)
    for m in BATCHES:
        rows = np.arange(m) if m <= 32 else np.sort(np.concatenate(
            [rng.choice(np.arange(r0, r0 + 16), 2, replace=False) for r0 in range(0, m, 16)]))
        for mode in MODES:
            step(m, mode)
            torch.cuda.synchronize()
            for li, (name, n, k) in enumerate(LAYERS):
                want[(m, mode, li)] = ys[(m, mode, li)].clone()
                ref[(m, mode, li)] = (rows, oracle.linear_rows(
                    oracle.FAST if mode == dps.MODE_FAST else oracle.FULL,
                    u16(xs_host[(m, k)]), rows, nsts[li].hi_ref,
                    nsts[li].res_ref if mode == dps.MODE_FULL else None))

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
            torch.cuda.synchronize()
            mg.replay(m, mode)
            torch.cuda.synchronize()
            for li in range(len(LAYERS)):
                got = ys[(m, mode, li)]
                assert torch.equal(got.view(torch.int16), want[(m, mode, li)].view(torch.int16)), \
                    (it, m, mode, li)
                rows, yref = ref[(m, mode, li)]
                assert_close(got[torch.from_numpy(rows).to(DEV)], yref,
                             "replay %d m=%d mode=%d layer %d" % (it, m, mode, li))
    with pytest.raises(KeyError):
        mg.replay(3, dps.MODE_FAST)
