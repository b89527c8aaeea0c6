"""Shared helpers for the GPU parity tests.

Inputs always come from paper_2609_34380_amd.workloads (seeded, CPU).  The
oracle splits the same FP16 weights itself; nothing it consumes is produced
by the HIP path.
"""
import numpy as np
import torch

import oracle
from paper_2609_34380_amd import dps, workloads

# acceptance bounds for linear outputs: relative Frobenius error and per-element max abs
REL_FRO = 1e-3
MAX_ABS = 2e-2

DEV = torch.device("cuda:0")


def u16(t):
    return t.contiguous().numpy().view(np.uint16)


def make_residual_host(numel, log2c, n_slots=None, slot_seed=None, filler_seed=None):
    """(pool uint8 numpy, slots int32 numpy) before any split."""
    c = 1 << log2c
    n_chunks = max(1, -(-numel // c))
    n_slots = n_chunks if n_slots is None else n_slots
    slots = workloads.chunk_slots(n_chunks, n_slots, slot_seed).numpy()
    if filler_seed is None:
        pool = np.zeros(n_slots * c, dtype=np.uint8)
    else:
        pool = workloads.kv_filler_pool(n_slots, log2c, filler_seed).numpy().copy()
    return pool, slots


class Nested:
    """One weight tensor split on both sides: GPU (dps) and oracle (CPU)."""

    def __init__(self, w_fp16, log2c, n_slots=None, slot_seed=None, filler_seed=None,
                 enc=dps.ENC_E5M2):
        numel = w_fp16.numel()
        pool, slots = make_residual_host(numel, log2c, n_slots, slot_seed, filler_seed)
        self.enc = enc
        self.res_ref = oracle.Residual(pool.copy(), slots, log2c)
        self.hi_ref = oracle.split(u16(w_fp16).reshape(w_fp16.shape), self.res_ref, enc=enc)
        self.res = dps.Residual(torch.from_numpy(pool).to(DEV), torch.from_numpy(slots).to(DEV),
                                log2c)
        self.nw = dps.split(w_fp16.to(DEV), self.res, enc=enc)
        self.shape = tuple(w_fp16.shape)

    def check_planes(self):
        torch.cuda.synchronize()
        assert np.array_equal(self.nw.hi.cpu().numpy(), self.hi_ref), "hi plane differs"
        assert np.array_equal(self.res.pool.cpu().numpy(), self.res_ref.pool), "pool differs"


def errors(y_gpu, y_ref):
    got = y_gpu.detach().cpu().to(torch.float64).numpy()
    ref = np.asarray(y_ref, dtype=np.float64)
    assert got.shape == ref.shape, (got.shape, ref.shape)
    diff = got - ref
    nref = np.linalg.norm(ref)
    rel = np.linalg.norm(diff) / nref if nref > 0 else np.linalg.norm(diff)
    return rel, float(np.abs(diff).max()) if diff.size else 0.0


def assert_close(y_gpu, y_ref, what=""):
    rel, mx = errors(y_gpu, y_ref)
    assert np.isfinite(rel) and rel <= REL_FRO and mx <= MAX_ABS, \
        "%s rel_fro=%.3e max_abs=%.3e" % (what, rel, mx)
    return rel, mx
