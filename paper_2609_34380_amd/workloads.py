"""Seeded synthetic inputs for the nested-precision linear layer.

This module only draws random inputs and describes shapes.  It holds none of
the method's arithmetic (no split, merge, addressing or product), so both the
HIP path and the CPU oracle can be fed from it without sharing any of the
computation under test.

The paper's models, weights and traces are not available; these stand in for
them with the shapes of a hidden-4096 / hidden-8192 transformer layer and the
value distributions of trained projection weights (N(0, 0.02)) and
activations (N(0, 1), optionally with a few outlier channels).
"""
from dataclasses import dataclass

import torch

# (name, N = output features, K = input features); Y[M][N] = X[M][K] . W[N][K]^T
H4096_SET = (("qkv", 6144, 4096), ("o", 4096, 4096),
             ("gate_up", 2 * 14336, 4096), ("down", 4096, 14336))
# QKV for hidden 8192 assumes 64 query + 8 key/value heads of 128.
H8192_SET = (("qkv", 10240, 8192), ("o", 8192, 8192),
             ("gate_up", 2 * 28672, 8192), ("down", 8192, 28672))
MOE_SHAPES = (("gate_up", 2 * 14336, 4096), ("down", 4096, 14336))

DECODE_M = (1, 8, 32, 128, 256)
PREFILL_M = (2048, 8192)


def _gen(seed, device):
    g = torch.Generator(device=device)
    g.manual_seed(int(seed))
    return g


def weight_fp16(n, k, seed, std=0.02, experts=None, device="cpu"):
    """FP16 weight [n][k] (or [experts][n][k]) drawn from N(0, std^2)."""
    shape = (n, k) if experts is None else (experts, n, k)
    w = torch.randn(shape, generator=_gen(seed, device), device=device, dtype=torch.float32)
    return (w * std).to(torch.float16)


def activations_fp16(m, k, seed, outlier_frac=0.0, outlier_scale=20.0, device="cpu"):
    """FP16 activations [m][k] ~ N(0, 1); round(outlier_frac * k) seeded
    channels (columns) are multiplied by outlier_scale."""
    g = _gen(seed, device)
    x = torch.randn((m, k), generator=g, device=device, dtype=torch.float32)
    n_out = int(round(outlier_frac * k))
    if n_out > 0:
        cols = torch.randperm(k, generator=g, device=device)[:n_out]
        x[:, cols] *= outlier_scale
    return x.to(torch.float16)


def n_chunks_for(numel, log2_chunk):
    c = 1 << log2_chunk
    return (numel + c - 1) // c


def chunk_slots(n_chunks, n_slots=None, seed=None):
    """int32 slot table.  seed None: identity (chunk c in slot c).  Otherwise
    n_chunks distinct slots drawn at random from n_slots."""
    if seed is None:
        return torch.arange(n_chunks, dtype=torch.int32)
    n_slots = n_chunks if n_slots is None else n_slots
    assert n_slots >= n_chunks
    perm = torch.randperm(n_slots, generator=_gen(seed, "cpu"))
    return perm[:n_chunks].to(torch.int32)


def kv_filler_pool(n_slots, log2_chunk, seed, device="cpu"):
    """A shared-region pool of n_slots chunks whose bytes are paged KV blocks
    (FP16 values ~ N(0, 1)); residual chunks are later written over some slots."""
    nbytes = n_slots << log2_chunk
    kv = torch.randn(nbytes // 2, generator=_gen(seed, device), device=device,
                     dtype=torch.float32).to(torch.float16)
    return kv.view(torch.uint8)


def kv_block_bytes(tokens=16, kv_heads=8, head_dim=128):
    """Bytes of one paged KV block: tokens x (K and V) x heads x dim x fp16."""
    return tokens * 2 * kv_heads * head_dim * 2


def moe_routing(tokens, experts, topk, seed):
    """Uniform random top-k routing without repeats.  Returns (token index of
    each routed row, sorted by expert; int64 offsets[experts + 1])."""
    g = _gen(seed, "cpu")
    choice = torch.stack([torch.randperm(experts, generator=g)[:topk] for _ in range(tokens)])
    expert_of_row = choice.reshape(-1)
    token_of_row = torch.arange(tokens).repeat_interleave(topk)
    order = torch.argsort(expert_of_row, stable=True)
    counts = torch.bincount(expert_of_row, minlength=experts)
    offsets = torch.zeros(experts + 1, dtype=torch.int64)
    offsets[1:] = torch.cumsum(counts, 0)
    return token_of_row[order], offsets


@dataclass
class WorkloadConfig:
    name: str
    description: str


CONFIGS = (
    WorkloadConfig("single_1024", "W 1024x1024 ~N(0,0.02), X 4x1024 ~N(0,1), 64 KiB chunks, "
                                  "identity table, fast and full"),
    WorkloadConfig("decode_h4096", "hidden-4096 layer set (QKV, O, gate+up, down), "
                                   "M in {1,8,32,128,256}, fast and full"),
    WorkloadConfig("prefill_h4096", "hidden-4096 layer set, M in {2048,8192}, 1% outlier "
                                    "channels x20; fast on FP8, full on FP16"),
    WorkloadConfig("moe_8x4096x14336", "8 experts, 512 tokens top-2, gate+up and down, "
                                       "fast and full"),
    WorkloadConfig("decode_h8192_scattered", "hidden-8192 set, M=64, 2 MiB residual chunks "
                                             "at random slots among KV blocks, modes alternate"),
)
