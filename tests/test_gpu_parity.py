"""HIP path vs the CPU oracle, element by element, on seeded inputs.

Bit-exact: split planes, merge, chunk addressing, E4M3 row quantization.
Tolerance (relative Frobenius <= 1e-3 and max abs <= 2e-2 against the fp64
oracle): every linear output.  Sizes span several tiles with ragged tails
on N, K and M, both residual addressing paths (a row's K range within one or
two chunks, and per-vector table lookups when chunks are small), scattered
slot tables and pools whose other slots hold KV-like filler.
"""
import numpy as np
import pytest
import torch

import oracle
from gpu_helpers import DEV, Nested, assert_close, errors, make_residual_host, u16
from paper_2609_34380_amd import dps, workloads

pytestmark = pytest.mark.gpu

FAST, FULL = dps.MODE_FAST, dps.MODE_FULL


def _omode(mode):
    return oracle.FAST if mode == FAST else oracle.FULL


# -----------------------------------------------------------------------------
# split / merge / addressing: bit-exact
# -----------------------------------------------------------------------------

def test_split_merge_single_layer_identity_table():
    """1024x1024 FP16, 64 KiB chunks, identity table (the single-layer workload)."""
    w = workloads.weight_fp16(1024, 1024, seed=0)
    nst = Nested(w, 16)
    nst.check_planes()
    back = dps.merge(nst.nw)
    torch.cuda.synchronize()
    assert torch.equal(back.cpu().view(torch.int16), w.view(torch.int16))


def test_split_merge_all_patterns_scattered():
    """All 65536 FP16 patterns plus a ragged tail of 13 words, 256-byte chunks at
    random slots of a pool whose other slots hold KV filler."""
    rng = np.random.default_rng(3)
    bits = np.concatenate([np.arange(65536, dtype=np.uint32).astype(np.uint16),
                           rng.integers(0, 65536, 13).astype(np.uint16)])
    w = torch.from_numpy(bits.view(np.int16).copy()).view(torch.float16)
    nst = Nested(w, 8, n_slots=600, slot_seed=4, filler_seed=5)
    nst.check_planes()
    back = dps.merge(nst.nw)
    torch.cuda.synchronize()
    assert np.array_equal(back.cpu().view(torch.int16).numpy().view(np.uint16), bits)


@pytest.mark.parametrize("numel,log2c,n_slots", [(1_000_003, 12, 400), (4096 * 14336, 21, 64),
                                                  (17, 4, 8)])
def test_split_scattered_pool(numel, log2c, n_slots):
    rng = np.random.default_rng(numel)
    bits = rng.integers(0, 65536, numel).astype(np.uint16)
    w = torch.from_numpy(bits.view(np.int16)).view(torch.float16)
    nst = Nested(w, log2c, n_slots=n_slots, slot_seed=7, filler_seed=8)
    nst.check_planes()
    back = dps.merge(nst.nw)
    torch.cuda.synchronize()
    assert np.array_equal(back.cpu().view(torch.int16).numpy().view(np.uint16), bits)


@pytest.mark.parametrize("i", range(12))
def test_split_merge_select_random(i):
    """Seeded random sizes (1 to 3 M words), chunks of 16 B to 4 MiB, identity
    or scattered tables over KV filler, random bit patterns or weights of
    small or wide range: the encoding choice, both planes and the merge
    bit-exact against the oracle (merge after split the identity for E5M2)."""
    rng = np.random.default_rng(30000 + i)
    numel = int(rng.integers(1, 3_000_000)) if i % 4 else int(rng.integers(1, 4000))
    log2c = int(rng.integers(4, 23))
    scattered = bool(rng.integers(0, 2))
    kind = i % 3
    if kind == 0:
        bits = rng.integers(0, 65536, numel).astype(np.uint16)
    else:
        bits = rng.normal(0, 0.02 if kind == 1 else 0.5, numel).astype(np.float16).view(np.uint16)
    want_e4m3 = bool(rng.integers(0, 2))
    n_chunks = max(1, -(-numel // (1 << log2c)))
    pool, slots = make_residual_host(numel, log2c, 2 * n_chunks + 3 if scattered else n_chunks,
                                     slot_seed=i if scattered else None,
                                     filler_seed=i + 1 if scattered else None)
    wd = torch.from_numpy(bits.view(np.float16).copy()).to(DEV)
    e_ref = oracle.select_enc(bits)
    assert int(dps.select_enc(wd).cpu()[0]) == e_ref
    enc = dps.ENC_E4M3 if (want_e4m3 and e_ref == oracle.E4M3) else dps.ENC_E5M2
    oenc = oracle.E4M3 if enc == dps.ENC_E4M3 else oracle.E5M2
    res_ref = oracle.Residual(pool.copy(), slots, log2c)
    hi_ref = oracle.split(bits, res_ref, enc=oenc)
    res = dps.Residual(torch.from_numpy(pool.copy()).to(DEV), torch.from_numpy(slots).to(DEV),
                       log2c)
    nw = dps.split(wd, res, enc=enc)
    back = dps.merge(nw)
    torch.cuda.synchronize()
    assert np.array_equal(nw.hi.cpu().numpy(), hi_ref)
    assert np.array_equal(res.pool.cpu().numpy(), res_ref.pool)
    merged = u16(back.cpu())
    assert np.array_equal(merged, oracle.merge(hi_ref, res_ref, enc=oenc).reshape(-1))
    if enc == dps.ENC_E5M2:
        assert np.array_equal(merged, bits)


def test_out_of_range_slot_is_never_dereferenced():
    """A slot entry outside the pool: the split drops those residual bytes, the
    merge reads them as zero, and nothing else changes."""
    log2c = 8
    numel = 4 * 256
    bits = np.random.default_rng(9).integers(0, 65536, numel).astype(np.uint16)
    w = torch.from_numpy(bits.view(np.int16)).view(torch.float16).to(DEV)
    pool = torch.full((4 * 256,), 0xA5, dtype=torch.uint8, device=DEV)
    slots = torch.tensor([2, 1000, 0, -5], dtype=torch.int32, device=DEV)
    res = dps.Residual(pool, slots, log2c)
    nw = dps.split(w, res)
    back = dps.merge(nw)
    torch.cuda.synchronize()
    p = pool.cpu().numpy().reshape(4, 256)
    low = bits.view(np.uint8)[0::2].reshape(4, 256)
    assert np.array_equal(p[2], low[0]) and np.array_equal(p[0], low[2])
    assert (p[1] == 0xA5).all() and (p[3] == 0xA5).all()
    want = bits.copy().reshape(4, 256)
    want[1] &= 0xFF00
    want[3] &= 0xFF00
    assert np.array_equal(back.cpu().view(torch.int16).numpy().view(np.uint16), want.ravel())


# -----------------------------------------------------------------------------
# FP8 row quantization: bit-exact
# -----------------------------------------------------------------------------

def test_quant_rows_bit_exact():
    x = workloads.activations_fp16(37, 4096, seed=11, outlier_frac=0.01, outlier_scale=20.0)
    x[0] = 0.0
    x[1] = torch.linspace(-65504, 65504, 4096).half()
    x[2] = (torch.randn(4096) * 1e-6).half()
    x[3, :] = 0.0
    x[3, 5] = 448.0
    x[3, 6] = 0.0146484375    # a tie between E4M3 neighbours at scale 1
    x[3, 7] = -0.0
    xq, s = dps.quant_rows_e4m3(x.to(DEV))
    torch.cuda.synchronize()
    xq_ref, s_ref = oracle.act_quant(u16(x))
    assert np.array_equal(s.cpu().numpy().astype(np.float64), s_ref)
    assert np.array_equal(xq.cpu().numpy(), xq_ref)


@pytest.mark.parametrize("k", [1024, 8192, 16384, 0])
def test_quant_rows_every_fp16_value(k):
    """Every finite FP16 value with |x| <= 448, at scale 1: in rows of k
    elements (each row ends with 448, so its scale is 1; rows of up to 16384
    elements take the wave-per-row kernel), or all in one row (k = 0, the
    block-per-row kernel)."""
    bits = np.arange(65536, dtype=np.uint32).astype(np.uint16)
    v = bits.view(np.float16).astype(np.float64)
    keep = bits[np.isfinite(v) & (np.abs(v) <= 448)]
    if k == 0:
        pad = (-keep.size) % 16
        mat = np.concatenate([keep, np.zeros(pad, np.uint16)]).reshape(1, -1)
    else:
        per = k - 1
        rows = -(-keep.size // per)
        body = np.concatenate([keep, np.zeros(rows * per - keep.size, np.uint16)])
        top = np.full((rows, 1), np.float16(448.0).view(np.uint16), np.uint16)
        mat = np.concatenate([body.reshape(rows, per), top], axis=1)
    x = torch.from_numpy(mat.view(np.int16).copy()).view(torch.float16)
    xq, s = dps.quant_rows_e4m3(x.to(DEV))
    torch.cuda.synchronize()
    xq_ref, s_ref = oracle.act_quant(mat)
    assert np.all(s_ref == 1.0) and np.all(s.cpu().numpy() == 1.0)
    assert np.array_equal(xq.cpu().numpy(), xq_ref)


# -----------------------------------------------------------------------------
# linear: tolerance against the fp64 oracle
# -----------------------------------------------------------------------------

# (m, n, k, log2c, scattered): decode-shaped (skinny kernel) and token-tiled
# (matrix-core GEMM) problems with ragged m, n and k.
LINEAR_CASES = [
    (4, 1024, 1024, 16, False),     # the single-layer workload
    (1, 1024, 1024, 16, False),
    (3, 1000, 1040, 12, True),
    (2, 8200, 2064, 10, True),      # 1-2 token kernel: two rows per wave, ragged K chunk,
                                    # residual rows over several chunks (table lookups)
    (4, 1024, 8192, 21, False),     # activations exactly fill the 64 KiB staging limit
    (2, 300, 14336, 16, True),      # long rows (the down projection's K)
    (16, 64, 2048, 8, True),        # chunks smaller than a K range: table lookups
    (17, 520, 4096, 21, True),
    (32, 768, 2048, 14, True),      # one full 32-token tile
    (33, 200, 1152, 10, True),
    (64, 1024, 4096, 21, False),
    (65, 384, 1024, 12, True),
    (130, 260, 2048, 8, True),
    (300, 512, 512, 16, True),
    (256, 640, 4096, 21, True),
    # layers above 2^24 weights take the 64- and 128-token tiles
    (65, 4100, 4112, 21, True),
    (130, 4100, 4112, 12, True),
    # dense kernel for up to 16 tokens (whole K per block, 16-row groups):
    # ragged row groups and K chunks, 1 KiB residual chunks that row pieces
    # straddle, chunks below 1 KiB (per-vector lookups), 1-8 groups per block
    (3, 8200, 4112, 10, True),       # 3 groups per block
    (5, 4100, 2064, 9, True),        # 2 groups, chunks of 512 bytes
    (8, 28672, 1024, 21, False),     # 7 groups (the gate+up rows at 8 tokens)
    (12, 6144, 4096, 21, True),      # 2 groups (the QKV rows)
    (16, 33000, 1040, 12, True),     # 8 groups, 258 blocks, 16-element K tail
    (9, 4096, 4096, 21, True),       # 1 group (the O rows)
    (1, 64, 33024, 12, True),        # one token whose activations exceed 64 KiB
    (7, 5, 2048, 12, True),          # fewer rows than one group
    (16, 17, 1024, 10, False),       # one row past a group
    (13, 4112, 4096, 21, True),      # 257 groups: two per block, the last block half empty
    (32, 4096, 4096, 21, True),      # 32 tokens: the wide-row GEMM's 32-token tile
]


def _case_id(c):
    return "m%d_n%d_k%d_c%d%s" % (c[0], c[1], c[2], c[3], "_scat" if c[4] else "")


@pytest.fixture(scope="module", params=LINEAR_CASES, ids=_case_id)
def linear_case(request):
    m, n, k, log2c, scattered = request.param
    w = workloads.weight_fp16(n, k, seed=100 + n)
    x = workloads.activations_fp16(m, k, seed=200 + m)
    numel = n * k
    n_chunks = -(-numel // (1 << log2c))
    if scattered:
        nst = Nested(w, log2c, n_slots=2 * n_chunks + 3, slot_seed=n + k, filler_seed=m)
    else:
        nst = Nested(w, log2c)
    return m, n, k, w, x, nst


def test_linear_planes(linear_case):
    linear_case[-1].check_planes()


@pytest.mark.parametrize("mode", [FAST, FULL], ids=["fast", "full"])
def test_linear_matches_oracle(linear_case, mode):
    m, n, k, w, x, nst = linear_case
    y = dps.linear(x.to(DEV), nst.nw, mode)
    torch.cuda.synchronize()
    ref = oracle.linear(_omode(mode), u16(x), nst.hi_ref,
                        nst.res_ref if mode == FULL else None)
    assert_close(y, ref, "mode=%d" % mode)


def test_fast_equals_full_with_zero_residual(linear_case):
    """Fast mode == full mode whose residual bytes are all zero, bit for bit."""
    m, n, k, w, x, nst = linear_case
    zero_res = dps.Residual(torch.zeros_like(nst.res.pool), nst.res.slots, nst.res.log2_chunk)
    nw0 = dps.NestedWeight(nst.nw.hi, zero_res)
    xd = x.to(DEV)
    y_fast = dps.linear(xd, nst.nw, FAST)
    y_full0 = dps.linear(xd, nw0, FULL)
    torch.cuda.synchronize()
    assert torch.equal(y_fast.view(torch.int16), y_full0.view(torch.int16))


def test_fast_never_reads_residual(linear_case):
    """Fast mode with the pool overwritten (0xFF), and with no residual at
    all, gives the same bits as with the intact residual."""
    m, n, k, w, x, nst = linear_case
    xd = x.to(DEV)
    y_clean = dps.linear(xd, nst.nw, FAST)
    poisoned = dps.Residual(torch.full_like(nst.res.pool, 0xFF), nst.res.slots,
                            nst.res.log2_chunk)
    y_poison = dps.linear(xd, dps.NestedWeight(nst.nw.hi, poisoned), FAST)
    y_none = dps.linear(xd, dps.NestedWeight(nst.nw.hi, None), FAST)
    torch.cuda.synchronize()
    assert torch.equal(y_clean.view(torch.int16), y_poison.view(torch.int16))
    assert torch.equal(y_clean.view(torch.int16), y_none.view(torch.int16))


def test_linear_is_deterministic(linear_case):
    m, n, k, w, x, nst = linear_case
    xd = x.to(DEV)
    a = dps.linear(xd, nst.nw, FULL)
    b = dps.linear(xd, nst.nw, FULL)
    torch.cuda.synchronize()
    assert torch.equal(a.view(torch.int16), b.view(torch.int16))


@pytest.mark.parametrize("m", [16, 200])
def test_one_hot_rows_select_weights_exactly(m):
    """x[r] = e_{j_r}: Y[r][c] is exactly W[c][j_r] (full) or its E5M2 part
    (fast); checks operand layout, merge and addressing end to end."""
    n, k = 272, 1024
    w = workloads.weight_fp16(n, k, seed=31)
    nst = Nested(w, 9, n_slots=4000, slot_seed=32, filler_seed=33)
    cols = torch.randperm(k, generator=torch.Generator().manual_seed(34))[:m]
    x = torch.zeros((m, k), dtype=torch.float16)
    x[torch.arange(m), cols] = 1.0
    for mode in (FULL, FAST):
        y = dps.linear(x.to(DEV), nst.nw, mode)
        torch.cuda.synchronize()
        if mode == FULL:
            want = w[:, cols].t().contiguous()
        else:
            want = torch.from_numpy(nst.hi_ref[:, cols.numpy()].T.copy()).view(
                torch.float8_e5m2).to(torch.float16)
        # value equality: a -0 weight times 1 plus +0 terms sums to +0 (IEEE)
        assert torch.equal(y.cpu().float(), want.float()), mode


def test_special_weight_values():
    """Subnormal, signed-zero and infinite weights through both modes."""
    n, k = 32, 256
    w = workloads.weight_fp16(n, k, seed=41)
    w[0, :] = 0.0
    w[1, :] = -0.0
    w[2, ::2] = 6.0e-8          # FP16 subnormal, E5M2 part is zero
    w[3, ::3] = 1.52587890625e-05   # E5M2 subnormal 2^-16
    w[4, 7] = float("inf")
    nst = Nested(w, 8)
    x = workloads.activations_fp16(8, k, seed=42)
    x[:, 7] = 0.5
    for mode in (FULL, FAST):
        y = dps.linear(x.to(DEV), nst.nw, mode)
        torch.cuda.synchronize()
        ref = oracle.linear(_omode(mode), u16(x), nst.hi_ref,
                            nst.res_ref if mode == FULL else None)
        got = y.cpu().double().numpy()
        assert np.isinf(got[:, 4]).all() and (np.sign(got[:, 4]) == np.sign(ref[:, 4])).all()
        keep = np.ones(n, bool)
        keep[4] = False
        assert_close(y[:, torch.from_numpy(keep).to(DEV)], ref[:, keep])


# -----------------------------------------------------------------------------
# FP8 activations (fast-mode prefill)
# -----------------------------------------------------------------------------

@pytest.mark.parametrize("m,n,k", [(128, 256, 1024), (200, 300, 2048), (17, 130, 4096),
                                   (513, 640, 1152)])
def test_linear_fp8_matches_oracle(m, n, k):
    w = workloads.weight_fp16(n, k, seed=51 + m)
    x = workloads.activations_fp16(m, k, seed=52 + m, outlier_frac=0.01, outlier_scale=20.0)
    nst = Nested(w, 21)
    y = dps.linear(x.to(DEV), nst.nw, FAST, act="fp8")
    torch.cuda.synchronize()
    xq, s = oracle.act_quant(u16(x))
    ref = oracle.linear_fp8(xq, s, nst.hi_ref)
    assert_close(y, ref)


def test_linear_fp8_activation_extremes():
    """FP8 activations with an all-zero row (scale 1), rows of tiny, 448-sized
    and near-FP16-maximum values, a row with one nonzero element and a row
    spanning many powers of two: the quantization bit-exact, each row's
    output within the bounds against the oracle, and outputs past the FP16
    range rounded to +-inf exactly where the exact value reaches 65520."""
    m, n, k = 64, 520, 1040
    w = workloads.weight_fp16(n, k, seed=5)
    rng = np.random.default_rng(6)
    x = rng.normal(0, 1, (m, k)).astype(np.float32)
    x[0] = 0
    x[1] = 1e-6 * x[1]
    x[2] = 448.0
    x[3] = np.where(x[3] >= 0, 60000.0, -60000.0)
    x[4, :] = 0
    x[4, 7] = 2.0 ** -20
    x[5] = 448.0 * 2.0 ** np.round(rng.normal(0, 3, k))
    xt = torch.from_numpy(np.clip(x, -65504, 65504).astype(np.float16))
    nst = Nested(w, 12)
    y = dps.linear(xt.to(DEV), nst.nw, FAST, act="fp8")
    xq_d, s_d = dps.quant_rows_e4m3(xt.to(DEV))
    torch.cuda.synchronize()
    xq, s = oracle.act_quant(u16(xt))
    assert np.array_equal(xq_d.cpu().numpy(), xq)
    assert np.array_equal(s_d.cpu().numpy().astype(np.float64), s)
    ref = oracle.linear_fp8(xq, s, nst.hi_ref)
    got = y.cpu().double().numpy()
    over = np.abs(ref) >= 65520.0
    assert over.any()
    assert np.array_equal(np.isinf(got), over)
    assert np.array_equal(np.sign(got[over]), np.sign(ref[over]))
    assert np.all(got[0] == 0)
    # Outputs span many binades here, so instead of the fixed bounds (stated
    # for outputs of moderate size) each one is held to its own error bound:
    # FP16 rounding of the exact value (half an ulp, or half the subnormal
    # step) plus fp32 accumulation over k terms, bounded by k * 2^-24 times
    # the sum of the products' magnitudes (operands decoded by torch).
    wv = torch.from_numpy(nst.hi_ref).view(torch.float8_e5m2).double().numpy()
    xv = torch.from_numpy(xq).view(torch.float8_e4m3fn).double().numpy() * s[:, None]
    sum_abs = np.abs(xv) @ np.abs(wv).T
    bound = 2.0 ** -11 * np.abs(ref) + 2.0 ** -25 + k * 2.0 ** -24 * sum_abs
    keep = ~over
    assert np.all(np.abs(got[keep] - ref[keep]) <= bound[keep])
    assert_close(torch.from_numpy(got[6:]), ref[6:], "rows of N(0, 1) activations")


# -----------------------------------------------------------------------------
# grouped (MoE)
# -----------------------------------------------------------------------------

@pytest.mark.parametrize("counts,n,k,log2c", [
    ((5, 0, 17, 64, 1, 3), 192, 512, 12),           # decode-sized groups, an empty expert
    ((100, 0, 300, 129, 7), 160, 1024, 10),          # token-tiled groups
    ((40, 0, 70, 3, 33), 256, 1024, 12),             # 32-token tiles, several per expert
    ((90, 20, 0, 100), 320, 768, 11),                # 64-token tiles
    ((128, 140, 120, 133, 110, 125, 131, 137), 256, 256, 21),
])
@pytest.mark.parametrize("mode", [FAST, FULL], ids=["fast", "full"])
def test_grouped_matches_oracle(counts, n, k, log2c, mode):
    e = len(counts)
    rows = sum(counts)
    w = workloads.weight_fp16(n, k, seed=61, experts=e)
    x = workloads.activations_fp16(rows, k, seed=62)
    offsets = np.zeros(e + 1, dtype=np.int64)
    offsets[1:] = np.cumsum(counts)
    numel = e * n * k
    n_chunks = -(-numel // (1 << log2c))
    nst = Nested(w, log2c, n_slots=n_chunks + 5, slot_seed=63, filler_seed=64)
    nst.check_planes()
    off_dev = torch.from_numpy(offsets.astype(np.int32)).to(DEV)
    y = dps.linear_grouped(x.to(DEV), off_dev, nst.nw, mode)
    torch.cuda.synchronize()
    ref = oracle.linear_grouped(_omode(mode), u16(x), offsets, nst.hi_ref,
                                nst.res_ref if mode == FULL else None)
    assert_close(y, ref)


@pytest.mark.parametrize("m", [1, 2, 5, 16, 40])
def test_grouped_single_expert_workspace_and_values(m):
    """One expert through dps_linear_grouped, with the workspace sized by
    dps_workspace_bytes (the grouped plan can split K where the dense plan
    of the same call does not), against the oracle."""
    n, k = 3459, 1504
    w = workloads.weight_fp16(n, k, seed=75)
    x = workloads.activations_fp16(m, k, seed=76)
    nst = Nested(w, 16)
    nw1 = dps.NestedWeight(nst.nw.hi.view(1, n, k), nst.res)
    off = torch.tensor([0, m], dtype=torch.int32, device=DEV)
    for mode in (FAST, FULL):
        y = dps.linear_grouped(x.to(DEV), off, nw1, mode)
        torch.cuda.synchronize()
        ref = oracle.linear(_omode(mode), u16(x), nst.hi_ref,
                            nst.res_ref if mode == FULL else None)
        assert_close(y, ref, "m=%d mode=%d" % (m, mode))


@pytest.mark.parametrize("counts,n,k", [
    ((5, 0, 17, 64, 1, 3), 192, 512),                  # short groups, an empty expert
    ((100, 0, 300, 129, 7), 160, 1024),                # ragged 128-token tiles, weight-tile tail
    ((128, 140, 120, 133, 110, 125, 131, 137), 256, 256),
    ((300, 0, 41), 256, 4096),                         # few weight tiles: K split
    ((129, 144, 145, 272, 273, 0), 256, 1040),         # tail rows (1-16) in last tiles, a K tail
])
@pytest.mark.parametrize("enc", [dps.ENC_E5M2, dps.ENC_E4M3], ids=["e5m2", "e4m3"])
def test_grouped_fp8_matches_oracle(counts, n, k, enc):
    """Grouped fast mode with FP8 activations: every row quantized with its
    own scale, then each expert's rows against its upper bytes."""
    e = len(counts)
    rows = sum(counts)
    w = workloads.weight_fp16(n, k, seed=91, experts=e)
    x = workloads.activations_fp16(rows, k, seed=92, outlier_frac=0.01, outlier_scale=20.0)
    offsets = np.zeros(e + 1, dtype=np.int64)
    offsets[1:] = np.cumsum(counts)
    nst = Nested(w, 16, enc=enc)
    off_dev = torch.from_numpy(offsets.astype(np.int32)).to(DEV)
    p = dps.plan_info(FAST, "fp8", rows, n, k, experts=e)
    assert p["kernel"] == "gemm_fp8"
    if k == 4096:
        assert p["splits"] > 1
    y = dps.linear_grouped(x.to(DEV), off_dev, nst.nw, FAST, act="fp8")
    torch.cuda.synchronize()
    xq, s = oracle.act_quant(u16(x))
    oenc = oracle.E4M3 if enc == dps.ENC_E4M3 else oracle.E5M2
    ref = np.zeros((rows, n))
    for ex in range(e):
        r0, r1 = offsets[ex], offsets[ex + 1]
        if r1 > r0:
            ref[r0:r1] = oracle.linear_fp8(xq[r0:r1], s[r0:r1], nst.hi_ref[ex], enc=oenc)
    assert_close(y, ref)


def test_grouped_single_expert_equals_dense():
    n, k, m = 300, 512, 90
    w = workloads.weight_fp16(n, k, seed=71)
    x = workloads.activations_fp16(m, k, seed=72).to(DEV)
    nst = Nested(w, 12)
    off = torch.tensor([0, m], dtype=torch.int32, device=DEV)
    nw3 = dps.NestedWeight(nst.nw.hi.view(1, n, k), nst.res)
    for mode in (FAST, FULL):
        a = dps.linear(x, nst.nw, mode)
        b = dps.linear_grouped(x, off, nw3, mode)
        torch.cuda.synchronize()
        assert torch.equal(a.view(torch.int16), b.view(torch.int16))


@pytest.mark.parametrize("counts,n,k", [
    ((129, 144, 545), 256, 1040),                # tails of 1 and 16 rows; 5 tiles; a K tail
    ((145, 272, 0, 273, 600), 384, 1040),        # 128 + 17; 128 + 144; empty; 128, 128, 17
    ((129, 144, 600), 128, 4112),                # one weight tile: four K ranges, the last ragged
])
@pytest.mark.parametrize("enc", [dps.ENC_E5M2, dps.ENC_E4M3], ids=["e5m2", "e4m3"])
@pytest.mark.parametrize("mode", [FAST, FULL], ids=["fast", "full"])
def test_grouped_tail_rows_match_oracle(counts, n, k, enc, mode):
    """Grouped calls on the 128-token tile: an expert's last tile takes up to
    16 rows past its 128 (129 or 144 rows: one tile; 145: 128 + 17; 272: 128
    + 144; 273: three tiles), against the oracle, in both nestings."""
    e = len(counts)
    rows = sum(counts)
    p = dps.plan_info(mode, "fp16", rows, n, k, experts=e)
    assert p["kernel"] == "gemm_f16" and p["tile_tokens"] == 128, p
    if n == 128:
        assert p["splits"] == 4 and k % p["ksplit"] != 0, p
    w = workloads.weight_fp16(n, k, seed=131, experts=e)
    x = workloads.activations_fp16(rows, k, seed=132)
    offsets = np.zeros(e + 1, dtype=np.int64)
    offsets[1:] = np.cumsum(counts)
    nst = Nested(w, 21, enc=enc)
    off_dev = torch.from_numpy(offsets.astype(np.int32)).to(DEV)
    y = dps.linear_grouped(x.to(DEV), off_dev, nst.nw, mode)
    torch.cuda.synchronize()
    oenc = oracle.E4M3 if enc == dps.ENC_E4M3 else oracle.E5M2
    ref = oracle.linear_grouped(_omode(mode), u16(x), offsets, nst.hi_ref,
                                nst.res_ref if mode == FULL else None, enc=oenc)
    assert_close(y, ref)


@pytest.mark.parametrize("seed", range(24))
def test_grouped_tail_rows_random(seed):
    """Seeded random grouped calls whose experts hold 0-39, 120-160 or
    250-290 rows (no tail, up to 16 tail rows past a 128-token tile, or a
    second tile with a tail), random N, K and chunk size, alternating the
    nesting and the mode, against the oracle."""
    rng = np.random.default_rng(7700 + seed)
    e = int(rng.integers(1, 5))
    counts = [int(rng.choice([rng.integers(0, 40), rng.integers(120, 161),
                              rng.integers(250, 291)])) for _ in range(e)]
    counts[0] = max(counts[0], 129)  # at least one expert past a tile
    rows = sum(counts)
    k = 16 * int(rng.integers(8, 160))
    n = int(rng.integers(1, 400))
    enc = dps.ENC_E4M3 if seed % 2 else dps.ENC_E5M2
    mode = FULL if (seed // 2) % 2 else FAST
    w = workloads.weight_fp16(n, k, seed=8000 + seed, experts=e)
    x = workloads.activations_fp16(rows, k, seed=9000 + seed)
    offsets = np.zeros(e + 1, dtype=np.int64)
    offsets[1:] = np.cumsum(counts)
    nst = Nested(w, int(rng.integers(8, 22)), enc=enc)
    off_dev = torch.from_numpy(offsets.astype(np.int32)).to(DEV)
    y = dps.linear_grouped(x.to(DEV), off_dev, nst.nw, mode)
    torch.cuda.synchronize()
    oenc = oracle.E4M3 if enc == dps.ENC_E4M3 else oracle.E5M2
    ref = oracle.linear_grouped(_omode(mode), u16(x), offsets, nst.hi_ref,
                                nst.res_ref if mode == FULL else None, enc=oenc)
    assert_close(y, ref, "counts=%s n=%d k=%d" % (counts, n, k))


@pytest.mark.parametrize("enc", [dps.ENC_E5M2, dps.ENC_E4M3], ids=["e5m2", "e4m3"])
@pytest.mark.parametrize("m", [257, 270, 272])
def test_grouped_tail_rows_equal_dense(m, enc):
    """One expert of 257-272 rows is two 128-token tiles grouped (the second
    with 1-16 tail rows) and three dense; both plans split K alike, and the
    tail rows go through the same MFMA (and K-half) order as a third tile's:
    the outputs agree bit for bit in both modes and with FP8 activations, in
    both nestings."""
    n, k = 300, 512
    w = workloads.weight_fp16(n, k, seed=141)
    x = workloads.activations_fp16(m, k, seed=142).to(DEV)
    nst = Nested(w, 12, enc=enc)
    off = torch.tensor([0, m], dtype=torch.int32, device=DEV)
    nw1 = dps.NestedWeight(nst.nw.hi.view(1, n, k), nst.res, enc)
    for mode, act in ((FAST, "fp16"), (FULL, "fp16"), (FAST, "fp8")):
        pd = dps.plan_info(mode, act, m, n, k)
        pg = dps.plan_info(mode, act, m, n, k, experts=1)
        assert pd == pg and pd["tile_tokens"] == 128, (pd, pg)
        a = dps.linear(x, nst.nw, mode, act=act)
        b = dps.linear_grouped(x, off, nw1, mode, act=act)
        torch.cuda.synchronize()
        assert torch.equal(a.view(torch.int16), b.view(torch.int16)), (m, mode, act)


# -----------------------------------------------------------------------------
# error paths on the device-side entry points
# -----------------------------------------------------------------------------

def test_workspace_too_small_is_rejected():
    n, k, m = 4096, 4096, 64    # 32 weight tiles: K is split, partials need room
    w = workloads.weight_fp16(n, k, seed=81)
    nst = Nested(w, 21)
    need = dps.workspace_bytes(FULL, 0, m, n, k)
    assert need > 0
    x = workloads.activations_fp16(m, k, seed=82).to(DEV)
    small = torch.empty(need - 256, dtype=torch.uint8, device=DEV)
    with pytest.raises(dps.DpsError) as ei:
        dps.linear(x, nst.nw, FULL, workspace=small)
    assert ei.value.status == 4
