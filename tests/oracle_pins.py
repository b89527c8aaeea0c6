"""Checks that pin the CPU oracle to facts outside itself.

Each pin_* function raises AssertionError when the oracle disagrees with
what the paper and the mathematics fix.  Every pin compares against an
independent source: a library routine (numpy's float16, torch's float8
types, numpy matmul, numpy fancy indexing), a hand-worked fixture, a closed
property, or brute force.  test_oracle_pins.py runs them on the oracle;
test_oracle_mutations.py plants mistakes in copies of the oracle and checks
that some pin fails for each.
"""
import os

import numpy as np
import torch

import oracle

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")

ALL16 = np.arange(65536, dtype=np.uint32).astype(np.uint16)


def _e5m2_lib(codes):
    """E5M2 values via torch's float8_e5m2 (library decode)."""
    t = torch.from_numpy(np.ascontiguousarray(codes, dtype=np.uint8))
    return t.view(torch.float8_e5m2).to(torch.float64).numpy()


def _e4m3_lib(codes):
    t = torch.from_numpy(np.ascontiguousarray(codes, dtype=np.uint8))
    return t.view(torch.float8_e4m3fn).to(torch.float64).numpy()


def _fp16_lib(bits):
    return np.ascontiguousarray(bits, dtype=np.uint16).view(np.float16).astype(np.float64)


def _same(a, b):
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    both_nan = np.isnan(a) & np.isnan(b)
    eq = (a == b) & (np.signbit(a) == np.signbit(b))
    return both_nan | eq


def identity_residual(numel, log2_chunk, extra_slots=0):
    c = 1 << log2_chunk
    n_chunks = max(1, -(-numel // c))
    pool = np.zeros((n_chunks + extra_slots) * c, dtype=np.uint8)
    return oracle.Residual(pool, np.arange(n_chunks, dtype=np.int32), log2_chunk)


def random_residual(numel, log2_chunk, n_slots, seed, fill=None):
    rng = np.random.default_rng(seed)
    c = 1 << log2_chunk
    n_chunks = max(1, -(-numel // c))
    assert n_slots >= n_chunks
    slots = rng.permutation(n_slots)[:n_chunks].astype(np.int32)
    if fill is None:
        pool = np.zeros(n_slots * c, dtype=np.uint8)
    else:
        pool = rng.integers(0, 256, size=n_slots * c, dtype=np.uint8)
    return oracle.Residual(pool, slots, log2_chunk)


def residual_stream_by_indexing(res, numel):
    """The logical residual stream read with numpy fancy indexing: the pool
    viewed as [slots][chunk bytes], rows picked by the table, flattened."""
    c = 1 << res.log2_chunk
    return res.pool.reshape(-1, c)[res.slots].reshape(-1)[:numel]


# --------------------------------------------------------------------------
# Number formats
# --------------------------------------------------------------------------

def pin_fp16_decode():
    """Closed-form E5M10 decode of all 65536 patterns == numpy float16."""
    got = np.array([oracle.fp16_value(int(b)) for b in ALL16])
    assert _same(got, _fp16_lib(ALL16)).all()


def pin_e5m2_decode():
    """Closed-form E5M2 decode of all 256 codes == torch float8_e5m2."""
    codes = np.arange(256, dtype=np.uint8)
    got = np.array([oracle.e5m2_value(int(c)) for c in codes])
    assert _same(got, _e5m2_lib(codes)).all()


def pin_e4m3_decode():
    """Closed-form E4M3 decode of all 256 codes == torch float8_e4m3fn."""
    codes = np.arange(256, dtype=np.uint8)
    got = np.array([oracle.e4m3_value(int(c)) for c in codes])
    assert _same(got, _e4m3_lib(codes)).all()


# --------------------------------------------------------------------------
# Split / merge / addressing
# --------------------------------------------------------------------------

def pin_golden_split():
    """Hand-worked split examples (tests/golden/nested_split_examples.txt)."""
    rows = []
    with open(os.path.join(GOLDEN, "nested_split_examples.txt")) as f:
        for line in f:
            if line.strip() and not line.startswith("#"):
                b, h, lo, fast, full = line.split()
                rows.append((int(b, 16), int(h, 16), int(lo, 16), float(fast), float(full)))
    w = np.array([r[0] for r in rows], dtype=np.uint16)
    res = identity_residual(w.size, 8)
    hi = oracle.split(w, res)
    lo = residual_stream_by_indexing(res, w.size)
    assert (hi == np.array([r[1] for r in rows], dtype=np.uint8)).all()
    assert (lo == np.array([r[2] for r in rows], dtype=np.uint8)).all()
    fast = np.array([oracle.e5m2_value(int(h)) for h in hi])
    full = np.array([oracle.fp16_value(int(b)) for b in oracle.merge(hi, res)])
    assert _same(fast, [r[3] for r in rows]).all()
    assert _same(full, [r[4] for r in rows]).all()


def pin_split_is_truncation():
    """For every finite FP16 x, the fast value of its upper byte is x truncated
    toward zero onto the E5M2 grid (largest-magnitude E5M2 value of the same
    sign with |v| <= |x|), the grid coming from torch's float8_e5m2."""
    res = identity_residual(ALL16.size, 12)
    hi = oracle.split(ALL16, res)
    x = _fp16_lib(ALL16)
    fast = _e5m2_lib(hi)
    grid = _e5m2_lib(np.arange(256, dtype=np.uint8))
    mags = np.unique(np.abs(grid[np.isfinite(grid)]))            # sorted, includes 0
    finite = np.isfinite(x)
    idx = np.searchsorted(mags, np.abs(x[finite]), side="right") - 1
    want = np.copysign(mags[idx], x[finite])
    assert _same(fast[finite], want).all()
    # +-inf keep their value; NaN stays non-finite in the E5M2 part
    inf = np.isinf(x)
    assert _same(fast[inf], x[inf]).all()
    assert (~np.isfinite(fast[np.isnan(x)])).all()


def pin_split_merge_identity():
    """merge(split(b)) == b for all 65536 patterns, identity and scattered tables,
    and the residual stream equals the little-endian low bytes (numpy view)."""
    low = ALL16.view(np.uint8)[0::2]
    for res in (identity_residual(ALL16.size, 16),
                random_residual(ALL16.size, 8, 1024, seed=5, fill=True),
                random_residual(ALL16.size, 12, 40, seed=6, fill=True)):
        hi = oracle.split(ALL16, res)
        assert (hi == ALL16.view(np.uint8)[1::2]).all()
        assert (residual_stream_by_indexing(res, ALL16.size) == low).all()
        assert (oracle.merge(hi, res) == ALL16).all()


def pin_residual_addressing():
    """Addresses of every logical byte == numpy fancy-index gather, for
    permuted tables and a partially used last chunk."""
    for numel, log2c, n_slots, seed in ((5000, 8, 64, 1), (70000, 12, 31, 2), (1, 8, 3, 3)):
        res = random_residual(numel, log2c, n_slots, seed)
        res.pool[:] = 0
        marks = np.arange(numel, dtype=np.int64)
        # write the logical index into the pool through the oracle's addresses
        flat = np.zeros(res.pool.size, dtype=np.int64) - 1
        for i in marks:
            flat[oracle.residual_addr(int(i), res)] = i
        c = 1 << log2c
        gathered = flat.reshape(-1, c)[res.slots].reshape(-1)[:numel]
        assert (gathered == marks).all()
    # out-of-range chunk / slot give -1
    res = random_residual(1000, 8, 8, seed=4)
    assert oracle.residual_addr(8 * 256, res) == -1
    bad = oracle.Residual(res.pool, np.array([0, 99, 1, 2], dtype=np.int32), 8)
    assert oracle.residual_addr(300, bad) == -1


# --------------------------------------------------------------------------
# Linear
# --------------------------------------------------------------------------

def _rand_fp16(shape, rng, scale=1.0):
    return (rng.standard_normal(shape) * scale).astype(np.float16).view(np.uint16)


def pin_linear_small():
    """Tiny GEMMs in both modes == numpy fp64 matmul of weights decoded by
    numpy float16 (full) or torch float8_e5m2 (fast), through random tables."""
    rng = np.random.default_rng(11)
    for (m, n, k, log2c) in ((1, 1, 16, 8), (3, 5, 32, 8), (7, 33, 48, 9), (16, 64, 64, 10),
                             (5, 17, 80, 8)):
        w = _rand_fp16((n, k), rng, 0.05)
        x = _rand_fp16((m, k), rng)
        res = random_residual(n * k, log2c, -(-n * k // (1 << log2c)) + 3, seed=m * 7 + n,
                              fill=True)
        hi = oracle.split(w, res)
        xd = _fp16_lib(x)
        y_full = oracle.linear(oracle.FULL, x, hi, res)
        assert np.allclose(y_full, xd @ _fp16_lib(w).T, rtol=1e-12, atol=1e-14)
        y_fast = oracle.linear(oracle.FAST, x, hi, None)
        assert np.allclose(y_fast, xd @ _e5m2_lib(hi).T, rtol=1e-12, atol=1e-14)


def pin_linear_one_hot():
    """x = unit vector e_j: Y[:, c] is exactly W[c][j] in both modes."""
    rng = np.random.default_rng(12)
    n, k = 9, 32
    w = _rand_fp16((n, k), rng, 0.05)
    res = identity_residual(n * k, 8)
    hi = oracle.split(w, res)
    x = np.zeros((k, k), dtype=np.float16)
    x[np.arange(k), np.arange(k)] = 1.0
    x = x.view(np.uint16)
    assert (oracle.linear(oracle.FULL, x, hi, res) == _fp16_lib(w).T).all()
    assert (oracle.linear(oracle.FAST, x, hi, None) == _e5m2_lib(hi).T).all()


def pin_fast_equals_full_with_zero_residual():
    """Fast mode == full mode on the same upper bytes with every residual byte 0."""
    rng = np.random.default_rng(13)
    m, n, k = 4, 12, 64
    w = _rand_fp16((n, k), rng, 0.05)
    x = _rand_fp16((m, k), rng)
    res = identity_residual(n * k, 8)
    hi = oracle.split(w, res)
    res.pool[:] = 0
    assert (oracle.linear(oracle.FAST, x, hi, None) ==
            oracle.linear(oracle.FULL, x, hi, res)).all()


def pin_grouped_is_loop_of_dense():
    """Grouped linear == per-expert numpy matmul on that expert's rows,
    including empty experts; expert e's residual starts at logical e*n*k."""
    rng = np.random.default_rng(14)
    e, n, k = 4, 10, 32
    w = _rand_fp16((e, n, k), rng, 0.05)
    offsets = np.array([0, 3, 3, 8, 9], dtype=np.int64)
    x = _rand_fp16((9, k), rng)
    res = random_residual(e * n * k, 8, 30, seed=15, fill=True)
    hi = oracle.split(w, res)
    xd = _fp16_lib(x)
    for mode in (oracle.FULL, oracle.FAST):
        y = oracle.linear_grouped(mode, x, offsets, hi, res if mode == oracle.FULL else None)
        for ex in range(e):
            r0, r1 = offsets[ex], offsets[ex + 1]
            wd = _fp16_lib(w[ex]) if mode == oracle.FULL else _e5m2_lib(hi[ex])
            assert np.allclose(y[r0:r1], xd[r0:r1] @ wd.T, rtol=1e-12, atol=1e-14)


def pin_linear_rows():
    """Row-sampled linear == the same rows of the full linear."""
    rng = np.random.default_rng(16)
    m, n, k = 11, 20, 48
    w = _rand_fp16((n, k), rng, 0.05)
    x = _rand_fp16((m, k), rng)
    res = random_residual(n * k, 8, 9, seed=17, fill=True)
    hi = oracle.split(w, res)
    rows = np.array([10, 0, 5, 5], dtype=np.int64)
    for mode, r in ((oracle.FULL, res), (oracle.FAST, None)):
        full = oracle.linear(mode, x, hi, r)
        assert (oracle.linear_rows(mode, x, rows, hi, r) == full[rows]).all()


# --------------------------------------------------------------------------
# FP8 activation path
# --------------------------------------------------------------------------

def pin_e4m3_rounding_exhaustive():
    """Every finite FP16 value with |x| <= 448, quantized at scale 1, equals
    torch's RNE cast float32 -> float8_e4m3fn, bit for bit."""
    x = _fp16_lib(ALL16)
    keep = np.isfinite(x) & (np.abs(x) <= 448.0)
    bits = ALL16[keep]
    row = np.concatenate([bits, np.array([np.float16(448.0)]).view(np.uint16)])
    xq, s = oracle.act_quant(row.reshape(1, -1))
    assert s[0] == 1.0
    want = torch.from_numpy(_fp16_lib(row).astype(np.float32)).to(torch.float8_e4m3fn)
    assert (xq[0] == want.view(torch.uint8).numpy()).all()


def pin_act_scale():
    """Row scale is a power of two with 448*s/2 < amax <= 448*s (s = 1 for an
    all-zero row), and the dequantized row is within half an E4M3 step."""
    rng = np.random.default_rng(18)
    rows = []
    for mag in (1e-6, 3e-3, 0.5, 1.0, 7.0, 448.0, 449.0, 896.0, 3000.0, 65504.0):
        r = rng.standard_normal(64) * mag / 3.0
        r[rng.integers(64)] = mag
        rows.append(np.clip(r, -65504, 65504))
    rows.append(np.zeros(64))
    x = np.array(rows).astype(np.float16)
    xq, s = oracle.act_quant(x.view(np.uint16))
    xd = x.astype(np.float64)
    for i in range(x.shape[0]):
        amax = np.abs(xd[i]).max()
        mant, _ = np.frexp(s[i])
        assert mant == 0.5, s[i]
        if amax == 0:
            assert s[i] == 1.0
        else:
            assert 448.0 * s[i] / 2 < amax <= 448.0 * s[i]
        deq = _e4m3_lib(xq[i]) * s[i]
        # half a step: relative 2^-4 for normals, absolute 2^-10 * s below 2^-6 * s
        bound = np.maximum(np.abs(xd[i]) * 2.0 ** -4, 2.0 ** -10 * s[i])
        assert (np.abs(deq - xd[i]) <= bound).all()


def pin_linear_fp8():
    """FP8 linear == s_r * (E4M3 decode via torch) @ (E5M2 decode via torch)^T."""
    rng = np.random.default_rng(19)
    m, n, k = 6, 14, 96
    x = _rand_fp16((m, k), rng, 3.0)
    w = _rand_fp16((n, k), rng, 0.05)
    res = identity_residual(n * k, 8)
    hi = oracle.split(w, res)
    xq, s = oracle.act_quant(x)
    y = oracle.linear_fp8(xq, s, hi)
    want = (_e4m3_lib(xq) * s[:, None]) @ _e5m2_lib(hi).T
    assert np.allclose(y, want, rtol=1e-12, atol=1e-14)


# --------------------------------------------------------------------------
# E4M3 nesting and the per-layer encoding choice
# --------------------------------------------------------------------------

def _e4m3_fast_lib(codes):
    """Fast-mode weights of E4M3 upper bytes: torch float8_e4m3fn times 2^-8."""
    return _e4m3_lib(codes) * 2.0 ** -8


def _eligible_e4m3(bits):
    """Words whose value is finite and below 1.875 in magnitude (numpy float16)."""
    x = _fp16_lib(bits)
    return np.isfinite(x) & (np.abs(x) < 1.875)


def pin_golden_split_e4m3():
    """Hand-worked E4M3 split examples (tests/golden/nested_split_e4m3_examples.txt)."""
    rows = []
    with open(os.path.join(GOLDEN, "nested_split_e4m3_examples.txt")) as f:
        for line in f:
            if line.strip() and not line.startswith("#"):
                b, h, lo, fast, full, elig = line.split()
                rows.append((int(b, 16), int(h, 16), int(lo, 16), float(fast), float(full),
                             int(elig)))
    w = np.array([r[0] for r in rows], dtype=np.uint16)
    res = identity_residual(w.size, 8)
    hi = oracle.split(w, res, enc=oracle.E4M3)
    lo = residual_stream_by_indexing(res, w.size)
    assert (hi == np.array([r[1] for r in rows], dtype=np.uint8)).all()
    assert (lo == np.array([r[2] for r in rows], dtype=np.uint8)).all()
    fast = np.array([oracle.fast_value(oracle.E4M3, int(h)) for h in hi])
    full = np.array([oracle.fp16_value(int(b)) for b in oracle.merge(hi, res, enc=oracle.E4M3)])
    assert _same(fast, [r[3] for r in rows]).all()
    assert _same(full, [r[4] for r in rows]).all()
    for r in rows:
        want = oracle.E4M3 if r[5] else oracle.E5M2
        assert oracle.select_enc(np.array([r[0]], dtype=np.uint16)) == want


def pin_e4m3_split_is_truncation():
    """For every FP16 x with |x| < 1.875 the E4M3 fast value is x truncated toward
    zero onto the grid {E4M3 values * 2^-8} (grid from torch's float8_e4m3fn), and
    its upper byte is the E4M3 code of that value."""
    res = identity_residual(ALL16.size, 12)
    hi = oracle.split(ALL16, res, enc=oracle.E4M3)
    keep = _eligible_e4m3(ALL16)
    x = _fp16_lib(ALL16)[keep]
    fast = np.array([oracle.fast_value(oracle.E4M3, int(h)) for h in hi[keep]])
    assert _same(fast, _e4m3_fast_lib(hi[keep])).all()
    grid = _e4m3_fast_lib(np.arange(256, dtype=np.uint8))
    mags = np.unique(np.abs(grid[np.isfinite(grid)]))
    idx = np.searchsorted(mags, np.abs(x), side="right") - 1
    assert _same(fast, np.copysign(mags[idx], x)).all()


def pin_e4m3_split_merge():
    """E4M3 split then merge returns every word whose exponent MSB is zero; a word
    with that bit set comes back with only that bit cleared (the field-keeping
    reading); residual bytes stay below 128, and a set top bit in a residual byte
    does not change the merged word."""
    for res in (identity_residual(ALL16.size, 16),
                random_residual(ALL16.size, 8, 1024, seed=7, fill=True)):
        hi = oracle.split(ALL16, res, enc=oracle.E4M3)
        lo = residual_stream_by_indexing(res, ALL16.size)
        assert (lo < 128).all()
        back = oracle.merge(hi, res, enc=oracle.E4M3)
        msb = (ALL16 & 0x4000) != 0
        assert (back[~msb] == ALL16[~msb]).all()
        assert ((back[msb] ^ ALL16[msb]) == 0x4000).all()
        c = 1 << res.log2_chunk
        res.pool.reshape(-1, c)[res.slots] |= 0x80
        assert (oracle.merge(hi, res, enc=oracle.E4M3) == back).all()


def pin_select_enc():
    """Per-layer choice: E4M3 for a single word exactly when |x| < 1.875 and x is
    finite (numpy float16), and for a layer exactly when all its words are."""
    got = np.array([oracle.select_enc(ALL16[i:i + 1]) for i in range(ALL16.size)])
    assert (got == np.where(_eligible_e4m3(ALL16), oracle.E4M3, oracle.E5M2)).all()
    rng = np.random.default_rng(21)
    ok = (rng.standard_normal(4096) * 0.3).clip(-1.8, 1.8).astype(np.float16)
    assert oracle.select_enc(ok) == oracle.E4M3
    assert oracle.select_enc(np.zeros(0, dtype=np.float16)) == oracle.E4M3
    for bad in (1.875, -1.875, 2.0, 100.0, np.inf, np.nan):
        w = ok.copy()
        w[rng.integers(w.size)] = bad
        assert oracle.select_enc(w) == oracle.E5M2, bad


def pin_linear_e4m3():
    """E4M3 layers: full mode == numpy fp64 matmul of the FP16 weights, fast mode ==
    matmul of torch-decoded E4M3 upper bytes times 2^-8, and fast == full over an
    all-zero residual; dense, one-hot, grouped and FP8-activation forms."""
    rng = np.random.default_rng(22)
    for (m, n, k, log2c) in ((1, 1, 16, 8), (3, 5, 32, 8), (7, 33, 48, 9), (5, 17, 80, 8)):
        w = _rand_fp16((n, k), rng, 0.4)
        w[_fp16_lib(w) > 1.8] = 0
        w[_fp16_lib(w) < -1.8] = 0
        x = _rand_fp16((m, k), rng)
        res = random_residual(n * k, log2c, -(-n * k // (1 << log2c)) + 3, seed=m + n,
                              fill=True)
        hi = oracle.split(w, res, enc=oracle.E4M3)
        xd = _fp16_lib(x)
        y = oracle.linear(oracle.FULL, x, hi, res, enc=oracle.E4M3)
        assert np.allclose(y, xd @ _fp16_lib(w).T, rtol=1e-12, atol=1e-14)
        y = oracle.linear(oracle.FAST, x, hi, None, enc=oracle.E4M3)
        assert np.allclose(y, xd @ _e4m3_fast_lib(hi).T, rtol=1e-12, atol=1e-14)
        assert (oracle.linear_rows(oracle.FAST, x, np.arange(m), hi, None, enc=oracle.E4M3)
                == y).all()
        zero = identity_residual(n * k, 8)
        assert (oracle.linear(oracle.FULL, x, hi, zero, enc=oracle.E4M3) == y).all()
    # one-hot rows read the weights back exactly
    n, k = 9, 32
    w = _rand_fp16((n, k), rng, 0.3)
    res = identity_residual(n * k, 8)
    hi = oracle.split(w, res, enc=oracle.E4M3)
    eye = np.eye(k, dtype=np.float16).view(np.uint16)
    assert (oracle.linear(oracle.FULL, eye, hi, res, enc=oracle.E4M3) == _fp16_lib(w).T).all()
    assert (oracle.linear(oracle.FAST, eye, hi, None, enc=oracle.E4M3)
            == _e4m3_fast_lib(hi).T).all()
    # grouped: expert e's rows against expert e's weights
    e, n, k = 3, 6, 32
    w = _rand_fp16((e, n, k), rng, 0.3)
    offsets = np.array([0, 2, 2, 5], dtype=np.int64)
    x = _rand_fp16((5, k), rng)
    res = random_residual(e * n * k, 8, 12, seed=23, fill=True)
    hi = oracle.split(w, res, enc=oracle.E4M3)
    for mode in (oracle.FULL, oracle.FAST):
        y = oracle.linear_grouped(mode, x, offsets, hi, res if mode == oracle.FULL else None,
                                  enc=oracle.E4M3)
        for ex in range(e):
            r0, r1 = offsets[ex], offsets[ex + 1]
            wd = _fp16_lib(w[ex]) if mode == oracle.FULL else _e4m3_fast_lib(hi[ex])
            assert np.allclose(y[r0:r1], _fp16_lib(x[r0:r1]) @ wd.T, rtol=1e-12, atol=1e-14)
    # FP8 activations against E4M3 weights
    m, n, k = 6, 14, 96
    x = _rand_fp16((m, k), rng, 3.0)
    w = _rand_fp16((n, k), rng, 0.3)
    hi = oracle.split(w, identity_residual(n * k, 8), enc=oracle.E4M3)
    xq, s = oracle.act_quant(x)
    y = oracle.linear_fp8(xq, s, hi, enc=oracle.E4M3)
    want = (_e4m3_lib(xq) * s[:, None]) @ _e4m3_fast_lib(hi).T
    assert np.allclose(y, want, rtol=1e-12, atol=1e-14)


# --------------------------------------------------------------------------
# Residual backup and restore
# --------------------------------------------------------------------------

def pin_backup_restore():
    """The backup is the split's residual stream (numpy fancy-index gather);
    restoring chunk ranges [c0, c1) of it into a pool overwritten with KV-like
    filler writes exactly those chunks' bytes (numpy scatter through the
    table) and leaves every other byte alone; the empty range is a no-op."""
    rng = np.random.default_rng(24)
    numel, log2c, n_slots = 5000, 8, 64
    w = _rand_fp16(numel, rng, 0.05)
    for enc in (oracle.E5M2, oracle.E4M3):
        res = random_residual(numel, log2c, n_slots, seed=25, fill=True)
        oracle.split(w, res, enc=enc)
        bk = oracle.backup(res, numel)
        assert (bk == residual_stream_by_indexing(res, numel)).all()
        c = 1 << log2c
        n_chunks = res.slots.size
        for c0, c1 in ((0, n_chunks), (3, 7), (n_chunks - 1, n_chunks), (5, 5)):
            pool = rng.integers(0, 256, res.pool.size, dtype=np.uint8)
            want = pool.copy().reshape(-1, c)
            lo, hi = c0 * c, min(c1 * c, numel)
            stream = np.zeros(c1 * c if c1 > c0 else 0, dtype=np.uint8)
            stream[:hi - lo] = bk[lo:hi]
            blocks = stream.reshape(-1, c)
            for j, chunk in enumerate(range(c0, c1)):
                nb = min(c, numel - chunk * c)
                want[res.slots[chunk], :nb] = blocks[j, :nb]
            r2 = oracle.Residual(pool, res.slots, log2c)
            oracle.restore(bk, r2, c0, c1)
            assert (r2.pool == want.reshape(-1)).all(), (c0, c1)
    # out-of-range chunk ranges are rejected
    res = random_residual(numel, log2c, n_slots, seed=26)
    bk = np.zeros(numel, dtype=np.uint8)
    for c0, c1 in ((-1, 2), (4, 3), (0, res.slots.size + 1)):
        try:
            oracle.restore(bk, res, c0, c1)
        except ValueError:
            continue
        raise AssertionError("range (%d, %d) accepted" % (c0, c1))


ALL_PINS = [
    pin_fp16_decode, pin_e5m2_decode, pin_e4m3_decode, pin_golden_split,
    pin_split_is_truncation, pin_split_merge_identity, pin_residual_addressing,
    pin_linear_small, pin_linear_one_hot, pin_fast_equals_full_with_zero_residual,
    pin_grouped_is_loop_of_dense, pin_linear_rows, pin_e4m3_rounding_exhaustive,
    pin_act_scale, pin_linear_fp8, pin_golden_split_e4m3, pin_e4m3_split_is_truncation,
    pin_e4m3_split_merge, pin_select_enc, pin_linear_e4m3, pin_backup_restore,
]
