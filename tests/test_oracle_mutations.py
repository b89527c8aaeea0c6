"""Plant plausible mistakes in copies of the oracle and check the pins catch them.

Each mutation is a one-place textual change to oracle/dps_oracle.c, compiled
with gcc into a temporary library on the CPU.  The test swaps that library in
for the real one and asserts that at least one pin fails.  This shows the
pins constrain every part of the oracle, not only that the oracle passes them.
"""
import ctypes
import os
import subprocess
import tempfile

import pytest

import oracle
import oracle_pins

SRC = os.path.join(os.path.dirname(oracle.__file__), "dps_oracle.c")

# (id, original text, mutated text)
MUTATIONS = [
    ("split_wrong_shift", "*hi = (uint8_t)(s * 128 + e * 4 + m / 256);",
     "*hi = (uint8_t)(s * 128 + e * 4 + m / 512);"),
    ("residual_lost", "*lo = (uint8_t)(m % 256);", "*lo = (uint8_t)(m % 128);"),
    ("merge_drops_residual_bit", "e * 1024 + mh * 256 + lo);", "e * 1024 + mh * 256 + lo / 2);"),
    ("e5m2_wrong_bias", "return sign * ldexp(1.0 + (double)m / 4.0, e - 15);",
     "return sign * ldexp(1.0 + (double)m / 4.0, e - 16);"),
    ("e5m2_subnormal_dropped", "return sign * ldexp((double)m / 4.0, -14);",
     "return sign * 0.0 * m;"),
    ("fp16_mantissa_width", "return sign * ldexp(1.0 + (double)m / 1024.0, e - 15);",
     "return sign * ldexp(1.0 + (double)m / 512.0, e - 15);"),
    ("table_ignored", "int64_t slot = slots[c];", "int64_t slot = c;"),
    ("chunk_offset_wrong", "int64_t phys = slot * chunk_bytes + (i % chunk_bytes);",
     "int64_t phys = slot * chunk_bytes + (i % (chunk_bytes / 2));"),
    ("weight_transposed", "int64_t i = w_base + c * k + kk;",
     "int64_t i = w_base + (kk % (c + 1)) * k + c % k;"),
    ("expert_base_dropped", "int64_t w_base = e * n * k;", "int64_t w_base = 0;"),
    ("fast_rounds_up", "wrow[kk] = oracle_fast_value(enc, hi[i]);",
     "wrow[kk] = oracle_fast_value(enc, (uint8_t)(hi[i] + 1));"),
    ("x_reversed", "v[i] = oracle_fp16_value(x[r0 * k + i]);",
     "v[i] = oracle_fp16_value(x[r0 * k + (i / k) * k + (k - 1 - i % k)]);"),
    ("rows_x_reversed", "xv[j * k + kk] = oracle_fp16_value(x[rows[j] * k + kk]);",
     "xv[j * k + kk] = oracle_fp16_value(x[rows[j] * k + (k - 1 - kk)]);"),
    ("dot_operand_reversed", "acc += a[kk] * b[kk];", "acc += a[kk] * b[k - 1 - kk];"),
    ("tie_to_odd", "(c & 1) == 0 && (best & 1) == 1", "(c & 1) == 1 && (best & 1) == 0"),
    ("scale_one_step_high", "while (a <= 448.0 * (s / 2.0))", "while (a <= 448.0 * (s / 4.0))"),
    ("fp8_scale_dropped", "y[r * n + c] = scale[r] * dot(xv + r * k, wrow, k);",
     "y[r * n + c] = dot(xv + r * k, wrow, k);"),
    ("e4m3_bias", "return sign * ldexp(1.0 + (double)m / 8.0, e - 7);",
     "return sign * ldexp(1.0 + (double)m / 8.0, e - 8);"),
    # E4M3 nesting and the encoding choice
    ("e4m3_split_exponent", "*hi = (uint8_t)(s * 128 + (e % 16) * 8 + m / 128);",
     "*hi = (uint8_t)(s * 128 + (e / 2) * 8 + m / 128);"),
    ("e4m3_residual_width", "*lo = (uint8_t)(m % 128);", "*lo = (uint8_t)(m % 64);"),
    ("e4m3_merge_reads_top_bit", "mh * 128 + lo % 128);", "mh * 128 + lo);"),
    ("e4m3_merge_exponent", "int e = (hi / 8) % 16, mh = hi % 8;",
     "int e = (hi / 8) % 16 + 1, mh = hi % 8;"),
    ("e4m3_fast_scale", "return ldexp(oracle_e4m3_value(hi), -8);",
     "return ldexp(oracle_e4m3_value(hi), -7);"),
    ("select_ignores_nan", "if (e >= 16 || isnan(oracle_e4m3_value(hi)))", "if (e >= 16)"),
    ("select_ignores_msb", "if (e >= 16 || isnan(oracle_e4m3_value(hi)))",
     "if (e >= 17 || isnan(oracle_e4m3_value(hi)))"),
    ("full_ignores_enc", "oracle_fp16_value(unnest_word(enc, hi[i], p < 0 ? 0 : pool[p]))",
     "oracle_fp16_value(unnest_word(0, hi[i], p < 0 ? 0 : pool[p]))"),
    ("fp8_ignores_enc", "wrow[kk] = oracle_fast_value(enc, hi[c * k + kk]);",
     "wrow[kk] = oracle_e5m2_value(hi[c * k + kk]);"),
    # backup and restore
    ("restore_whole_stream", "for (int64_t i = c0 * chunk_bytes; i < c1 * chunk_bytes && i < numel; ++i) {",
     "for (int64_t i = 0; i < numel; ++i) {"),
    ("restore_shifted", "        pool[p] = backup[i];", "        pool[p] = backup[i > 0 ? i - 1 : 0];"),
    ("backup_identity_table", "        backup[i] = pool[p];", "        backup[i] = pool[i];"),
    ("restore_range_unchecked", "    if (c0 < 0 || c1 < c0 || c1 > used)", "    if (c0 < 0 || c1 < c0)"),
]


@pytest.mark.parametrize("mid,old,new", MUTATIONS, ids=[m[0] for m in MUTATIONS])
def test_pins_catch_planted_mistake(mid, old, new, monkeypatch):
    text = open(SRC).read()
    assert text.count(old) >= 1, "mutation anchor not found: %s" % mid
    mutated = text.replace(old, new, 1)
    with tempfile.TemporaryDirectory() as d:
        src = os.path.join(d, "m.c")
        lib = os.path.join(d, "libm.so")
        with open(src, "w") as f:
            f.write(mutated)
        subprocess.run(["gcc", "-std=c11", "-O2", "-fopenmp", "-fPIC", "-shared", "-w",
                        "-o", lib, src, "-lm"], check=True)
        real = oracle._load()
        # reuse the real library's ctypes signatures on the mutated one
        mlib = ctypes.CDLL(lib)
        for name in dir(real):
            if name.startswith("oracle_"):
                fn = getattr(real, name)
                mf = getattr(mlib, name)
                mf.argtypes, mf.restype = fn.argtypes, fn.restype
        monkeypatch.setattr(oracle, "_lib", mlib)
        failed = []
        for pin in oracle_pins.ALL_PINS:
            try:
                pin()
            except (AssertionError, ValueError):
                failed.append(pin.__name__)
        assert failed, "no pin caught mutation %s" % mid
