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
    ("split_wrong_shift", "hi[i] = (uint8_t)(w[i] / 256);", "hi[i] = (uint8_t)(w[i] / 128);"),
    ("residual_lost", "(uint8_t)(w[i] % 256);", "(uint8_t)(w[i] % 128);"),
    ("merge_swapped", "w_out[i] = (uint16_t)((uint16_t)hi[i] * 256 + pool[p]);",
     "w_out[i] = (uint16_t)((uint16_t)pool[p] * 256 + hi[i]);"),
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
    ("fast_rounds_up", "wrow[kk] = oracle_e5m2_value(hi[i]);",
     "wrow[kk] = oracle_e5m2_value((uint8_t)(hi[i] + 1));"),
    ("x_reversed", "acc += oracle_fp16_value(x[r * k + kk]) * wrow[kk];",
     "acc += oracle_fp16_value(x[r * k + (k - 1 - kk)]) * wrow[kk];"),
    ("tie_to_odd", "(c & 1) == 0 && (best & 1) == 1", "(c & 1) == 1 && (best & 1) == 0"),
    ("scale_one_step_high", "while (a <= 448.0 * (s / 2.0))", "while (a <= 448.0 * (s / 4.0))"),
    ("fp8_scale_dropped", "y[r * n + c] = scale[r] * acc;", "y[r * n + c] = acc;"),
    ("e4m3_bias", "return sign * ldexp(1.0 + (double)m / 8.0, e - 7);",
     "return sign * ldexp(1.0 + (double)m / 8.0, e - 8);"),
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
