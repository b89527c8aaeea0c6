"""CPU oracle for the DPS nested-precision linear layer.

TEST INFRASTRUCTURE: only tests/, the smoke check and the benchmark's
CPU-baseline leg may import this package.  The product path (the HIP library
and its Python binding) never imports it, and it imports nothing from them.

A thin ctypes layer over dps_oracle.c; every computation happens in that C
file.  Inputs and outputs are numpy arrays on the host.
"""
import ctypes
import os

import numpy as np

from . import build as _build

_lib = None

FULL = 0
FAST = 1
E5M2 = 0
E4M3 = 1


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_build.LIB):
        _build.build()
    lib = ctypes.CDLL(_build.LIB)
    P = ctypes.c_void_p
    I64 = ctypes.c_int64
    I32 = ctypes.c_int32
    lib.oracle_fp16_value.argtypes = [ctypes.c_uint16]
    lib.oracle_fp16_value.restype = ctypes.c_double
    lib.oracle_e5m2_value.argtypes = [ctypes.c_uint8]
    lib.oracle_e5m2_value.restype = ctypes.c_double
    lib.oracle_e4m3_value.argtypes = [ctypes.c_uint8]
    lib.oracle_e4m3_value.restype = ctypes.c_double
    lib.oracle_e4m3_rne.argtypes = [ctypes.c_double, P]
    lib.oracle_e4m3_rne.restype = ctypes.c_int
    lib.oracle_residual_addr.argtypes = [I64, P, I64, I32, I64]
    lib.oracle_residual_addr.restype = I64
    C = ctypes.c_int
    lib.oracle_fast_value.argtypes = [C, ctypes.c_uint8]
    lib.oracle_fast_value.restype = ctypes.c_double
    lib.oracle_select_enc.argtypes = [P, I64]
    lib.oracle_select_enc.restype = ctypes.c_int
    lib.oracle_split.argtypes = [C, P, I64, P, P, I64, P, I64, I32]
    lib.oracle_split.restype = ctypes.c_int
    lib.oracle_merge.argtypes = [C, P, P, I64, P, I64, I32, I64, P]
    lib.oracle_merge.restype = ctypes.c_int
    lib.oracle_restore.argtypes = [P, I64, I64, I64, P, I64, P, I64, I32]
    lib.oracle_restore.restype = ctypes.c_int
    lib.oracle_backup.argtypes = [P, I64, P, I64, I32, I64, P]
    lib.oracle_backup.restype = ctypes.c_int
    lib.oracle_linear.argtypes = [C, C, P, I64, I64, I64, P, P, I64, P, I64, I32, P]
    lib.oracle_linear.restype = ctypes.c_int
    lib.oracle_linear_grouped.argtypes = [C, C, P, P, I64, I64, I64, P, P, I64,
                                          P, I64, I32, P]
    lib.oracle_linear_grouped.restype = ctypes.c_int
    lib.oracle_linear_rows.argtypes = [C, C, P, P, I64, I64, I64, P, P, I64, P,
                                       I64, I32, P]
    lib.oracle_linear_rows.restype = ctypes.c_int
    lib.oracle_act_quant.argtypes = [P, I64, I64, P, P]
    lib.oracle_act_quant.restype = ctypes.c_int
    lib.oracle_linear_fp8.argtypes = [C, P, P, I64, I64, I64, P, P]
    lib.oracle_linear_fp8.restype = ctypes.c_int
    lib.oracle_num_threads.argtypes = []
    lib.oracle_num_threads.restype = ctypes.c_int
    lib.oracle_set_num_threads.argtypes = [ctypes.c_int]
    lib.oracle_set_num_threads.restype = ctypes.c_int
    _lib = lib
    return lib


def _ptr(a):
    if a is None:
        return None
    assert a.flags["C_CONTIGUOUS"], "oracle inputs must be C-contiguous"
    return a.ctypes.data


def _u16(a):
    a = np.ascontiguousarray(a)
    if a.dtype == np.float16:
        a = a.view(np.uint16)
    assert a.dtype == np.uint16, a.dtype
    return a


def _check(rc, what):
    if rc != 0:
        raise ValueError("oracle %s rejected its arguments (rc=%d)" % (what, rc))


class Residual:
    """Residual plane descriptor on the host: pool bytes + chunk slot table."""

    def __init__(self, pool, slots, log2_chunk):
        self.pool = np.ascontiguousarray(pool, dtype=np.uint8)
        self.slots = np.ascontiguousarray(slots, dtype=np.int32)
        self.log2_chunk = int(log2_chunk)

    def args(self):
        return (_ptr(self.pool), self.pool.size, _ptr(self.slots), self.slots.size,
                self.log2_chunk)


def fp16_value(bits):
    lib = _load()
    return lib.oracle_fp16_value(int(bits))


def e5m2_value(code):
    lib = _load()
    return lib.oracle_e5m2_value(int(code))


def e4m3_value(code):
    lib = _load()
    return lib.oracle_e4m3_value(int(code))


def e4m3_rne(v):
    lib = _load()
    out = ctypes.c_uint8(0)
    _check(lib.oracle_e4m3_rne(float(v), ctypes.addressof(out)), "e4m3_rne")
    return out.value


def residual_addr(i, res: Residual):
    lib = _load()
    return lib.oracle_residual_addr(int(i), _ptr(res.slots), res.slots.size,
                                    res.log2_chunk, res.pool.size)


def fast_value(enc, code):
    """Fast-mode weight value of one upper byte under encoding enc."""
    return _load().oracle_fast_value(enc, int(code))


def select_enc(w):
    """Per-layer nested encoding for FP16 words w (any shape): E4M3 or E5M2."""
    lib = _load()
    w = _u16(w)
    return lib.oracle_select_enc(_ptr(w), w.size)


def split(w, res: Residual, enc=E5M2):
    """FP16 words (any shape) -> hi plane (same shape, uint8); writes res.pool."""
    lib = _load()
    w = _u16(w)
    hi = np.empty(w.shape, dtype=np.uint8)
    _check(lib.oracle_split(enc, _ptr(w), w.size, _ptr(hi), *res.args()), "split")
    return hi


def merge(hi, res: Residual, enc=E5M2):
    lib = _load()
    hi = np.ascontiguousarray(hi, dtype=np.uint8)
    out = np.empty(hi.shape, dtype=np.uint16)
    pool, pool_bytes, slots, n_chunks, log2c = res.args()
    _check(lib.oracle_merge(enc, _ptr(hi), pool, pool_bytes, slots, n_chunks, log2c, hi.size,
                            _ptr(out)), "merge")
    return out


def restore(backup, res: Residual, c0=0, c1=None):
    """Write logical chunks [c0, c1) of the residual stream `backup` (uint8,
    numel bytes) into res.pool through the table (in place)."""
    lib = _load()
    backup = np.ascontiguousarray(backup, dtype=np.uint8)
    c = 1 << res.log2_chunk
    if c1 is None:
        c1 = -(-backup.size // c)
    pool, pool_bytes, slots, n_chunks, log2c = res.args()
    _check(lib.oracle_restore(_ptr(backup), backup.size, int(c0), int(c1), pool, pool_bytes,
                              slots, n_chunks, log2c), "restore")


def backup(res: Residual, numel):
    """The residual's logical byte stream (numel bytes) read through the table."""
    lib = _load()
    out = np.empty(int(numel), dtype=np.uint8)
    pool, pool_bytes, slots, n_chunks, log2c = res.args()
    _check(lib.oracle_backup(pool, pool_bytes, slots, n_chunks, log2c, out.size, _ptr(out)),
           "backup")
    return out


def _res_args(res):
    if res is None:
        return (None, 0, None, 0, 0)
    return res.args()


def linear(mode, x, hi, res=None, enc=E5M2):
    """x: fp16 bits [m][k]; hi: uint8 [n][k] -> fp64 [m][n]."""
    lib = _load()
    x = _u16(x)
    hi = np.ascontiguousarray(hi, dtype=np.uint8)
    m, k = x.shape
    n = hi.shape[0]
    assert hi.shape == (n, k)
    y = np.empty((m, n), dtype=np.float64)
    _check(lib.oracle_linear(mode, enc, _ptr(x), m, n, k, _ptr(hi), *_res_args(res), _ptr(y)),
           "linear")
    return y


def linear_rows(mode, x, rows, hi, res=None, enc=E5M2):
    """Dense linear on the listed rows of x only -> fp64 [len(rows)][n]."""
    lib = _load()
    x = _u16(x)
    hi = np.ascontiguousarray(hi, dtype=np.uint8)
    rows = np.ascontiguousarray(rows, dtype=np.int64)
    k = x.shape[1]
    n = hi.shape[0]
    assert hi.shape == (n, k)
    assert rows.size == 0 or (rows.min() >= 0 and rows.max() < x.shape[0])
    y = np.empty((rows.size, n), dtype=np.float64)
    _check(lib.oracle_linear_rows(mode, enc, _ptr(x), _ptr(rows), rows.size, n, k, _ptr(hi),
                                  *_res_args(res), _ptr(y)), "linear_rows")
    return y


def linear_grouped(mode, x_sorted, offsets, hi, res=None, enc=E5M2):
    """x_sorted fp16 bits [rows][k]; offsets int [E+1]; hi uint8 [E][n][k] -> fp64 [rows][n]."""
    lib = _load()
    x = _u16(x_sorted)
    hi = np.ascontiguousarray(hi, dtype=np.uint8)
    offsets = np.ascontiguousarray(offsets, dtype=np.int64)
    e, n, k = hi.shape
    assert offsets.size == e + 1 and x.shape[1] == k and offsets[-1] == x.shape[0]
    y = np.empty((x.shape[0], n), dtype=np.float64)
    _check(lib.oracle_linear_grouped(mode, enc, _ptr(x), _ptr(offsets), e, n, k, _ptr(hi),
                                     *_res_args(res), _ptr(y)), "linear_grouped")
    return y


def act_quant(x):
    """fp16 bits [m][k] -> (E4M3 codes uint8 [m][k], fp64 power-of-two scale [m])."""
    lib = _load()
    x = _u16(x)
    m, k = x.shape
    xq = np.empty((m, k), dtype=np.uint8)
    s = np.empty(m, dtype=np.float64)
    _check(lib.oracle_act_quant(_ptr(x), m, k, _ptr(xq), _ptr(s)), "act_quant")
    return xq, s


def linear_fp8(xq, scale, hi, enc=E5M2):
    lib = _load()
    xq = np.ascontiguousarray(xq, dtype=np.uint8)
    scale = np.ascontiguousarray(scale, dtype=np.float64)
    hi = np.ascontiguousarray(hi, dtype=np.uint8)
    m, k = xq.shape
    n = hi.shape[0]
    assert hi.shape == (n, k) and scale.shape == (m,)
    y = np.empty((m, n), dtype=np.float64)
    _check(lib.oracle_linear_fp8(enc, _ptr(xq), _ptr(scale), m, n, k, _ptr(hi), _ptr(y)),
           "linear_fp8")
    return y


def num_threads():
    return _load().oracle_num_threads()


def set_num_threads(n):
    """Threads the linear routines use from now on; returns the previous count."""
    return _load().oracle_set_num_threads(int(n))
