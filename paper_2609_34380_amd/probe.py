"""Python binding of libdps_probe (include/dps_probe.h): the measured ceilings
of the MI355X units the nested linear layer is bound by -- a streaming read
of HBM with 16-byte loads, back-to-back FP16 / FP8 MFMAs on register
operands, and the GEMMs' global -> LDS fill per CU.  Argument marshalling only; the kernels are in dps_probe.hip.
Not part of the nested-linear boundary: the benchmark states its roofline
fractions against these as well as against the published peaks.
"""
import ctypes
import os

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libdps_probe.so")
EXPORTED = ("dps_probe_stream_read", "dps_probe_mfma", "dps_probe_lds_fill", "dps_probe_mfma_lds")
FLOPS_PER_MFMA = {0: 16384, 1: 65536}  # 16x16x32 FP16, 16x16x128 FP8

_lib = None


def load_library(path=LIB_PATH):
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError("libdps_probe.so is not built (%s); run __graft_entry__.build()" % path)
    lib = ctypes.CDLL(path)
    P, I64, C = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int
    lib.dps_probe_stream_read.argtypes = [P, I64, C, P, I64, P]
    lib.dps_probe_stream_read.restype = C
    lib.dps_probe_mfma.argtypes = [C, C, I64, P, P]
    lib.dps_probe_mfma.restype = C
    lib.dps_probe_lds_fill.argtypes = [P, I64, C, C, I64, P, P]
    lib.dps_probe_lds_fill.restype = C
    lib.dps_probe_mfma_lds.argtypes = [C, C, C, C, I64, P, P]
    lib.dps_probe_mfma_lds.restype = C
    _lib = lib
    return lib


def _stream():
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def _check(rc, what):
    if rc != 0:
        raise RuntimeError("%s failed (status %d)" % (what, rc))


def stream_read(buf, out, nontemporal=False):
    """Read every byte of the uint8 device tensor buf once; out: uint32 device
    tensor, one word per block (its length sets the grid)."""
    lib = load_library()
    assert buf.is_cuda and buf.dtype == torch.uint8 and buf.is_contiguous()
    assert out.is_cuda and out.dtype == torch.int32 and out.is_contiguous()
    _check(lib.dps_probe_stream_read(ctypes.c_void_p(buf.data_ptr()), buf.numel(),
                                     1 if nontemporal else 0, ctypes.c_void_p(out.data_ptr()),
                                     out.numel(), _stream()), "dps_probe_stream_read")


def mfma(fp8, iters, out):
    """Blocks of four waves, each issuing 8 * iters MFMAs; out: float32 device
    tensor of blocks * 256 elements (its length sets the grid)."""
    lib = load_library()
    assert out.is_cuda and out.dtype == torch.float32 and out.numel() % 256 == 0
    _check(lib.dps_probe_mfma(1 if fp8 else 0, int(iters), out.numel() // 256,
                              ctypes.c_void_p(out.data_ptr()), _stream()), "dps_probe_mfma")


def lds_fill(buf, window_bytes, loaders, stages, out):
    """One block per element of out (int32 device tensor; use one per CU),
    each with `loaders` waves filling `stages` 64 KiB stages of LDS from the
    first window_bytes of the uint8 device tensor buf."""
    lib = load_library()
    assert buf.is_cuda and buf.dtype == torch.uint8 and buf.numel() >= window_bytes
    assert out.is_cuda and out.dtype == torch.int32 and out.is_contiguous()
    _check(lib.dps_probe_lds_fill(ctypes.c_void_p(buf.data_ptr()), int(window_bytes), int(loaders),
                                  int(stages), out.numel(), ctypes.c_void_p(out.data_ptr()),
                                  _stream()), "dps_probe_lds_fill")


MFMA_LDS_SHAPES = {0: (8, 64, 128), 1: (4, 128, 64)}   # waves, wave-tile rows, tokens


def mfma_lds(shape, merge, barrier, iters, blocks, out):
    """The GEMMs' compute loop from LDS (dps_probe_mfma_lds); out: float32
    device tensor of at least blocks * 64 * waves elements.  Returns the
    flops the launch performs."""
    lib = load_library()
    waves, tn, tm = MFMA_LDS_SHAPES[shape]
    assert out.is_cuda and out.dtype == torch.float32 and out.numel() >= blocks * 64 * waves
    _check(lib.dps_probe_mfma_lds(int(shape), int(bool(merge)), int(bool(barrier)), int(iters),
                                  int(blocks), ctypes.c_void_p(out.data_ptr()), _stream()),
           "dps_probe_mfma_lds")
    return blocks * waves * (tn // 16) * (tm // 16) * 2 * 16384.0 * iters
