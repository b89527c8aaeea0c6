"""Python binding of libdps (include/dps.h): argument marshalling only.

Every computation runs in the HIP kernels of libdps.so; this module turns
torch tensors into device pointers, passes torch's current HIP stream, and
turns status codes into exceptions.  PyTorch provides device memory and
streams, nothing else.  If libdps.so is not built, the first call raises.
"""
import ctypes
import os

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libdps.so")

MODE_FULL = 0
MODE_FAST = 1
ENC_E5M2 = 0
ENC_E4M3 = 1
ACT_FP16 = 0
ACT_FP8_ROWSCALE = 1

_STATUS = {0: "DPS_OK", 1: "DPS_ERR_INVALID_ARG", 2: "DPS_ERR_ALIGNMENT",
           3: "DPS_ERR_UNSUPPORTED", 4: "DPS_ERR_WORKSPACE", 5: "DPS_ERR_HIP",
           6: "DPS_ERR_NO_SPACE", 7: "DPS_ERR_TIMEOUT"}
ERR_NO_SPACE = 6
UNIT_FREE, UNIT_BACKED, UNIT_AVAIL, UNIT_FULL, UNIT_RESTORING = 0, 1, 2, 3, 4

EXPORTED = ("dps_select_enc", "dps_split", "dps_merge", "dps_restore", "dps_backup", "dps_quant_rows_e4m3", "dps_workspace_bytes",
            "dps_plan_info", "dps_linear", "dps_linear_static", "dps_linear_grouped", "dps_status_str", "dps_last_error",
            "dps_sum_create", "dps_sum_destroy", "dps_sum_alloc", "dps_sum_free",
            "dps_sum_restore_begin", "dps_sum_restore_done", "dps_sum_mode",
            "dps_sum_unit_state", "dps_sum_unit_of", "dps_sum_counts", "dps_sum_slots",
            "dps_vmm_granularity", "dps_vmm_create", "dps_vmm_kv_view", "dps_vmm_unit_bytes",
            "dps_vmm_map_residual", "dps_vmm_remap", "dps_vmm_unmap_residual", "dps_vmm_destroy",
            "dps_vmm_last_error", "dps_restore_worker_create", "dps_restore_worker_kick",
            "dps_restore_worker_wait_idle", "dps_restore_worker_restored",
            "dps_restore_worker_destroy", "dps_restore_worker_last_error")


class DpsError(RuntimeError):
    def __init__(self, status, detail):
        self.status = status
        self.name = _STATUS.get(status, str(status))
        super().__init__("%s: %s" % (self.name, detail))


class CResidual(ctypes.Structure):
    _fields_ = [("pool", ctypes.c_void_p), ("pool_bytes", ctypes.c_int64),
                ("slots", ctypes.c_void_p), ("n_chunks", ctypes.c_int64),
                ("log2_chunk", ctypes.c_int32)]


class CRestoreTarget(ctypes.Structure):
    _fields_ = [("backup", ctypes.c_void_p), ("numel", ctypes.c_int64), ("res", CResidual)]


class CWeight(ctypes.Structure):
    _fields_ = [("hi", ctypes.c_void_p), ("res", CResidual), ("experts", ctypes.c_int64),
                ("n", ctypes.c_int64), ("k", ctypes.c_int64), ("enc", ctypes.c_int32)]


_lib = None


def load_library(path=LIB_PATH):
    """Load libdps.so and declare its C signatures.  Raises if it is absent."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError("libdps.so is not built (%s); run __graft_entry__.build() or "
                           "python -m paper_2609_34380_amd.csrc.build" % path)
    lib = ctypes.CDLL(path)
    P, I64, I32, U32 = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32, ctypes.c_uint32
    ST = ctypes.c_int
    lib.dps_select_enc.argtypes = [P, I64, P, P]
    lib.dps_select_enc.restype = ST
    lib.dps_split.argtypes = [ctypes.c_int, P, I64, P, ctypes.POINTER(CResidual), P]
    lib.dps_split.restype = ST
    lib.dps_merge.argtypes = [ctypes.c_int, P, ctypes.POINTER(CResidual), I64, P, P]
    lib.dps_merge.restype = ST
    lib.dps_restore.argtypes = [P, I64, ctypes.POINTER(CResidual), P, I64, I64, I64, P]
    lib.dps_restore.restype = ST
    lib.dps_backup.argtypes = [ctypes.POINTER(CResidual), P, I64, P, I64, P]
    lib.dps_backup.restype = ST
    lib.dps_quant_rows_e4m3.argtypes = [P, I64, I64, P, P, P]
    lib.dps_quant_rows_e4m3.restype = ST
    lib.dps_workspace_bytes.argtypes = [ctypes.c_int, U32, I64, I64, I64, I64]
    lib.dps_workspace_bytes.restype = ctypes.c_size_t
    lib.dps_plan_info.argtypes = [ctypes.c_int, U32, I64, I64, I64, I64, I32, P]
    lib.dps_plan_info.restype = ST
    lib.dps_linear.argtypes = [ctypes.c_int, U32, P, I64, ctypes.POINTER(CWeight), P, P,
                               ctypes.c_size_t, P]
    lib.dps_linear.restype = ST
    lib.dps_linear_static.argtypes = [ctypes.c_int, U32, P, I64, ctypes.POINTER(CWeight), P, P]
    lib.dps_linear_static.restype = ST
    lib.dps_linear_grouped.argtypes = [ctypes.c_int, U32, P, P, I64, ctypes.POINTER(CWeight),
                                       P, P, ctypes.c_size_t, P]
    lib.dps_linear_grouped.restype = ST
    PI64 = ctypes.POINTER(I64)
    lib.dps_sum_create.argtypes = [I64, I64, I64, ctypes.POINTER(P)]
    lib.dps_sum_create.restype = ST
    lib.dps_sum_destroy.argtypes = [P]
    lib.dps_sum_destroy.restype = None
    lib.dps_sum_alloc.argtypes = [P, I64, P]
    lib.dps_sum_alloc.restype = ST
    lib.dps_sum_free.argtypes = [P, P, I64, ctypes.POINTER(I32)]
    lib.dps_sum_free.restype = ST
    lib.dps_sum_restore_begin.argtypes = [P, PI64, PI64]
    lib.dps_sum_restore_begin.restype = ST
    lib.dps_sum_restore_done.argtypes = [P, I64]
    lib.dps_sum_restore_done.restype = ST
    lib.dps_sum_mode.argtypes = [P]
    lib.dps_sum_mode.restype = I32
    lib.dps_sum_unit_state.argtypes = [P, I64]
    lib.dps_sum_unit_state.restype = I32
    lib.dps_sum_unit_of.argtypes = [P, I64]
    lib.dps_sum_unit_of.restype = I64
    lib.dps_sum_counts.argtypes = [P, P]
    lib.dps_sum_counts.restype = ST
    lib.dps_sum_slots.argtypes = [P, I64, I64, I64, P]
    lib.dps_sum_slots.restype = ST
    lib.dps_vmm_granularity.argtypes = [PI64]
    lib.dps_vmm_granularity.restype = ST
    lib.dps_vmm_create.argtypes = [I64, I64, ctypes.POINTER(P)]
    lib.dps_vmm_create.restype = ST
    lib.dps_vmm_kv_view.argtypes = [P]
    lib.dps_vmm_kv_view.restype = P
    lib.dps_vmm_unit_bytes.argtypes = [P]
    lib.dps_vmm_unit_bytes.restype = I64
    lib.dps_vmm_map_residual.argtypes = [P, P, I64, ctypes.POINTER(P)]
    lib.dps_vmm_map_residual.restype = ST
    lib.dps_vmm_remap.argtypes = [P, P, I64, I32]
    lib.dps_vmm_remap.restype = ST
    lib.dps_vmm_unmap_residual.argtypes = [P, P]
    lib.dps_vmm_unmap_residual.restype = ST
    lib.dps_vmm_destroy.argtypes = [P]
    lib.dps_vmm_destroy.restype = None
    lib.dps_vmm_last_error.argtypes = []
    lib.dps_vmm_last_error.restype = ctypes.c_char_p
    lib.dps_restore_worker_create.argtypes = [P, P, I64, I64, I64, ctypes.POINTER(P)]
    lib.dps_restore_worker_create.restype = ST
    lib.dps_restore_worker_kick.argtypes = [P]
    lib.dps_restore_worker_kick.restype = ST
    lib.dps_restore_worker_wait_idle.argtypes = [P, I64]
    lib.dps_restore_worker_wait_idle.restype = ST
    lib.dps_restore_worker_restored.argtypes = [P]
    lib.dps_restore_worker_restored.restype = I64
    lib.dps_restore_worker_destroy.argtypes = [P]
    lib.dps_restore_worker_destroy.restype = None
    lib.dps_restore_worker_last_error.argtypes = []
    lib.dps_restore_worker_last_error.restype = ctypes.c_char_p
    lib.dps_status_str.argtypes = [ST]
    lib.dps_status_str.restype = ctypes.c_char_p
    lib.dps_last_error.argtypes = []
    lib.dps_last_error.restype = ctypes.c_char_p
    _lib = lib
    return lib


def _check(status):
    if status != 0:
        detail = _lib.dps_last_error().decode()
        raise DpsError(status, detail)


def _stream():
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _require_cuda(*tensors):
    for t in tensors:
        if t is not None and not t.is_cuda:
            raise ValueError("libdps works on device tensors only")


class Residual:
    """Residual plane of one tensor: a shared pool (uint8 device tensor) plus
    the int32 device table slots[chunk] = pool slot of that chunk."""

    def __init__(self, pool, slots, log2_chunk):
        _require_cuda(pool, slots)
        assert pool.dtype == torch.uint8 and slots.dtype == torch.int32
        self.pool = pool
        self.slots = slots
        self.log2_chunk = int(log2_chunk)

    def c(self):
        return CResidual(self.pool.data_ptr(), self.pool.numel(), self.slots.data_ptr(),
                         self.slots.numel(), self.log2_chunk)


def _null_residual():
    return CResidual(None, 0, None, 0, 0)


class NestedWeight:
    """A nested weight: upper-byte plane hi ([n][k] or [experts][n][k], uint8),
    its residual (None when only fast mode will be used) and the encoding
    (ENC_E5M2 or ENC_E4M3) both were split with."""

    def __init__(self, hi, residual, enc=ENC_E5M2):
        _require_cuda(hi)
        assert hi.dtype == torch.uint8 and hi.is_contiguous()
        assert enc in (ENC_E5M2, ENC_E4M3)
        self.hi = hi
        self.residual = residual
        self.enc = enc
        if hi.dim() == 2:
            self.experts, self.n, self.k = 1, hi.shape[0], hi.shape[1]
        elif hi.dim() == 3:
            self.experts, self.n, self.k = hi.shape
        else:   # a plain byte plane (split / merge only)
            self.experts, self.n, self.k = 1, 1, hi.numel()
        self._c = None

    def c(self):
        if self._c is None:
            res = self.residual.c() if self.residual is not None else _null_residual()
            self._c = CWeight(self.hi.data_ptr(), res, self.experts, self.n, self.k, self.enc)
        return self._c


def select_enc(w, out=None):
    """Per-layer encoding for FP16 weights w (dps_select_enc): an int32 device
    tensor of one element holding ENC_E4M3 or ENC_E5M2 once the stream runs."""
    lib = load_library()
    _require_cuda(w)
    assert w.dtype == torch.float16 and w.is_contiguous()
    if out is None:
        out = torch.empty(1, dtype=torch.int32, device=w.device)
    _check(lib.dps_select_enc(_ptr(w), w.numel(), _ptr(out), _stream()))
    return out


def split(w, residual, hi=None, enc=ENC_E5M2):
    """FP16 weights -> NestedWeight; the residual bytes are written into
    residual.pool through its chunk table (dps_split)."""
    lib = load_library()
    _require_cuda(w)
    assert w.dtype == torch.float16 and w.is_contiguous()
    if hi is None:
        hi = torch.empty(w.shape, dtype=torch.uint8, device=w.device)
    res = residual.c()
    _check(lib.dps_split(enc, _ptr(w), w.numel(), _ptr(hi), ctypes.byref(res), _stream()))
    return NestedWeight(hi, residual, enc)


def merge(nw, out=None):
    """NestedWeight -> the FP16 weights its two parts describe (dps_merge)."""
    lib = load_library()
    if out is None:
        out = torch.empty(nw.hi.shape, dtype=torch.float16, device=nw.hi.device)
    res = nw.residual.c()
    _check(lib.dps_merge(nw.enc, _ptr(nw.hi), ctypes.byref(res), nw.hi.numel(), _ptr(out),
                         _stream()))
    return out


COPY_BYTES = 4 << 20   # restore copy size used in the paper


def _host_slots(residual, slots_host):
    if slots_host is None:
        slots_host = residual.slots.cpu()
    assert slots_host.dtype == torch.int32 and not slots_host.is_cuda
    return slots_host.contiguous()


def backup(residual, numel, out=None, slots_host=None, copy_bytes=COPY_BYTES):
    """The residual's logical byte stream copied into host memory (dps_backup).
    out: a uint8 CPU tensor of numel bytes, pinned for asynchronous copies
    (a new pinned tensor by default).  Completion follows the current stream."""
    lib = load_library()
    slots_host = _host_slots(residual, slots_host)
    if out is None:
        out = torch.empty(numel, dtype=torch.uint8, pin_memory=True)
    assert out.dtype == torch.uint8 and not out.is_cuda and out.numel() >= numel
    res = residual.c()
    _check(lib.dps_backup(ctypes.byref(res), _ptr(slots_host), numel, _ptr(out), copy_bytes,
                          _stream()))
    return out


def restore(backup_host, residual, numel=None, chunk_begin=0, chunk_end=None, slots_host=None,
            copy_bytes=COPY_BYTES):
    """Copy logical chunks [chunk_begin, chunk_end) of the residual stream from
    the host backup into the pool (dps_restore), on the current stream."""
    lib = load_library()
    assert backup_host.dtype == torch.uint8 and not backup_host.is_cuda
    numel = backup_host.numel() if numel is None else numel
    slots_host = _host_slots(residual, slots_host)
    if chunk_end is None:
        chunk_end = -(-numel // (1 << residual.log2_chunk))
    res = residual.c()
    _check(lib.dps_restore(_ptr(backup_host), numel, ctypes.byref(res), _ptr(slots_host),
                           chunk_begin, chunk_end, copy_bytes, _stream()))


def quant_rows_e4m3(x):
    """FP16 [m][k] -> (E4M3 codes uint8 [m][k], float32 power-of-two row scale [m])."""
    lib = load_library()
    _require_cuda(x)
    assert x.dtype == torch.float16 and x.dim() == 2 and x.is_contiguous()
    m, k = x.shape
    xq = torch.empty((m, k), dtype=torch.uint8, device=x.device)
    scale = torch.empty(m, dtype=torch.float32, device=x.device)
    _check(lib.dps_quant_rows_e4m3(_ptr(x), m, k, _ptr(xq), _ptr(scale), _stream()))
    return xq, scale


def workspace_bytes(mode, act, rows, n, k, experts=1):
    lib = load_library()
    return lib.dps_workspace_bytes(mode, act, rows, n, k, experts)


KERNEL_NAMES = {0: "gemv", 1: "rows", 2: "decode", 3: "gemm_f16", 4: "gemm_fp8"}


def plan_info(mode, act, rows, n, k, experts=1, log2_chunk=21):
    """The launch plan of a linear call (dps_plan_info): a dict with the
    kernel family, weight rows and token rows per block tile, K splits and
    K elements per split."""
    lib = load_library()
    info = (ctypes.c_int64 * 5)()
    _check(lib.dps_plan_info(mode, _act_flag(act), rows, n, k, experts, log2_chunk, info))
    return {"kernel": KERNEL_NAMES[info[0]], "tile_rows": info[1], "tile_tokens": info[2],
            "splits": info[3], "ksplit": info[4]}


def _act_flag(act):
    if act in ("fp16", ACT_FP16):
        return ACT_FP16
    if act in ("fp8", ACT_FP8_ROWSCALE):
        return ACT_FP8_ROWSCALE
    raise ValueError("act must be 'fp16' or 'fp8'")


def _workspace(mode, flag, rows, nw, device, workspace):
    need = workspace_bytes(mode, flag, rows, nw.n, nw.k, nw.experts)
    if need == 0:
        return None, 0
    if workspace is None:
        workspace = torch.empty(need, dtype=torch.uint8, device=device)
    return workspace, workspace.numel()


def linear(x, nw, mode, act="fp16", out=None, workspace=None):
    """Y = X . W^T through dps_linear; mode MODE_FULL or MODE_FAST."""
    lib = load_library()
    _require_cuda(x)
    assert x.dtype == torch.float16 and x.dim() == 2 and x.is_contiguous()
    flag = _act_flag(act)
    m = x.shape[0]
    if out is None:
        out = torch.empty((m, nw.n), dtype=torch.float16, device=x.device)
    ws, ws_bytes = _workspace(mode, flag, m, nw, x.device, workspace)
    _check(lib.dps_linear(mode, flag, _ptr(x), m, ctypes.byref(nw.c()), _ptr(out), _ptr(ws),
                          ws_bytes, _stream()))
    return out


STATIC_SCRATCH_BYTES = 64 << 20   # DPS_STATIC_SCRATCH_BYTES


def linear_static(x, nw, mode, act="fp16", out=None):
    """Y = X . W^T through dps_linear_static: the library's static device
    scratch instead of a workspace, so the call allocates nothing (beyond
    `out` when it is not given)."""
    lib = load_library()
    _require_cuda(x)
    assert x.dtype == torch.float16 and x.dim() == 2 and x.is_contiguous()
    flag = _act_flag(act)
    m = x.shape[0]
    if out is None:
        out = torch.empty((m, nw.n), dtype=torch.float16, device=x.device)
    _check(lib.dps_linear_static(mode, flag, _ptr(x), m, ctypes.byref(nw.c()), _ptr(out),
                                 _stream()))
    return out


def linear_grouped(x_sorted, offsets, nw, mode, act="fp16", out=None, workspace=None):
    """MoE grouped linear through dps_linear_grouped; offsets is an int32
    device tensor of experts + 1 row offsets."""
    lib = load_library()
    _require_cuda(x_sorted, offsets)
    assert offsets.dtype == torch.int32 and offsets.numel() == nw.experts + 1
    flag = _act_flag(act)
    rows = x_sorted.shape[0]
    if out is None:
        out = torch.empty((rows, nw.n), dtype=torch.float16, device=x_sorted.device)
    ws, ws_bytes = _workspace(mode, flag, rows, nw, x_sorted.device, workspace)
    _check(lib.dps_linear_grouped(mode, flag, _ptr(x_sorted), _ptr(offsets), rows,
                                  ctypes.byref(nw.c()), _ptr(out), _ptr(ws), ws_bytes,
                                  _stream()))
    return out


def make_residual(numel, log2_chunk, device, slots=None, pool=None):
    """A residual for `numel` weights: by default a pool of exactly the chunks
    needed with the identity table."""
    c = 1 << log2_chunk
    n_chunks = max(1, -(-numel // c))
    if slots is None:
        slots = torch.arange(n_chunks, dtype=torch.int32)
    slots = slots.to(device=device, dtype=torch.int32)
    if pool is None:
        pool = torch.zeros(max(n_chunks, int(slots.max().item()) + 1) * c, dtype=torch.uint8,
                           device=device)
    return Residual(pool, slots, log2_chunk)


class SumManager:
    """The SUM manager's unit bookkeeping (dps_sum_*): n_units units of
    blocks_per_unit KV blocks, residual r initially bound to unit r."""

    COUNT_NAMES = ("free", "backed", "avail", "full", "restoring", "stale", "evicted",
                   "free_blocks")

    def __init__(self, n_units, blocks_per_unit, n_res):
        lib = load_library()
        h = ctypes.c_void_p()
        _check(lib.dps_sum_create(n_units, blocks_per_unit, n_res, ctypes.byref(h)))
        self._h = h
        self.n_units, self.blocks_per_unit, self.n_res = n_units, blocks_per_unit, n_res

    def close(self):
        if self._h:
            _lib.dps_sum_destroy(self._h)
            self._h = ctypes.c_void_p()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def alloc(self, n):
        """n block ids (a list), or None when the request does not fit."""
        out = (ctypes.c_int64 * max(n, 1))()
        st = _lib.dps_sum_alloc(self._h, n, out)
        if st == ERR_NO_SPACE:
            return None
        _check(st)
        return list(out[:n])

    def free(self, blocks):
        """Free the listed blocks; returns True when restoration should wake."""
        arr = (ctypes.c_int64 * max(len(blocks), 1))(*blocks)
        wake = ctypes.c_int32(0)
        _check(_lib.dps_sum_free(self._h, arr, len(blocks), ctypes.byref(wake)))
        return bool(wake.value)

    def restore_begin(self):
        """(residual, unit) now held for a restore, or None."""
        r, u = ctypes.c_int64(), ctypes.c_int64()
        _check(_lib.dps_sum_restore_begin(self._h, ctypes.byref(r), ctypes.byref(u)))
        return None if r.value < 0 else (r.value, u.value)

    def restore_done(self, residual):
        _check(_lib.dps_sum_restore_done(self._h, residual))

    @property
    def mode(self):
        return _lib.dps_sum_mode(self._h)

    def unit_state(self, unit):
        return _lib.dps_sum_unit_state(self._h, unit)

    def unit_of(self, residual):
        return _lib.dps_sum_unit_of(self._h, residual)

    def counts(self):
        c = (ctypes.c_int64 * 8)()
        _check(_lib.dps_sum_counts(self._h, c))
        return dict(zip(self.COUNT_NAMES, c[:]))

    def slots(self, residual, chunks_per_unit, n_chunks):
        """Host int32 slot table of the residual in its unit."""
        out = torch.empty(max(n_chunks, 1), dtype=torch.int32)
        _check(_lib.dps_sum_slots(self._h, residual, chunks_per_unit, n_chunks,
                                  ctypes.c_void_p(out.data_ptr())))
        return out[:n_chunks]


class _DeviceBytes:
    """A __cuda_array_interface__ over device bytes the library mapped, so
    torch can view them (torch.as_tensor) without owning them."""

    def __init__(self, ptr, nbytes):
        self.__cuda_array_interface__ = {"shape": (int(nbytes),), "typestr": "|u1",
                                         "data": (int(ptr), False), "version": 3,
                                         "strides": None}


def _check_vmm(status):
    if status != 0:
        raise DpsError(status, _lib.dps_vmm_last_error().decode())


def vmm_granularity():
    """Minimum VMM allocation granularity of the current device, bytes."""
    lib = load_library()
    g = ctypes.c_int64()
    _check_vmm(lib.dps_vmm_granularity(ctypes.byref(g)))
    return g.value


class VmmRegion:
    """The shared region through the HIP virtual memory API (dps_vmm_*):
    n_units physical units of unit_bytes, all mapped into the KV view
    (`kv`, a uint8 device tensor over n_units * unit_bytes), and residual
    views mapping chosen units in chunk order.  The tensors returned view
    memory the region owns: drop them before unmapping or closing."""

    def __init__(self, n_units, unit_bytes, device=None):
        lib = load_library()
        self.device = torch.device(device) if device is not None else torch.device(
            "cuda", torch.cuda.current_device())
        h = ctypes.c_void_p()
        with torch.cuda.device(self.device):
            _check_vmm(lib.dps_vmm_create(n_units, unit_bytes, ctypes.byref(h)))
        self._h = h
        self.n_units, self.unit_bytes = int(n_units), int(unit_bytes)
        self.log2_unit = self.unit_bytes.bit_length() - 1
        self.kv = torch.as_tensor(_DeviceBytes(lib.dps_vmm_kv_view(h), n_units * unit_bytes),
                                  device=self.device)

    def map_residual(self, units):
        """A residual view (uint8 device tensor of len(units) * unit_bytes)
        whose piece i maps unit units[i]."""
        arr = (ctypes.c_int32 * len(units))(*[int(u) for u in units])
        va = ctypes.c_void_p()
        _check_vmm(_lib.dps_vmm_map_residual(self._h, arr, len(units), ctypes.byref(va)))
        return torch.as_tensor(_DeviceBytes(va.value, len(units) * self.unit_bytes),
                               device=self.device)

    def remap(self, view, piece, unit):
        _check_vmm(_lib.dps_vmm_remap(self._h, ctypes.c_void_p(view.data_ptr()), int(piece),
                                      int(unit)))

    def unmap(self, view):
        _check_vmm(_lib.dps_vmm_unmap_residual(self._h, ctypes.c_void_p(view.data_ptr())))

    def residual(self, view):
        """The Residual descriptor of a view: the view as its pool, the
        identity chunk table, chunks of one unit."""
        n = view.numel() // self.unit_bytes
        slots = torch.arange(n, dtype=torch.int32, device=self.device)
        return Residual(view, slots, self.log2_unit)

    def close(self):
        if self._h:
            self.kv = None
            _lib.dps_vmm_destroy(self._h)
            self._h = ctypes.c_void_p()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


class RestoreWorker:
    """The SUM manager's restore worker (dps_restore_worker_*): a native
    thread that, when kicked, restores every evicted residual the manager
    hands out -- rewrites its device chunk table to the new unit, copies the
    host backup in on its own stream, reports the restore done.
    targets[r] = (backup pinned uint8 CPU tensor, numel, Residual) of the
    manager's residual r; the tensors must outlive the worker."""

    def __init__(self, sum_manager, targets, chunks_per_unit, copy_bytes=COPY_BYTES):
        lib = load_library()
        arr = (CRestoreTarget * len(targets))()
        for i, (bk, numel, res) in enumerate(targets):
            assert bk.dtype == torch.uint8 and not bk.is_cuda and bk.numel() >= numel
            arr[i] = CRestoreTarget(bk.data_ptr(), int(numel), res.c())
        self._keep = (sum_manager, targets)
        h = ctypes.c_void_p()
        rc = lib.dps_restore_worker_create(sum_manager._h, arr, len(targets), chunks_per_unit,
                                           copy_bytes, ctypes.byref(h))
        if rc != 0:
            raise DpsError(rc, lib.dps_restore_worker_last_error().decode())
        self._h = h

    def kick(self):
        _check(_lib.dps_restore_worker_kick(self._h))

    def wait_idle(self, timeout_ms=60000):
        rc = _lib.dps_restore_worker_wait_idle(self._h, int(timeout_ms))
        if rc != 0:
            raise DpsError(rc, _lib.dps_restore_worker_last_error().decode())

    @property
    def restored(self):
        return _lib.dps_restore_worker_restored(self._h)

    def close(self):
        if self._h:
            _lib.dps_restore_worker_destroy(self._h)
            self._h = ctypes.c_void_p()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
