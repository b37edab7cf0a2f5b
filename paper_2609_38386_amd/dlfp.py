"""Python binding of libdlfp: argument marshalling only.

Every function here has the name of the C entry point it calls and does no
arithmetic of its own: tensors are passed as ``data_ptr()`` plus the current
HIP stream, host arrays as numpy buffers.  If the compiled library is missing,
loading raises -- there is no fallback path.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

import numpy as np

HEAD_DIM = 128
PAGE_SIZE = 16
TILE_ROWS = 128
WORK_INTS = 16
WORKSPACE_HEADER = 256
MAX_GROUPS = 65536
WORKSPACE_PARTIALS = WORKSPACE_HEADER + 4 * MAX_GROUPS
UNCAPPED = -1

_LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libdlfp.so")
_lib = None

STATUS = {0: "DLFP_OK", -1: "DLFP_EINVAL", -2: "DLFP_ERANGE", -3: "DLFP_ENOSPC",
          -4: "DLFP_EHIP", -5: "DLFP_EUNSUPPORTED"}


class DlfpError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        msg = lib().dlfp_status_string(status).decode()
        super().__init__(f"{where}: {STATUS.get(status, status)} ({msg})")


class dlfp_dims(ctypes.Structure):
    _fields_ = [("num_q_heads", ctypes.c_int32), ("num_kv_heads", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("page_size", ctypes.c_int32)]


class dlfp_tuning(ctypes.Structure):
    _fields_ = [("decode_split_tokens", ctypes.c_int32), ("prefill_split_tokens", ctypes.c_int32),
                ("target_units", ctypes.c_int32), ("prefill_tile_tokens", ctypes.c_int32),
                ("prefill_lead_units", ctypes.c_int32),
                ("decode_pages_in_flight", ctypes.c_int32)]


_P32 = ctypes.POINTER(ctypes.c_int32)


class dlfp_meta(ctypes.Structure):
    _fields_ = [("cu_q", _P32), ("q_pos0", _P32), ("slot_mapping", _P32), ("work", _P32),
                ("cap_seqs", ctypes.c_int32), ("cap_tokens", ctypes.c_int32),
                ("cap_work", ctypes.c_int32),
                ("num_seqs", ctypes.c_int32), ("num_tokens", ctypes.c_int32),
                ("num_units", ctypes.c_int32), ("num_prefill_units", ctypes.c_int32),
                ("num_groups", ctypes.c_int32), ("decode_split_tokens", ctypes.c_int32),
                ("prefill_split_tokens", ctypes.c_int32), ("workspace_bytes", ctypes.c_int64),
                ("num_append", ctypes.c_int32), ("num_waiting_units", ctypes.c_int32),
                ("prefill_lead_units", ctypes.c_int32),
                ("decode_pages_in_flight", ctypes.c_int32)]


class dlfp_controller(ctypes.Structure):
    _fields_ = [("target_ms", ctypes.c_double), ("c_initial", ctypes.c_int32),
                ("c_min", ctypes.c_int32), ("c_max", ctypes.c_int32),
                ("quantum", ctypes.c_int32), ("cap", ctypes.c_int32)]


EXPORTS = ["dlfp_build_varlen_meta", "dlfp_kv_append", "dlfp_attention_mixed",
           "dlfp_append_attention_mixed", "dlfp_append_attention_mixed_static",
           "dlfp_linear_bf16",
           "dlfp_workspace_init", "dlfp_workspace_error", "dlfp_controller_init",
           "dlfp_controller_step", "dlfp_timer_create", "dlfp_timer_destroy", "dlfp_timer_start",
           "dlfp_timer_stop", "dlfp_timer_elapsed_ms", "dlfp_stream_hold", "dlfp_status_string",
           "dlfp_version"]


def lib_path() -> str:
    return _LIB_PATH


def lib():
    """Load libdlfp.so (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH):
        raise RuntimeError(f"{_LIB_PATH} is missing: build it with "
                           "`python -m paper_2609_38386_amd.build`")
    L = ctypes.CDLL(_LIB_PATH)
    vp, i32, i64, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t
    L.dlfp_build_varlen_meta.argtypes = [ctypes.POINTER(dlfp_dims), ctypes.POINTER(dlfp_tuning),
                                         i32, _P32, _P32, _P32, i32, i32,
                                         ctypes.POINTER(dlfp_meta)]
    L.dlfp_kv_append.argtypes = [ctypes.POINTER(dlfp_dims), i32, vp, vp, vp, vp, vp, i32, vp]
    L.dlfp_attention_mixed.argtypes = [ctypes.POINTER(dlfp_dims), ctypes.POINTER(dlfp_meta),
                                       vp, vp, i32, i32, vp, vp, vp, ctypes.c_float,
                                       vp, i32, vp, sz, vp]
    L.dlfp_append_attention_mixed.argtypes = [ctypes.POINTER(dlfp_dims),
                                              ctypes.POINTER(dlfp_meta), vp, vp, i32, i32, vp,
                                              vp, vp, vp, vp, ctypes.c_float, vp, i32, vp, sz,
                                              vp]
    L.dlfp_append_attention_mixed_static.argtypes = [ctypes.POINTER(dlfp_dims),
                                                     ctypes.POINTER(dlfp_meta), vp, vp, i32, i32,
                                                     vp, vp, vp, vp, vp, ctypes.c_float, vp, i32,
                                                     vp]
    L.dlfp_linear_bf16.argtypes = [i32, i32, i32, vp, i32, vp, vp, i32, i32, vp]
    L.dlfp_workspace_init.argtypes = [vp, sz, vp]
    L.dlfp_workspace_error.argtypes = [vp, _P32, vp]
    L.dlfp_controller_init.argtypes = [ctypes.POINTER(dlfp_controller), ctypes.c_double, i32, i32,
                                       i32, i32]
    L.dlfp_controller_step.argtypes = [ctypes.POINTER(dlfp_controller), i32, i32,
                                       ctypes.c_double, _P32]
    L.dlfp_timer_create.argtypes = [ctypes.POINTER(vp)]
    L.dlfp_timer_destroy.argtypes = [vp]
    L.dlfp_timer_start.argtypes = [vp, vp]
    L.dlfp_timer_stop.argtypes = [vp, vp]
    L.dlfp_timer_elapsed_ms.argtypes = [vp, ctypes.POINTER(ctypes.c_double)]
    L.dlfp_stream_hold.argtypes = [ctypes.c_int32, vp]
    L.dlfp_status_string.argtypes = [ctypes.c_int]
    L.dlfp_status_string.restype = ctypes.c_char_p
    L.dlfp_version.argtypes = []
    for name in EXPORTS:
        if name != "dlfp_status_string":
            getattr(L, name).restype = ctypes.c_int
    _lib = L
    return L


def _check(status: int, where: str):
    if status != 0:
        raise DlfpError(status, where)


def _ptr32(a: np.ndarray):
    return a.ctypes.data_as(_P32)


def _stream(stream) -> ctypes.c_void_p:
    if stream is None:
        import torch
        stream = torch.cuda.current_stream()
    handle = getattr(stream, "cuda_stream", stream)
    return ctypes.c_void_p(int(handle))


def _dptr(t) -> ctypes.c_void_p:
    return ctypes.c_void_p(int(t.data_ptr()))


def make_dims(num_q_heads: int, num_kv_heads: int, head_dim: int = HEAD_DIM,
              page_size: int = PAGE_SIZE) -> dlfp_dims:
    return dlfp_dims(num_q_heads, num_kv_heads, head_dim, page_size)


class Meta:
    """Host metadata of one packed batch (arrays owned here, counts from the library)."""

    def __init__(self, cap_seqs: int, cap_tokens: int, cap_work: int):
        self.cu_q = np.zeros(cap_seqs + 1, dtype=np.int32)
        self.q_pos0 = np.zeros(max(cap_seqs, 1), dtype=np.int32)
        self.slot_mapping = np.zeros(max(cap_tokens, 1), dtype=np.int32)
        self.work_buf = np.zeros((max(cap_work, 1), WORK_INTS), dtype=np.int32)
        self.c = dlfp_meta(_ptr32(self.cu_q), _ptr32(self.q_pos0), _ptr32(self.slot_mapping),
                           _ptr32(self.work_buf), cap_seqs, cap_tokens, cap_work)

    def __getattr__(self, name):
        c = self.__dict__.get("c")
        if c is not None and name in dict(dlfp_meta._fields_):
            return getattr(c, name)
        raise AttributeError(name)

    @property
    def work(self) -> np.ndarray:
        return self.work_buf[:self.c.num_units]

    @property
    def append_records(self) -> np.ndarray:
        return self.work_buf[self.c.num_units:self.c.num_units + self.c.num_append]

    @property
    def records(self) -> np.ndarray:
        """Units followed by append records: what the device copy of the work list holds."""
        return self.work_buf[:self.c.num_units + self.c.num_append]


def dlfp_build_varlen_meta(dims: dlfp_dims, q_len, kv_len, block_table: np.ndarray,
                           num_blocks: int, tuning: Optional[dlfp_tuning] = None) -> Meta:
    """Build metadata; sizes the host arrays with a first capacity-probing call."""
    L = lib()
    q_len = np.ascontiguousarray(q_len, dtype=np.int32)
    kv_len = np.ascontiguousarray(kv_len, dtype=np.int32)
    bt = np.ascontiguousarray(block_table, dtype=np.int32)
    n = len(q_len)
    if bt.ndim != 2 or bt.shape[0] != n:
        raise ValueError("block_table must be [num_seqs][max_blocks]")
    tn = tuning if tuning is not None else dlfp_tuning(0, 0, 0)
    probe = Meta(0, 0, 0)
    st = L.dlfp_build_varlen_meta(ctypes.byref(dims), ctypes.byref(tn), n, _ptr32(q_len),
                                  _ptr32(kv_len), _ptr32(bt), bt.shape[1], int(num_blocks),
                                  ctypes.byref(probe.c))
    if st not in (0, -3):
        _check(st, "dlfp_build_varlen_meta")
    meta = Meta(probe.c.num_seqs, probe.c.num_tokens, probe.c.num_units + probe.c.num_append)
    st = L.dlfp_build_varlen_meta(ctypes.byref(dims), ctypes.byref(tn), n, _ptr32(q_len),
                                  _ptr32(kv_len), _ptr32(bt), bt.shape[1], int(num_blocks),
                                  ctypes.byref(meta.c))
    _check(st, "dlfp_build_varlen_meta")
    return meta


def dlfp_kv_append(dims: dlfp_dims, k_new, v_new, slot_mapping, k_cache, v_cache,
                   stream=None) -> None:
    """k_new/v_new: bf16 [T][Hkv][128]; slot_mapping: int32 [T]; caches per the pool layout."""
    n = int(slot_mapping.shape[0])
    num_blocks = int(k_cache.shape[0])
    st = lib().dlfp_kv_append(ctypes.byref(dims), n, _dptr(k_new), _dptr(v_new),
                              _dptr(slot_mapping), _dptr(k_cache), _dptr(v_cache), num_blocks,
                              _stream(stream))
    _check(st, "dlfp_kv_append")


def dlfp_attention_mixed(dims: dlfp_dims, meta: Meta, d_work, d_block_table, q, k_cache,
                         v_cache, scale: float, out, workspace, stream=None) -> None:
    """out dtype selects the output precision (bfloat16 or float32)."""
    import torch
    out_dtype = {torch.bfloat16: 0, torch.float32: 1}[out.dtype]
    st = lib().dlfp_attention_mixed(
        ctypes.byref(dims), ctypes.byref(meta.c), _dptr(d_work), _dptr(d_block_table),
        int(d_block_table.shape[1]),
        int(k_cache.shape[0]), _dptr(q), _dptr(k_cache), _dptr(v_cache), float(scale),
        _dptr(out), out_dtype, _dptr(workspace), int(workspace.numel() * workspace.element_size()),
        _stream(stream))
    _check(st, "dlfp_attention_mixed")


def dlfp_append_attention_mixed(dims: dlfp_dims, meta: Meta, d_work, d_block_table, q, k_new,
                                v_new, k_cache, v_cache, scale: float, out, workspace,
                                stream=None) -> None:
    """dlfp_kv_append + dlfp_attention_mixed in one launch; d_work holds meta.records."""
    import torch
    out_dtype = {torch.bfloat16: 0, torch.float32: 1}[out.dtype]
    st = lib().dlfp_append_attention_mixed(
        ctypes.byref(dims), ctypes.byref(meta.c), _dptr(d_work), _dptr(d_block_table),
        int(d_block_table.shape[1]), int(k_cache.shape[0]), _dptr(q), _dptr(k_new),
        _dptr(v_new), _dptr(k_cache), _dptr(v_cache), float(scale), _dptr(out), out_dtype,
        _dptr(workspace), int(workspace.numel() * workspace.element_size()), _stream(stream))
    _check(st, "dlfp_append_attention_mixed")


STATIC_WORKSPACE_BYTES = 128 << 20


def dlfp_append_attention_mixed_static(dims: dlfp_dims, meta: Meta, d_work, d_block_table, q,
                                       k_new, v_new, k_cache, v_cache, scale: float, out,
                                       stream=None) -> None:
    """dlfp_append_attention_mixed on the library's own device workspace (no allocation)."""
    import torch
    out_dtype = {torch.bfloat16: 0, torch.float32: 1}[out.dtype]
    st = lib().dlfp_append_attention_mixed_static(
        ctypes.byref(dims), ctypes.byref(meta.c), _dptr(d_work), _dptr(d_block_table),
        int(d_block_table.shape[1]), int(k_cache.shape[0]), _dptr(q), _dptr(k_new),
        _dptr(v_new), _dptr(k_cache), _dptr(v_cache), float(scale), _dptr(out), out_dtype,
        _stream(stream))
    _check(st, "dlfp_append_attention_mixed_static")


def dlfp_linear_bf16(x, w, out, stream=None) -> None:
    """out[i][j] = sum_l x[i][l] w[j][l]; x: bf16 [m][k] (rows may be strided),
    w: bf16 [n][k], out: bf16 or float32 [m][n] (rows may be strided)."""
    import torch
    m, k = int(x.shape[0]), int(x.shape[1])
    n = int(w.shape[0])
    if int(w.shape[1]) != k or tuple(out.shape) != (m, n):
        raise ValueError("shapes disagree")
    if x.stride(1) != 1 or w.stride(1) != 1 or out.stride(1) != 1 or not w.is_contiguous():
        raise ValueError("rows must be contiguous")
    out_dtype = {torch.bfloat16: 0, torch.float32: 1}[out.dtype]
    st = lib().dlfp_linear_bf16(m, n, k, _dptr(x), int(x.stride(0)), _dptr(w), _dptr(out),
                                int(out.stride(0)), out_dtype, _stream(stream))
    _check(st, "dlfp_linear_bf16")


def dlfp_workspace_init(workspace, stream=None) -> None:
    st = lib().dlfp_workspace_init(_dptr(workspace),
                                   int(workspace.numel() * workspace.element_size()),
                                   _stream(stream))
    _check(st, "dlfp_workspace_init")


def dlfp_workspace_error(workspace, stream=None) -> int:
    v = np.zeros(1, dtype=np.int32)
    st = lib().dlfp_workspace_error(_dptr(workspace), _ptr32(v), _stream(stream))
    _check(st, "dlfp_workspace_error")
    return int(v[0])


def dlfp_controller_init(target_ms: float, c_initial: int, c_min: int, c_max: int,
                         quantum: int = 128) -> dlfp_controller:
    c = dlfp_controller()
    _check(lib().dlfp_controller_init(ctypes.byref(c), float(target_ms), c_initial, c_min, c_max,
                                      quantum), "dlfp_controller_init")
    return c


def dlfp_controller_step(ctrl: dlfp_controller, num_decoding_next: int, last_was_guarded: bool,
                         observed_ms: float) -> int:
    out = ctypes.c_int32(0)
    _check(lib().dlfp_controller_step(ctypes.byref(ctrl), int(num_decoding_next),
                                      1 if last_was_guarded else 0, float(observed_ms),
                                      ctypes.byref(out)), "dlfp_controller_step")
    return int(out.value)


MAX_HOLD_US = 10000


def dlfp_stream_hold(microseconds: int, stream=None) -> None:
    """Idle the stream for `microseconds` of device time so that launches enqueued
    meanwhile run back to back (see dlfp.h)."""
    _check(lib().dlfp_stream_hold(int(microseconds), _stream(stream)), "dlfp_stream_hold")


class Timer:
    """dlfp_timer_*: HIP events around an iteration's device work."""

    def __init__(self):
        self.h = ctypes.c_void_p()
        _check(lib().dlfp_timer_create(ctypes.byref(self.h)), "dlfp_timer_create")

    def start(self, stream=None):
        _check(lib().dlfp_timer_start(self.h, _stream(stream)), "dlfp_timer_start")

    def stop(self, stream=None):
        _check(lib().dlfp_timer_stop(self.h, _stream(stream)), "dlfp_timer_stop")

    def elapsed_ms(self) -> float:
        ms = ctypes.c_double(0.0)
        _check(lib().dlfp_timer_elapsed_ms(self.h, ctypes.byref(ms)), "dlfp_timer_elapsed_ms")
        return float(ms.value)

    def close(self):
        if self.h:
            lib().dlfp_timer_destroy(self.h)
            self.h = ctypes.c_void_p()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
