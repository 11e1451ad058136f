"""Thin ctypes binding of libsparda.so (argument marshalling only).

Each function keeps the C name and argument order of include/sparda.h.  Tensors are torch
tensors on the GPU (bf16 tensors as torch.bfloat16, block indices as torch.int16); they are
passed as raw pointers, and every step runs in the library's HIP kernels.  ``stream`` defaults to
torch's current stream.  A nonzero status raises SpardaError with the library's detail text.
The library must have been built (``paper_2606_04511_amd.build.build()``); there is no fallback.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass, field

import torch

_LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libsparda.so")

SPARDA_OK = 0
SPARDA_ERR_INVALID_ARG = -1
SPARDA_ERR_UNSUPPORTED = -2
SPARDA_ERR_WORKSPACE = -3
SPARDA_ERR_HOST_NOT_MAPPED = -4
SPARDA_ERR_HIP = -5
SPARDA_OP_FORECAST_SELECT = 1
SPARDA_OP_SPARSE_ATTN = 2
SPARDA_OP_MULTIHEAD_SELECT = 3
SPARDA_OP_INDEXER_KL = 4
SPARDA_OP_DECODE_STEP = 5
SPARDA_NOALLOC_SCRATCH_BYTES = 4718592  # the static scratch of sparda_sparse_attn_noalloc (include/sparda.h)

EXPORTED = ("sparda_compress_keys", "sparda_forecast_select", "sparda_forecast_score_max", "sparda_multihead_select",
            "sparda_sparse_attn", "sparda_sparse_attn_noalloc", "sparda_gather_blocks", "sparda_stage_append_kv", "sparda_writeback_kv", "sparda_plan_staging", "sparda_indexer_kl",
            "sparda_workspace_size", "sparda_status_string", "sparda_last_error_detail")


class _CShape(ctypes.Structure):
    _fields_ = [
        ("struct_size", ctypes.c_uint32), ("batch", ctypes.c_int32), ("n_kv_heads", ctypes.c_int32),
        ("group_size", ctypes.c_int32), ("head_dim", ctypes.c_int32), ("block_size", ctypes.c_int32),
        ("cmp_kernel", ctypes.c_int32), ("cmp_stride", ctypes.c_int32), ("n_init", ctypes.c_int32),
        ("n_local", ctypes.c_int32), ("k_total", ctypes.c_int32), ("t_cap", ctypes.c_int64),
        ("nc_cap", ctypes.c_int64),
    ]


@dataclass
class SpardaShape:
    batch: int
    n_kv_heads: int
    group_size: int
    k_total: int
    t_cap: int
    nc_cap: int
    n_init: int = 1
    n_local: int = 2
    head_dim: int = 128
    block_size: int = 64
    cmp_kernel: int = 64
    cmp_stride: int = 64
    _c: _CShape = field(default=None, repr=False, compare=False)

    @property
    def n_q_heads(self) -> int:
        return self.n_kv_heads * self.group_size

    def c(self) -> _CShape:
        return _CShape(ctypes.sizeof(_CShape), self.batch, self.n_kv_heads, self.group_size, self.head_dim,
                       self.block_size, self.cmp_kernel, self.cmp_stride, self.n_init, self.n_local, self.k_total,
                       self.t_cap, self.nc_cap)


class SpardaError(RuntimeError):
    def __init__(self, status: int, name: str, detail: str):
        super().__init__(f"{name} failed: {status_string(status)} ({detail})")
        self.status = status


_lib = None


def library_path() -> str:
    return _LIB_PATH


def load() -> ctypes.CDLL:
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            raise RuntimeError(f"{_LIB_PATH} is not built; run paper_2606_04511_amd.build.build() first "
                               "(there is no non-HIP fallback)")
        lib = ctypes.CDLL(_LIB_PATH)
        P, S = ctypes.c_void_p, ctypes.POINTER(_CShape)
        i32, i64 = ctypes.c_int32, ctypes.c_int64
        lib.sparda_compress_keys.argtypes = [S, P, i64, i32, i32, P, P]
        lib.sparda_forecast_select.argtypes = [S, P, i32, i64, P, P, P, P, ctypes.c_size_t, P]
        lib.sparda_forecast_score_max.argtypes = [S, P, i32, i64, P, P, P]
        lib.sparda_multihead_select.argtypes = [S, P, i32, i64, P, ctypes.c_float, P, P, P, ctypes.c_size_t, P]
        lib.sparda_sparse_attn.argtypes = [S, P, i32, i64, P, P, i32, P, P, ctypes.c_float, P, P, ctypes.c_size_t, P]
        lib.sparda_sparse_attn_noalloc.argtypes = [S, P, i32, i64, P, P, i32, P, P, ctypes.c_float, P, P]
        lib.sparda_decode_step.argtypes = [S, P, i64, P, P, P, P, ctypes.c_float, P, P, P, P, ctypes.c_size_t, P]
        lib.sparda_plan_staging.argtypes = [S, P, P, i64, P, P, P, P, P, P, P]
        lib.sparda_indexer_kl.argtypes = [S, P, P, P, P, i32, i64, ctypes.c_float, i32, P, P, P, ctypes.c_size_t, P]
        lib.sparda_gather_blocks.argtypes = [S, P, P, P, P, P, P, i32, P]
        lib.sparda_writeback_kv.argtypes = [S, P, P, i32, i64, P, P, i32, P]
        lib.sparda_stage_append_kv.argtypes = [S, P, P, i64, P, P, P, P, P]
        lib.sparda_workspace_size.argtypes = [S, i32, i32, i64, ctypes.POINTER(ctypes.c_size_t)]
        for name in ("sparda_compress_keys", "sparda_forecast_select", "sparda_forecast_score_max",
                     "sparda_multihead_select", "sparda_sparse_attn", "sparda_sparse_attn_noalloc", "sparda_decode_step",
                     "sparda_gather_blocks",
                     "sparda_stage_append_kv", "sparda_writeback_kv", "sparda_plan_staging", "sparda_indexer_kl",
                     "sparda_workspace_size"):
            getattr(lib, name).restype = ctypes.c_int
        lib.sparda_status_string.argtypes = [ctypes.c_int]
        lib.sparda_status_string.restype = ctypes.c_char_p
        lib.sparda_last_error_detail.argtypes = []
        lib.sparda_last_error_detail.restype = ctypes.c_char_p
        _lib = lib
    return _lib


def status_string(status: int) -> str:
    return load().sparda_status_string(int(status)).decode()


def last_error_detail() -> str:
    return load().sparda_last_error_detail().decode()


def _check(rc: int, name: str):
    if rc != SPARDA_OK:
        raise SpardaError(rc, name, last_error_detail())


def _p(x):
    """Raw pointer of a tensor (or an int address / None)."""
    if x is None:
        return None
    if isinstance(x, int):
        return x
    return x.data_ptr()


def _stream(stream):
    if stream is None:
        return torch.cuda.current_stream().cuda_stream if torch.cuda.is_available() else 0
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def sparda_workspace_size(shape: SpardaShape, op: int, n_q: int, q_pos0: int) -> int:
    n = ctypes.c_size_t(0)
    cs = shape.c()
    _check(load().sparda_workspace_size(ctypes.byref(cs), op, n_q, q_pos0, ctypes.byref(n)), "sparda_workspace_size")
    return int(n.value)


def sparda_compress_keys(shape: SpardaShape, k_cache, t_ctx: int, win_begin: int, win_end: int, k_cmp, stream=None):
    cs = shape.c()
    _check(load().sparda_compress_keys(ctypes.byref(cs), _p(k_cache), t_ctx, win_begin, win_end, _p(k_cmp),
                                       _stream(stream)), "sparda_compress_keys")


def sparda_forecast_select(shape: SpardaShape, f, n_q: int, q_pos0: int, k_cmp, sel, cnt, ws=None, ws_bytes: int = 0,
                           stream=None):
    cs = shape.c()
    if ws is not None and not isinstance(ws, int) and ws_bytes == 0:
        ws_bytes = ws.numel() * ws.element_size()
    _check(load().sparda_forecast_select(ctypes.byref(cs), _p(f), n_q, q_pos0, _p(k_cmp), _p(sel), _p(cnt), _p(ws),
                                         ws_bytes, _stream(stream)), "sparda_forecast_select")


def sparda_forecast_score_max(shape: SpardaShape, f, n_q: int, q_pos0: int, k_cmp, row_max, stream=None):
    cs = shape.c()
    _check(load().sparda_forecast_score_max(ctypes.byref(cs), _p(f), n_q, q_pos0, _p(k_cmp), _p(row_max),
                                            _stream(stream)), "sparda_forecast_score_max")


def sparda_multihead_select(shape: SpardaShape, q, n_q: int, q_pos0: int, k_cmp, sm_scale: float, sel, cnt, ws=None,
                            ws_bytes: int = 0, stream=None):
    cs = shape.c()
    if ws is not None and not isinstance(ws, int) and ws_bytes == 0:
        ws_bytes = ws.numel() * ws.element_size()
    _check(load().sparda_multihead_select(ctypes.byref(cs), _p(q), n_q, q_pos0, _p(k_cmp), float(sm_scale), _p(sel),
                                          _p(cnt), _p(ws), ws_bytes, _stream(stream)), "sparda_multihead_select")


def sparda_sparse_attn(shape: SpardaShape, q, n_q: int, q_pos0: int, k, v, kv_mode: int, sel, cnt, sm_scale: float, o,
                       ws=None, ws_bytes: int = 0, stream=None):
    cs = shape.c()
    if ws is not None and not isinstance(ws, int) and ws_bytes == 0:
        ws_bytes = ws.numel() * ws.element_size()
    _check(load().sparda_sparse_attn(ctypes.byref(cs), _p(q), n_q, q_pos0, _p(k), _p(v), kv_mode, _p(sel), _p(cnt),
                                     float(sm_scale), _p(o), _p(ws), ws_bytes, _stream(stream)), "sparda_sparse_attn")


def sparda_decode_step(shape: SpardaShape, f, q_pos: int, k_cmp, q, k, v, sm_scale: float, sel, cnt, o, ws=None,
                       ws_bytes: int = 0, stream=None):
    cs = shape.c()
    if ws is not None and not isinstance(ws, int) and ws_bytes == 0:
        ws_bytes = ws.numel() * ws.element_size()
    _check(load().sparda_decode_step(ctypes.byref(cs), _p(f), q_pos, _p(k_cmp), _p(q), _p(k), _p(v), float(sm_scale),
                                     _p(sel), _p(cnt), _p(o), _p(ws), ws_bytes, _stream(stream)), "sparda_decode_step")


def sparda_sparse_attn_noalloc(shape: SpardaShape, q, n_q: int, q_pos0: int, k, v, kv_mode: int, sel, cnt,
                               sm_scale: float, o, stream=None):
    cs = shape.c()
    _check(load().sparda_sparse_attn_noalloc(ctypes.byref(cs), _p(q), n_q, q_pos0, _p(k), _p(v), kv_mode, _p(sel),
                                             _p(cnt), float(sm_scale), _p(o), _stream(stream)),
           "sparda_sparse_attn_noalloc")


def sparda_gather_blocks(shape: SpardaShape, host_k, host_v, sel, cnt, stage_k, stage_v, n_workgroups: int,
                         stream=None):
    cs = shape.c()
    _check(load().sparda_gather_blocks(ctypes.byref(cs), _p(host_k), _p(host_v), _p(sel), _p(cnt), _p(stage_k),
                                       _p(stage_v), n_workgroups, _stream(stream)), "sparda_gather_blocks")


def sparda_stage_append_kv(shape: SpardaShape, k_new, v_new, q_pos: int, sel, cnt, stage_k, stage_v, stream=None):
    cs = shape.c()
    _check(load().sparda_stage_append_kv(ctypes.byref(cs), _p(k_new), _p(v_new), q_pos, _p(sel), _p(cnt), _p(stage_k),
                                         _p(stage_v), _stream(stream)), "sparda_stage_append_kv")


def sparda_writeback_kv(shape: SpardaShape, k_new, v_new, n_new: int, pos0: int, host_k, host_v, n_workgroups: int,
                        stream=None):
    cs = shape.c()
    _check(load().sparda_writeback_kv(ctypes.byref(cs), _p(k_new), _p(v_new), n_new, pos0, _p(host_k), _p(host_v),
                                      n_workgroups, _stream(stream)), "sparda_writeback_kv")


def sparda_plan_staging(shape: SpardaShape, sel, cnt, q_pos: int, slot_blk, slot_len, fetch, sel_staged, stage_cnt,
                        n_fetch, stream=None):
    cs = shape.c()
    _check(load().sparda_plan_staging(ctypes.byref(cs), _p(sel), _p(cnt), q_pos, _p(slot_blk), _p(slot_len), _p(fetch),
                                      _p(sel_staged), _p(stage_cnt), _p(n_fetch), _stream(stream)),
           "sparda_plan_staging")


def sparda_indexer_kl(shape: SpardaShape, q, k, f, k_cmp, n_q: int, q_pos0: int, sm_scale: float, k_top: int, loss, d_f,
                      ws=None, ws_bytes: int = 0, stream=None):
    cs = shape.c()
    if ws is not None and not isinstance(ws, int) and ws_bytes == 0:
        ws_bytes = ws.numel() * ws.element_size()
    _check(load().sparda_indexer_kl(ctypes.byref(cs), _p(q), _p(k), _p(f), _p(k_cmp), n_q, q_pos0, float(sm_scale),
                                    k_top, _p(loss), _p(d_f), _p(ws), ws_bytes, _stream(stream)), "sparda_indexer_kl")
