"""CPU oracle for SparDA's selection + block-sparse attention path (test infrastructure).

Only the test suite, the smoke check and the benchmark's CPU-baseline leg may import this
package.  It wraps ``sparda_oracle.c`` (plain float64 loops written from the paper) with ctypes
and takes/returns numpy arrays: bf16 tensors travel as ``uint16`` bit patterns, block indices as
``int16``.  It shares no code with the HIP library.

Function map (paper sections in the C file):
  compress_keys  -- Eq. 2 (mean-pooled compressed keys over windows of l_C tokens at stride s_C)
  select_row / forecast_select -- Eq. 1 + Eq. 4 (forced init/local blocks U top-k of the
                    max-pooled Forecast block scores)
  forecast_score_max -- Eq. 4 scores of each row's candidates reduced to their maximum (the
                    scoring of the selection without its top-k)
  multihead_select_row / multihead_select -- the InfLLM-V2 selector SparDA replaces (Sec. 3):
                    per-head softmax over the compressed keys, summed over the group, max-pooled
  attend_row / sparse_attn     -- Eq. 1 + Eq. 5 (softmax attention over the attended blocks)
  gather_blocks                -- Sec. 4.3 / Alg. 2 (selected blocks copied into staging)
  writeback_kv                 -- Sec. 5.3 (new K/V rows written into the host pools)
  stage_append_kv              -- Alg. 2 (the decoded token appended to the staged copy of its block)
  indexer_kl_row               -- Sec. 4.2, Eq. 6-7 (the indexer-training KL over the target's top-k
                                  partition, and its gradient with respect to the Forecast row)
  plan_staging                 -- App. C, NOSI step reuse (keep the previous step's staged blocks,
                                  fetch only the newly selected ones)
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from dataclasses import dataclass

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "sparda_oracle.c")
_LIB = os.path.join(_HERE, "libsparda_oracle.so")

OK = 0
ERR_INVALID_ARG = -1
ERR_UNSUPPORTED = -2


def build(force: bool = True) -> str:
    """Compile the oracle with gcc (plain C11 + OpenMP, no fast-math)."""
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp%d" % os.getpid()
        cmd = ["gcc", "-std=c11", "-O2", "-fopenmp", "-fPIC", "-shared", "-Wall", "-Wextra",
               "-fno-fast-math", _SRC, "-o", tmp, "-lm"]
        subprocess.run(cmd, check=True)
        os.replace(tmp, _LIB)
    return _LIB


class _Shape(ctypes.Structure):
    _fields_ = [
        ("batch", ctypes.c_int32), ("n_kv_heads", ctypes.c_int32),
        ("group_size", ctypes.c_int32), ("head_dim", ctypes.c_int32),
        ("block_size", ctypes.c_int32), ("cmp_kernel", ctypes.c_int32), ("cmp_stride", ctypes.c_int32),
        ("n_init", ctypes.c_int32), ("n_local", ctypes.c_int32), ("k_total", ctypes.c_int32),
        ("t_cap", ctypes.c_int64), ("nc_cap", ctypes.c_int64),
    ]


@dataclass(frozen=True)
class Shape:
    batch: int
    n_kv_heads: int
    group_size: int
    head_dim: int = 128
    block_size: int = 64
    n_init: int = 1
    n_local: int = 2
    k_total: int = 16
    t_cap: int = 4096
    nc_cap: int = 64
    cmp_kernel: int | None = None
    cmp_stride: int | None = None

    @property
    def n_q_heads(self) -> int:
        return self.n_kv_heads * self.group_size

    def c(self) -> _Shape:
        return _Shape(self.batch, self.n_kv_heads, self.group_size, self.head_dim, self.block_size,
                      self.block_size if self.cmp_kernel is None else self.cmp_kernel,
                      self.block_size if self.cmp_stride is None else self.cmp_stride,
                      self.n_init, self.n_local, self.k_total, self.t_cap, self.nc_cap)


_lib = None


def open_library(path: str):
    """Load an oracle shared library and declare its prototypes."""
    lib = ctypes.CDLL(path)
    P = ctypes.c_void_p
    S = ctypes.POINTER(_Shape)
    i32, i64, f64 = ctypes.c_int32, ctypes.c_int64, ctypes.c_double
    lib.sparda_ref_bf16_to_f64.argtypes = [ctypes.c_uint16]
    lib.sparda_ref_bf16_to_f64.restype = f64
    lib.sparda_ref_f64_to_bf16.argtypes = [f64]
    lib.sparda_ref_f64_to_bf16.restype = ctypes.c_uint16
    lib.sparda_ref_set_threads.argtypes = [ctypes.c_int]
    lib.sparda_ref_set_threads.restype = ctypes.c_int
    lib.sparda_ref_compress_keys.argtypes = [S, P, i64, i32, i32, P]
    lib.sparda_ref_select_row.argtypes = [S, P, i32, i64, P, i32, i32, i32, P, P, P, P]
    lib.sparda_ref_forecast_select.argtypes = [S, P, i32, i64, P, P, P]
    lib.sparda_ref_forecast_score_max.argtypes = [S, P, i32, i64, P, P]
    lib.sparda_ref_multihead_select_row.argtypes = [S, P, i32, i64, P, f64, i32, i32, i32, P, P, P, P]
    lib.sparda_ref_multihead_select.argtypes = [S, P, i32, i64, P, f64, P, P]
    lib.sparda_ref_attend_row.argtypes = [S, P, i32, i64, P, P, i32, P, P, f64, i32, i32, i32, P]
    lib.sparda_ref_sparse_attn.argtypes = [S, P, i32, i64, P, P, i32, P, P, f64, P]
    lib.sparda_ref_gather_blocks.argtypes = [S, P, P, P, P, P, P]
    lib.sparda_ref_writeback_kv.argtypes = [S, P, P, i32, i64, P, P]
    lib.sparda_ref_stage_append_kv.argtypes = [S, P, P, i64, P, P, P, P]
    lib.sparda_ref_plan_staging.argtypes = [S, P, P, i64, P, P, P, P, P]
    lib.sparda_ref_indexer_kl_row.argtypes = [S, P, P, i64, i32, i32, P, P, i32, i64, f64, i32, i32, i32, i32, P, P,
                                              P, P]
    for name in ("compress_keys", "select_row", "forecast_select", "forecast_score_max", "multihead_select_row", "multihead_select",
                 "attend_row", "sparse_attn", "gather_blocks", "writeback_kv", "stage_append_kv", "plan_staging",
                 "indexer_kl_row"):
        getattr(lib, "sparda_ref_" + name).restype = ctypes.c_int
    return lib


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build(force=True)
        _lib = open_library(_LIB)
    return _lib


def build_variant(src_text: str, out_path: str) -> str:
    """Compile an edited copy of the oracle source (used by the tests that plant mistakes)."""
    c_path = out_path + ".c"
    with open(c_path, "w") as fh:
        fh.write(src_text)
    subprocess.run(["gcc", "-std=c11", "-O1", "-fopenmp", "-fPIC", "-shared", "-fno-fast-math", c_path,
                    "-o", out_path, "-lm"], check=True)
    return out_path


def source_text() -> str:
    with open(_SRC) as fh:
        return fh.read()


class use_library:
    """Context manager: route this module's functions through another oracle library."""

    def __init__(self, path: str):
        self.path = path

    def __enter__(self):
        global _lib
        self._saved = _load()
        _lib = open_library(self.path)
        return self

    def __exit__(self, *exc):
        global _lib
        _lib = self._saved
        return False


class OracleError(RuntimeError):
    def __init__(self, rc: int, what: str):
        super().__init__(f"oracle {what} returned {rc}")
        self.rc = rc


def _ptr(a: np.ndarray | None):
    if a is None:
        return None
    assert a.flags["C_CONTIGUOUS"], "oracle arrays must be C-contiguous"
    return a.ctypes.data_as(ctypes.c_void_p)


def _check(rc: int, what: str):
    if rc != OK:
        raise OracleError(rc, what)


def _u16(a: np.ndarray) -> np.ndarray:
    a = np.ascontiguousarray(a)
    if a.dtype != np.uint16:
        raise TypeError("bf16 tensors are passed as uint16 bit patterns")
    return a


def set_threads(n: int) -> int:
    """Threads of the oracle's OpenMP loops (n < 1 only reports); returns the count in effect."""
    return int(_load().sparda_ref_set_threads(int(n)))


def bf16_to_f64(bits: int) -> float:
    return _load().sparda_ref_bf16_to_f64(int(bits))


def f64_to_bf16(x: float) -> int:
    return int(_load().sparda_ref_f64_to_bf16(float(x)))


def compress_keys(shape: Shape, k: np.ndarray, t_ctx: int, w_begin: int, w_end: int,
                  k_cmp: np.ndarray | None = None) -> np.ndarray:
    """K~ for compressed-key windows [w_begin, w_end) (blocks when window = stride = block);
    k: uint16 [B][Hkv][t_cap][D]."""
    k = _u16(k)
    if k_cmp is None:
        k_cmp = np.zeros((shape.batch, shape.n_kv_heads, shape.nc_cap, shape.head_dim), np.uint16)
    cs = shape.c()
    _check(_load().sparda_ref_compress_keys(ctypes.byref(cs), _ptr(k), t_ctx, w_begin, w_end, _ptr(k_cmp)),
           "compress_keys")
    return k_cmp


def select_row_windows(shape: Shape, f: np.ndarray, n_q: int, q_pos0: int, k_cmp: np.ndarray, b: int, m: int,
                       r: int):
    """(sel_row int16[k_total], cnt, scores float64[n_blocks] with NaN for non-candidates,
    wins int32[n_blocks]: the window that gives each candidate block its max-pooled score)."""
    f, k_cmp = _u16(f), _u16(k_cmp)
    nb = -(-shape.t_cap // shape.block_size)
    sel = np.empty(shape.k_total, np.int16)
    cnt = np.zeros(1, np.int16)
    scores = np.empty(max(nb, 1), np.float64)
    wins = np.empty(max(nb, 1), np.int32)
    cs = shape.c()
    _check(_load().sparda_ref_select_row(ctypes.byref(cs), _ptr(f), n_q, q_pos0, _ptr(k_cmp), b, m, r,
                                         _ptr(sel), _ptr(cnt), _ptr(scores), _ptr(wins)), "select_row")
    return sel, int(cnt[0]), scores[:nb], wins[:nb]


def select_row(shape: Shape, f: np.ndarray, n_q: int, q_pos0: int, k_cmp: np.ndarray, b: int, m: int, r: int):
    """(sel_row int16[k_total], cnt, scores float64[n_blocks] with NaN for non-candidates)."""
    sel, cnt, scores, _ = select_row_windows(shape, f, n_q, q_pos0, k_cmp, b, m, r)
    return sel, cnt, scores


def forecast_select(shape: Shape, f: np.ndarray, n_q: int, q_pos0: int, k_cmp: np.ndarray):
    """sel int16 [B][Hkv][n_q][k_total], cnt int16 [B][Hkv][n_q]."""
    f, k_cmp = _u16(f), _u16(k_cmp)
    sel = np.empty((shape.batch, shape.n_kv_heads, n_q, shape.k_total), np.int16)
    cnt = np.empty((shape.batch, shape.n_kv_heads, n_q), np.int16)
    cs = shape.c()
    _check(_load().sparda_ref_forecast_select(ctypes.byref(cs), _ptr(f), n_q, q_pos0, _ptr(k_cmp), _ptr(sel),
                                              _ptr(cnt)), "forecast_select")
    return sel, cnt


def forecast_score_max(shape: Shape, f: np.ndarray, n_q: int, q_pos0: int, k_cmp: np.ndarray) -> np.ndarray:
    """Each row's largest candidate score, float64 [B][Hkv][n_q] (-inf without candidates)."""
    f, k_cmp = _u16(f), _u16(k_cmp)
    out = np.empty((shape.batch, shape.n_kv_heads, n_q), np.float64)
    cs = shape.c()
    _check(_load().sparda_ref_forecast_score_max(ctypes.byref(cs), _ptr(f), n_q, q_pos0, _ptr(k_cmp), _ptr(out)),
           "forecast_score_max")
    return out


def multihead_select_row(shape: Shape, q: np.ndarray, n_q: int, q_pos0: int, k_cmp: np.ndarray, sm_scale: float,
                         b: int, m: int, r: int):
    """The InfLLM-V2 multi-head selector for one row: (sel_row, cnt, block scores with NaN for
    non-candidates, wins); q: uint16 [B][Hq][n_q][D]."""
    q, k_cmp = _u16(q), _u16(k_cmp)
    nb = -(-shape.t_cap // shape.block_size)
    sel = np.empty(shape.k_total, np.int16)
    cnt = np.zeros(1, np.int16)
    scores = np.empty(max(nb, 1), np.float64)
    wins = np.empty(max(nb, 1), np.int32)
    cs = shape.c()
    _check(_load().sparda_ref_multihead_select_row(ctypes.byref(cs), _ptr(q), n_q, q_pos0, _ptr(k_cmp),
                                                   float(sm_scale), b, m, r, _ptr(sel), _ptr(cnt), _ptr(scores),
                                                   _ptr(wins)), "multihead_select_row")
    return sel, int(cnt[0]), scores[:nb], wins[:nb]


def multihead_select(shape: Shape, q: np.ndarray, n_q: int, q_pos0: int, k_cmp: np.ndarray, sm_scale: float):
    """sel int16 [B][Hkv][n_q][k_total], cnt int16 [B][Hkv][n_q] of the multi-head selector."""
    q, k_cmp = _u16(q), _u16(k_cmp)
    sel = np.empty((shape.batch, shape.n_kv_heads, n_q, shape.k_total), np.int16)
    cnt = np.empty((shape.batch, shape.n_kv_heads, n_q), np.int16)
    cs = shape.c()
    _check(_load().sparda_ref_multihead_select(ctypes.byref(cs), _ptr(q), n_q, q_pos0, _ptr(k_cmp), float(sm_scale),
                                               _ptr(sel), _ptr(cnt)), "multihead_select")
    return sel, cnt


def attend_row(shape: Shape, q, n_q, q_pos0, k, v, kv_mode, sel, cnt, sm_scale, b, h, r) -> np.ndarray:
    q, k, v = _u16(q), _u16(k), _u16(v)
    sel = np.ascontiguousarray(sel, np.int16)
    cnt = np.ascontiguousarray(cnt, np.int16)
    out = np.empty(shape.head_dim, np.float64)
    cs = shape.c()
    _check(_load().sparda_ref_attend_row(ctypes.byref(cs), _ptr(q), n_q, q_pos0, _ptr(k), _ptr(v), kv_mode,
                                         _ptr(sel), _ptr(cnt), float(sm_scale), b, h, r, _ptr(out)),
           "attend_row")
    return out


def sparse_attn(shape: Shape, q, n_q, q_pos0, k, v, kv_mode, sel, cnt, sm_scale) -> np.ndarray:
    """float64 [B][Hq][n_q][D]."""
    q, k, v = _u16(q), _u16(k), _u16(v)
    sel = np.ascontiguousarray(sel, np.int16)
    cnt = np.ascontiguousarray(cnt, np.int16)
    o = np.empty((shape.batch, shape.n_q_heads, n_q, shape.head_dim), np.float64)
    cs = shape.c()
    _check(_load().sparda_ref_sparse_attn(ctypes.byref(cs), _ptr(q), n_q, q_pos0, _ptr(k), _ptr(v), kv_mode,
                                          _ptr(sel), _ptr(cnt), float(sm_scale), _ptr(o)), "sparse_attn")
    return o


def gather_blocks(shape: Shape, host_k, host_v, sel, cnt, stage_k=None, stage_v=None):
    host_k, host_v = _u16(host_k), _u16(host_v)
    sel = np.ascontiguousarray(sel, np.int16)
    cnt = np.ascontiguousarray(cnt, np.int16)
    st = (shape.batch, shape.n_kv_heads, shape.k_total, shape.block_size, shape.head_dim)
    if stage_k is None:
        stage_k = np.zeros(st, np.uint16)
    if stage_v is None:
        stage_v = np.zeros(st, np.uint16)
    cs = shape.c()
    _check(_load().sparda_ref_gather_blocks(ctypes.byref(cs), _ptr(host_k), _ptr(host_v), _ptr(sel), _ptr(cnt),
                                            _ptr(stage_k), _ptr(stage_v)), "gather_blocks")
    return stage_k, stage_v


def writeback_kv(shape: Shape, k_new, v_new, n_new: int, pos0: int, host_k, host_v):
    """Copies of host_k, host_v (uint16 [B][Hkv][t_cap][D]) with the new rows written at pos0."""
    k_new, v_new = _u16(k_new), _u16(v_new)
    hk, hv = np.array(_u16(host_k), copy=True), np.array(_u16(host_v), copy=True)
    cs = shape.c()
    _check(_load().sparda_ref_writeback_kv(ctypes.byref(cs), _ptr(k_new), _ptr(v_new), n_new, pos0, _ptr(hk),
                                           _ptr(hv)), "writeback_kv")
    return hk, hv


def stage_append_kv(shape: Shape, k_new, v_new, q_pos: int, sel, cnt, stage_k, stage_v):
    """Copies of stage_k, stage_v (uint16 [B][Hkv][k_total][L][D]) with the token at q_pos (k_new,
    v_new: uint16 [B][Hkv][D]) written into every slot s < cnt that holds its block."""
    k_new, v_new = _u16(k_new), _u16(v_new)
    sk, sv = np.array(_u16(stage_k), copy=True), np.array(_u16(stage_v), copy=True)
    sel = np.ascontiguousarray(sel, np.int16)
    cnt = np.ascontiguousarray(cnt, np.int16)
    cs = shape.c()
    _check(_load().sparda_ref_stage_append_kv(ctypes.byref(cs), _ptr(k_new), _ptr(v_new), q_pos, _ptr(sel), _ptr(cnt),
                                              _ptr(sk), _ptr(sv)), "stage_append_kv")
    return sk, sv


def plan_staging(shape: Shape, sel, cnt, q_pos: int, slot_blk, slot_len):
    """One decode step's staging plan; slot_blk / slot_len (int16 [B][Hkv][k_total]) are updated in
    place.  Returns (fetch, sel_staged, n_fetch)."""
    sel = np.ascontiguousarray(sel, np.int16).reshape(shape.batch, shape.n_kv_heads, shape.k_total)
    cnt = np.ascontiguousarray(cnt, np.int16).reshape(shape.batch, shape.n_kv_heads)
    assert slot_blk.dtype == np.int16 and slot_len.dtype == np.int16
    assert slot_blk.flags["C_CONTIGUOUS"] and slot_len.flags["C_CONTIGUOUS"]
    fetch = np.empty_like(slot_blk)
    staged = np.empty_like(slot_blk)
    n_fetch = np.empty((shape.batch, shape.n_kv_heads), np.int32)
    cs = shape.c()
    _check(_load().sparda_ref_plan_staging(ctypes.byref(cs), _ptr(sel), _ptr(cnt), q_pos, _ptr(slot_blk),
                                           _ptr(slot_len), _ptr(fetch), _ptr(staged), _ptr(n_fetch)), "plan_staging")
    return fetch, staged, n_fetch


def indexer_kl_row(shape: Shape, q, kc_tgt, lt: int, st: int, f, kc_pred, n_q: int, q_pos0: int, sm_scale: float,
                   k_top: int, b: int, m: int, r: int):
    """(loss, dF float64[D], selected positions int32[k_top] (-1 padded), n_selected) of one row;
    shape's cmp_kernel / cmp_stride give the prediction grid, kc_tgt: uint16 [B][Hkv][nt_cap][D]."""
    q, kc_tgt, f, kc_pred = _u16(q), _u16(kc_tgt), _u16(f), _u16(kc_pred)
    loss = np.zeros(1, np.float64)
    dF = np.empty(shape.head_dim, np.float64)
    sel = np.empty(max(k_top, 1), np.int32)
    n_sel = np.zeros(1, np.int32)
    cs = shape.c()
    _check(_load().sparda_ref_indexer_kl_row(ctypes.byref(cs), _ptr(q), _ptr(kc_tgt), kc_tgt.shape[2], lt, st,
                                             _ptr(f), _ptr(kc_pred), n_q, q_pos0, float(sm_scale), k_top, b, m, r,
                                             _ptr(loss), _ptr(dF), _ptr(sel), _ptr(n_sel)), "indexer_kl_row")
    return float(loss[0]), dF, sel[:k_top], int(n_sel[0])
