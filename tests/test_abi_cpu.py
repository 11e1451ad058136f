"""Host-side checks of the C ABI that need no GPU.

The library must load, export every function declared in include/*.h, and reject bad arguments
before it makes any HIP call.  Every call below fails validation, so nothing is launched.
"""
import ctypes
import glob
import math
import os
import re
import subprocess

import pytest

import paper_2606_04511_amd.sparda as sp

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
FAKE = 0x7F0000000000  # 16-byte aligned, never dereferenced: validation fails before any launch


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(sp.library_path()):
        from paper_2606_04511_amd import build
        build.build()
    return sp.load()


def declared_functions():
    names = []
    for h in glob.glob(os.path.join(ROOT, "include", "*.h")):
        text = open(h).read()
        names += re.findall(r"^(?:int|const char\*)\s+(sparda_\w+)\s*\(", text, flags=re.M)
    return sorted(set(names))


def test_every_declared_function_is_exported(lib):
    names = declared_functions()
    assert {"sparda_compress_keys", "sparda_forecast_select", "sparda_sparse_attn",
            "sparda_gather_blocks"} <= set(names)
    out = subprocess.run(["nm", "-D", "--defined-only", sp.library_path()], capture_output=True, text=True,
                         check=True).stdout
    exported = set(re.findall(r"\bT (sparda_\w+)", out))
    for n in names:
        assert n in exported, f"{n} declared in include/ but not exported"
        assert getattr(lib, n) is not None


def test_no_torch_symbols_in_the_library(lib):
    out = subprocess.run(["nm", "-D", sp.library_path()], capture_output=True, text=True, check=True).stdout
    names = [line.split()[-1] for line in out.splitlines() if line.strip()]  # symbol names, not addresses
    assert not [n for n in names if "torch" in n or "c10" in n]


def shape(**kw):
    base = dict(batch=2, n_kv_heads=8, group_size=4, k_total=16, t_cap=4096, nc_cap=64)
    base.update(kw)
    return sp.SpardaShape(**base)


def rc_of(fn, *args):
    with pytest.raises(sp.SpardaError) as ei:
        fn(*args)
    return ei.value.status


@pytest.mark.parametrize("kw,status", [
    (dict(head_dim=64), sp.SPARDA_ERR_UNSUPPORTED),
    (dict(block_size=32), sp.SPARDA_ERR_UNSUPPORTED),
    (dict(cmp_kernel=32, cmp_stride=32), sp.SPARDA_ERR_UNSUPPORTED),
    (dict(cmp_kernel=16, cmp_stride=8), sp.SPARDA_ERR_UNSUPPORTED),
    (dict(group_size=17), sp.SPARDA_ERR_UNSUPPORTED),
    (dict(group_size=0), sp.SPARDA_ERR_INVALID_ARG),
    (dict(k_total=2), sp.SPARDA_ERR_INVALID_ARG),
    (dict(n_local=0), sp.SPARDA_ERR_INVALID_ARG),
    (dict(t_cap=100), sp.SPARDA_ERR_INVALID_ARG),
    (dict(t_cap=64 * 40000), sp.SPARDA_ERR_UNSUPPORTED),
    (dict(k_total=40000), sp.SPARDA_ERR_UNSUPPORTED),
])
def test_shape_validation(lib, kw, status):
    assert rc_of(sp.sparda_compress_keys, shape(**kw), FAKE, 4096, 0, 1, FAKE, 0) == status
    assert sp.last_error_detail() != ""


def test_struct_size_and_null_shape(lib):
    cs = shape().c()
    cs.struct_size = 12
    assert lib.sparda_compress_keys(ctypes.byref(cs), FAKE, 4096, 0, 1, FAKE, None) == sp.SPARDA_ERR_INVALID_ARG
    assert lib.sparda_compress_keys(None, FAKE, 4096, 0, 1, FAKE, None) == sp.SPARDA_ERR_INVALID_ARG


def test_compress_argument_errors(lib):
    s = shape()
    assert rc_of(sp.sparda_compress_keys, s, None, 4096, 0, 1, FAKE, 0) == sp.SPARDA_ERR_INVALID_ARG
    assert rc_of(sp.sparda_compress_keys, s, FAKE + 2, 4096, 0, 1, FAKE, 0) == sp.SPARDA_ERR_INVALID_ARG
    assert rc_of(sp.sparda_compress_keys, s, FAKE, 100, 0, 2, FAKE, 0) == sp.SPARDA_ERR_INVALID_ARG  # incomplete
    assert rc_of(sp.sparda_compress_keys, s, FAKE, 4096, 0, 65, FAKE, 0) == sp.SPARDA_ERR_INVALID_ARG  # > t_ctx
    assert rc_of(sp.sparda_compress_keys, shape(nc_cap=10), FAKE, 4096, 0, 11, FAKE, 0) == sp.SPARDA_ERR_INVALID_ARG
    assert rc_of(sp.sparda_compress_keys, s, FAKE, 5000, 0, 1, FAKE, 0) == sp.SPARDA_ERR_INVALID_ARG  # t_ctx > t_cap
    sp.sparda_compress_keys(s, FAKE, 4096, 3, 3, FAKE, 0)  # empty range: a no-op, nothing launched


def test_select_argument_errors(lib):
    s = shape()
    f = sp.sparda_forecast_select
    assert rc_of(f, s, FAKE, 0, 4095, FAKE, FAKE, FAKE, None, 0, 0) == sp.SPARDA_ERR_INVALID_ARG  # n_q
    assert rc_of(f, s, FAKE, 1, 4096, FAKE, FAKE, FAKE, None, 0, 0) == sp.SPARDA_ERR_INVALID_ARG  # p >= t_cap
    assert rc_of(f, s, FAKE, 1, -1, FAKE, FAKE, FAKE, None, 0, 0) == sp.SPARDA_ERR_INVALID_ARG
    assert rc_of(f, shape(nc_cap=30), FAKE, 1, 4095, FAKE, FAKE, FAKE, None, 0, 0) == sp.SPARDA_ERR_INVALID_ARG
    assert rc_of(f, s, FAKE, 1, 4095, FAKE, FAKE + 1, FAKE, None, 0, 0) == sp.SPARDA_ERR_INVALID_ARG  # sel align
    # multi-row rows with more than 512 candidates take the row-wise path, which needs scratch
    sl = shape(t_cap=65536, nc_cap=1024)
    assert rc_of(f, sl, FAKE, 2, 65534, FAKE, FAKE, FAKE, None, 0, 0) == sp.SPARDA_ERR_WORKSPACE
    need = sp.sparda_workspace_size(sl, sp.SPARDA_OP_FORECAST_SELECT, 2, 65534)
    assert need == 2 * 8 * 2 * 1024 * 4  # rows x stride(1021 -> 1024) x float
    assert rc_of(f, sl, FAKE, 2, 65534, FAKE, FAKE, FAKE, FAKE, need - 4, 0) == sp.SPARDA_ERR_WORKSPACE


def test_score_max_argument_errors(lib):
    """The scoring contraction alone: the (64, 64) grid only, the same row and K~ checks as the
    selection, a 4-byte aligned float output."""
    s = shape()
    m = sp.sparda_forecast_score_max
    assert rc_of(m, s, FAKE, 0, 4095, FAKE, FAKE, 0) == sp.SPARDA_ERR_INVALID_ARG       # n_q
    assert rc_of(m, s, FAKE, 1, 4096, FAKE, FAKE, 0) == sp.SPARDA_ERR_INVALID_ARG       # p >= t_cap
    assert rc_of(m, s, None, 1, 4095, FAKE, FAKE, 0) == sp.SPARDA_ERR_INVALID_ARG       # f
    assert rc_of(m, s, FAKE, 1, 4095, FAKE, FAKE + 2, 0) == sp.SPARDA_ERR_INVALID_ARG   # row_max align
    assert rc_of(m, shape(nc_cap=61), FAKE, 1, 4095, FAKE, FAKE, 0) == sp.SPARDA_ERR_INVALID_ARG  # block 61
    assert rc_of(m, shape(nc_cap=255, cmp_kernel=32, cmp_stride=16), FAKE, 1, 4095, FAKE, FAKE, 0) == \
        sp.SPARDA_ERR_UNSUPPORTED


def test_writeback_argument_errors(lib):
    s = shape()
    wb = sp.sparda_writeback_kv
    assert rc_of(wb, s, FAKE, FAKE, 0, 100, FAKE, FAKE, 8, 0) == sp.SPARDA_ERR_INVALID_ARG      # n_new
    assert rc_of(wb, s, FAKE, FAKE, 2, 4095, FAKE, FAKE, 8, 0) == sp.SPARDA_ERR_INVALID_ARG     # past t_cap
    assert rc_of(wb, s, FAKE, FAKE, 1, -1, FAKE, FAKE, 8, 0) == sp.SPARDA_ERR_INVALID_ARG
    assert rc_of(wb, s, FAKE, FAKE, 1, 100, FAKE, FAKE, 0, 0) == sp.SPARDA_ERR_INVALID_ARG      # n_workgroups
    assert rc_of(wb, s, None, FAKE, 1, 100, FAKE, FAKE, 8, 0) == sp.SPARDA_ERR_INVALID_ARG
    assert rc_of(wb, s, FAKE, FAKE, 1, 100, FAKE + 8, FAKE, 8, 0) == sp.SPARDA_ERR_INVALID_ARG  # alignment


def test_paper_grid_arguments(lib):
    """The (32, 16) grid: compress takes a window range, nc_cap counts windows, selection needs
    every window that overlaps a candidate block of the last row."""
    g = dict(cmp_kernel=32, cmp_stride=16)
    s = shape(nc_cap=255, **g)  # windows of a 4096-token cache: (4096 - 32) / 16 + 1
    c = sp.sparda_compress_keys
    assert rc_of(c, s, FAKE, 4096, 0, 256, FAKE, 0) == sp.SPARDA_ERR_INVALID_ARG      # > nc_cap
    assert rc_of(c, s, FAKE, 300, 0, 18, FAKE, 0) == sp.SPARDA_ERR_INVALID_ARG        # window 17 ends at 304
    assert rc_of(c, s, FAKE, 4096, 5, 4, FAKE, 0) == sp.SPARDA_ERR_INVALID_ARG        # reversed range
    c(s, FAKE, 4096, 7, 7, FAKE, 0)                                                   # empty: no-op
    f = sp.sparda_forecast_select
    # decode at p = 4095: candidates [1, 61]; block 61's last window is 4 * 61 + 3 = 247
    assert rc_of(f, shape(nc_cap=247, **g), FAKE, 1, 4095, FAKE, FAKE, FAKE, None, 0, 0) == \
        sp.SPARDA_ERR_INVALID_ARG
    assert sp.sparda_workspace_size(shape(nc_cap=248, **g), sp.SPARDA_OP_FORECAST_SELECT, 1, 4095) == 0  # fused
    # multi-row calls with at most 512 candidates per row take the fused tile kernel: no workspace
    assert sp.sparda_workspace_size(shape(nc_cap=255, **g), sp.SPARDA_OP_FORECAST_SELECT, 64, 4032) == 0
    # more candidates take the row-wise path: the last row (p = 40959, candidates [1, 637]) scores
    # windows 3 .. 2551
    big = shape(t_cap=65536, nc_cap=4095, **g)
    need = sp.sparda_workspace_size(big, sp.SPARDA_OP_FORECAST_SELECT, 64, 40896)
    assert need == 2 * 8 * 64 * 2552 * 4  # rows x stride(2549 -> 2552) x float
    assert rc_of(f, big, FAKE, 64, 40896, FAKE, FAKE, FAKE, FAKE, need - 4, 0) == sp.SPARDA_ERR_WORKSPACE
    # nc_cap may count up to four windows per block on this grid
    assert sp.sparda_workspace_size(shape(t_cap=131072, nc_cap=8191, batch=32, k_total=64, **g),
                                    sp.SPARDA_OP_FORECAST_SELECT, 1, 131071) == 0


def test_attention_argument_errors(lib):
    s = shape()
    a = sp.sparda_sparse_attn
    sc = 1 / math.sqrt(128)
    assert rc_of(a, s, FAKE, 1, 4095, FAKE, FAKE, 2, FAKE, FAKE, sc, FAKE, None, 0, 0) == sp.SPARDA_ERR_INVALID_ARG
    assert rc_of(a, s, FAKE, 2, 4094, FAKE, FAKE, 1, FAKE, FAKE, sc, FAKE, None, 0, 0) == sp.SPARDA_ERR_INVALID_ARG
    assert rc_of(a, s, FAKE, 1, 4095, FAKE, FAKE, 0, FAKE, FAKE, float("nan"), FAKE, None, 0, 0) == \
        sp.SPARDA_ERR_INVALID_ARG
    assert rc_of(a, s, None, 1, 4095, FAKE, FAKE, 0, FAKE, FAKE, sc, FAKE, None, 0, 0) == sp.SPARDA_ERR_INVALID_ARG
    assert rc_of(a, s, FAKE, 1, 4095, FAKE, FAKE, 0, FAKE, FAKE, sc, FAKE, None, 0, 0) == sp.SPARDA_ERR_WORKSPACE
    assert sp.sparda_workspace_size(s, sp.SPARDA_OP_SPARSE_ATTN, 1, 4095) > 0  # 16 rows: split


def test_attention_noalloc_argument_errors(lib):
    # the same validation as sparda_sparse_attn, before any HIP call; no workspace is needed
    s = shape()
    a = sp.sparda_sparse_attn_noalloc
    sc = 1 / math.sqrt(128)
    assert rc_of(a, s, FAKE, 1, 4095, FAKE, FAKE, 2, FAKE, FAKE, sc, FAKE, 0) == sp.SPARDA_ERR_INVALID_ARG
    assert rc_of(a, s, FAKE, 2, 4094, FAKE, FAKE, 1, FAKE, FAKE, sc, FAKE, 0) == sp.SPARDA_ERR_INVALID_ARG
    assert rc_of(a, s, None, 1, 4095, FAKE, FAKE, 0, FAKE, FAKE, sc, FAKE, 0) == sp.SPARDA_ERR_INVALID_ARG
    assert rc_of(a, shape(head_dim=64), FAKE, 1, 4095, FAKE, FAKE, 0, FAKE, FAKE, sc, FAKE, 0) == \
        sp.SPARDA_ERR_UNSUPPORTED
    # the largest split partials any call can need fit the static scratch: below 256 rows there are
    # at most ceil(256 / rows) splits per row, so rows x splits <= 511, at 16 heads of 130 floats
    worst = 0
    for rows in range(1, 256):
        s2 = shape(batch=rows, n_kv_heads=1, group_size=16, k_total=1024, t_cap=65536, nc_cap=1024)
        worst = max(worst, sp.sparda_workspace_size(s2, sp.SPARDA_OP_SPARSE_ATTN, 1, 65535))
    assert 0 < worst <= sp.SPARDA_NOALLOC_SCRATCH_BYTES
    assert worst == 510 * 16 * 130 * 4


def test_decode_step_argument_errors(lib):
    """The fused decode step validates both halves (select, then attention) before any HIP call,
    and its workspace is the larger of the two calls' workspaces."""
    s = shape()
    d = sp.sparda_decode_step
    sc = 1 / math.sqrt(128)
    # f, q_pos, k_cmp, q, k, v, sm_scale, sel, cnt, o, ws, ws_bytes, stream
    assert rc_of(d, s, None, 4095, FAKE, FAKE, FAKE, FAKE, sc, FAKE, FAKE, FAKE, None, 0, 0) == sp.SPARDA_ERR_INVALID_ARG
    assert rc_of(d, s, FAKE, 4096, FAKE, FAKE, FAKE, FAKE, sc, FAKE, FAKE, FAKE, None, 0, 0) == sp.SPARDA_ERR_INVALID_ARG
    assert rc_of(d, s, FAKE, 4095, FAKE, None, FAKE, FAKE, sc, FAKE, FAKE, FAKE, None, 0, 0) == sp.SPARDA_ERR_INVALID_ARG
    assert rc_of(d, s, FAKE, 4095, FAKE, FAKE, FAKE, FAKE, float("inf"), FAKE, FAKE, FAKE, None, 0, 0) == \
        sp.SPARDA_ERR_INVALID_ARG
    assert rc_of(d, s, FAKE, 4095, FAKE, FAKE, FAKE, FAKE, sc, FAKE, FAKE, None, None, 0, 0) == sp.SPARDA_ERR_INVALID_ARG
    # 16 rows: the attention splits its rows, so the step needs the attention's workspace beside
    # the selection's (256-byte aligned), since the fused kernel's workgroups read scores while
    # others write partials
    need = sp.sparda_workspace_size(s, sp.SPARDA_OP_DECODE_STEP, 1, 4095)
    sel_ws = sp.sparda_workspace_size(s, sp.SPARDA_OP_FORECAST_SELECT, 1, 4095)
    att_ws = sp.sparda_workspace_size(s, sp.SPARDA_OP_SPARSE_ATTN, 1, 4095)
    assert att_ws > 0 and need == -(-sel_ws // 256) * 256 + att_ws
    # 2 rows of 2045 windows: the split select path's scores and the attention's partials
    s2 = shape(batch=1, n_kv_heads=2, k_total=64, t_cap=131072, nc_cap=2048)
    sel_ws = sp.sparda_workspace_size(s2, sp.SPARDA_OP_FORECAST_SELECT, 1, 131071)
    att_ws = sp.sparda_workspace_size(s2, sp.SPARDA_OP_SPARSE_ATTN, 1, 131071)
    assert sel_ws > 0 and att_ws > 0
    assert sp.sparda_workspace_size(s2, sp.SPARDA_OP_DECODE_STEP, 1, 131071) == -(-sel_ws // 256) * 256 + att_ws
    assert rc_of(d, s, FAKE, 4095, FAKE, FAKE, FAKE, FAKE, sc, FAKE, FAKE, FAKE, None, 0, 0) == sp.SPARDA_ERR_WORKSPACE
    assert rc_of(d, s, FAKE, 4095, FAKE, FAKE, FAKE, FAKE, sc, FAKE, FAKE, FAKE, FAKE, need - 16, 0) == \
        sp.SPARDA_ERR_WORKSPACE
    # 128K, B32, 8 KV heads: both halves run one workgroup per row (the fused kernel): no workspace
    big = shape(batch=32, k_total=64, t_cap=131072, nc_cap=2048)
    assert sp.sparda_workspace_size(big, sp.SPARDA_OP_DECODE_STEP, 1, 131071) == 0
    assert rc_of(sp.sparda_workspace_size, big, sp.SPARDA_OP_DECODE_STEP, 2, 131070) == sp.SPARDA_ERR_INVALID_ARG


def test_stage_append_argument_errors(lib):
    s = shape()
    a = sp.sparda_stage_append_kv
    assert rc_of(a, s, FAKE, FAKE, 4096, FAKE, FAKE, FAKE, FAKE, 0) == sp.SPARDA_ERR_INVALID_ARG  # q_pos >= t_cap
    assert rc_of(a, s, FAKE, FAKE, -1, FAKE, FAKE, FAKE, FAKE, 0) == sp.SPARDA_ERR_INVALID_ARG
    assert rc_of(a, s, FAKE, None, 10, FAKE, FAKE, FAKE, FAKE, 0) == sp.SPARDA_ERR_INVALID_ARG
    assert rc_of(a, shape(block_size=32), FAKE, FAKE, 10, FAKE, FAKE, FAKE, FAKE, 0) == sp.SPARDA_ERR_UNSUPPORTED


def test_gather_argument_errors(lib):
    s = shape()
    g = sp.sparda_gather_blocks
    assert rc_of(g, s, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 0, 0) == sp.SPARDA_ERR_INVALID_ARG
    assert rc_of(g, s, None, FAKE, FAKE, FAKE, FAKE, FAKE, 8, 0) == sp.SPARDA_ERR_INVALID_ARG


def test_workspace_sizes(lib):
    # decode at 128K, B32: fused select (scores stay in LDS); 256 rows fill the chip, one split
    s2 = shape(batch=32, k_total=64, t_cap=131072, nc_cap=2048)
    assert sp.sparda_workspace_size(s2, sp.SPARDA_OP_FORECAST_SELECT, 1, 131071) == 0
    assert sp.sparda_workspace_size(s2, sp.SPARDA_OP_SPARSE_ATTN, 1, 131071) == 0
    # decode at 32K, B8: 64 rows -> 4 splits (about one workgroup per CU) x 4 heads x (128 + 2)
    # floats per row
    s1 = shape(batch=8, k_total=64, t_cap=32768, nc_cap=512)
    assert sp.sparda_workspace_size(s1, sp.SPARDA_OP_SPARSE_ATTN, 1, 32767) == 64 * 4 * 4 * 130 * 4
    # full 32K prefill: fused tiles, no score scratch; one split per row
    s3 = shape(batch=1, k_total=64, t_cap=32768, nc_cap=512)
    assert sp.sparda_workspace_size(s3, sp.SPARDA_OP_FORECAST_SELECT, 32768, 0) == 0
    assert sp.sparda_workspace_size(s3, sp.SPARDA_OP_SPARSE_ATTN, 32768, 0) == 0
    assert rc_of(sp.sparda_workspace_size, s3, 9, 1, 0) == sp.SPARDA_ERR_INVALID_ARG
    # a 20-row chunk of one group: the tiled kernel (G divides 16) needs no partials; with G = 3
    # the per-row kernel splits each row's block list over workgroups
    s4 = shape(batch=1, n_kv_heads=1, group_size=4, k_total=16, t_cap=8192, nc_cap=128)
    assert sp.sparda_workspace_size(s4, sp.SPARDA_OP_SPARSE_ATTN, 20, 4000) == 0
    s5 = shape(batch=1, n_kv_heads=1, group_size=3, k_total=16, t_cap=8192, nc_cap=128)
    assert sp.sparda_workspace_size(s5, sp.SPARDA_OP_SPARSE_ATTN, 20, 4000) > 0
    # a chunk past 4096 blocks (256K tokens) is beyond the tiles' LDS bitmaps: the per-row kernel
    s6 = shape(batch=1, n_kv_heads=1, group_size=4, k_total=16, t_cap=524288, nc_cap=8192)
    assert sp.sparda_workspace_size(s6, sp.SPARDA_OP_SPARSE_ATTN, 20, 524000) > 0
    assert sp.sparda_workspace_size(s6, sp.SPARDA_OP_SPARSE_ATTN, 20, 200000) == 0


def test_multihead_select_arguments(lib):
    """The InfLLM-V2 multi-head selector: the softmax of every head runs over every compressed key
    complete at the last row's position, so nc_cap must reach that key; the temperature must be a
    positive number; decode with G in {1, 2, 4, 8} is fused (no workspace), other calls keep every
    head's window scores plus the shared scores per row."""
    m = sp.sparda_multihead_select
    sc = 1 / math.sqrt(128)
    s = shape(nc_cap=64)  # blocks 0 .. 63 of a 4096-token cache
    assert rc_of(m, shape(nc_cap=63), FAKE, 1, 4095, FAKE, sc, FAKE, FAKE, None, 0, 0) == sp.SPARDA_ERR_INVALID_ARG
    for bad in (0.0, -1.0, float("nan"), float("inf")):
        assert rc_of(m, s, FAKE, 1, 4095, FAKE, bad, FAKE, FAKE, None, 0, 0) == sp.SPARDA_ERR_INVALID_ARG
    assert rc_of(m, s, None, 1, 4095, FAKE, sc, FAKE, FAKE, None, 0, 0) == sp.SPARDA_ERR_INVALID_ARG
    op = sp.SPARDA_OP_MULTIHEAD_SELECT
    assert sp.sparda_workspace_size(s, op, 1, 4095) == 0  # fused decode
    # 128K decode on the (32, 16) grid: 4 x 8191 window scores + 2045 block scores fit in LDS
    g = shape(batch=32, k_total=64, t_cap=131072, nc_cap=8191, cmp_kernel=32, cmp_stride=16)
    assert sp.sparda_workspace_size(g, op, 1, 131071) == 0
    # G = 16 there, and G = 3: the two-pass fused kernel keeps only the shared scores in LDS
    g16 = shape(batch=32, n_kv_heads=2, group_size=16, k_total=64, t_cap=131072, nc_cap=8191, cmp_kernel=32,
                cmp_stride=16)
    assert sp.sparda_workspace_size(g16, op, 1, 131071) == 0
    assert sp.sparda_workspace_size(shape(group_size=3), op, 1, 4095) == 0
    # 512K tokens on the (32, 16) grid: 32767 windows + 8189 candidates exceed LDS: row-wise decode,
    # (4 + 1) x 32768 floats per row
    big = shape(batch=1, n_kv_heads=2, t_cap=524288, nc_cap=32767, k_total=64, cmp_kernel=32, cmp_stride=16)
    assert sp.sparda_workspace_size(big, op, 1, 524287) == 2 * 5 * 32768 * 4
    # multi-row: the last row (p = 4095) has 64 complete blocks
    need = sp.sparda_workspace_size(s, op, 100, 3996)
    assert need == 2 * 8 * 100 * 5 * 64 * 4
    assert rc_of(m, s, FAKE, 100, 3996, FAKE, sc, FAKE, FAKE, FAKE, need - 4, 0) == sp.SPARDA_ERR_WORKSPACE
    # rows that take every candidate need no scores
    assert sp.sparda_workspace_size(shape(k_total=64), op, 100, 3996) == 0


def test_plan_staging_arguments(lib):
    pl = sp.sparda_plan_staging
    s = shape()
    assert rc_of(pl, s, FAKE, FAKE, 4096, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 0) == sp.SPARDA_ERR_INVALID_ARG  # q_pos
    assert rc_of(pl, s, FAKE, FAKE, -1, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 0) == sp.SPARDA_ERR_INVALID_ARG
    assert rc_of(pl, s, FAKE, FAKE, 100, None, FAKE, FAKE, FAKE, FAKE, FAKE, 0) == sp.SPARDA_ERR_INVALID_ARG
    assert rc_of(pl, s, FAKE, FAKE, 100, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE + 2, 0) == sp.SPARDA_ERR_INVALID_ARG
    big = shape(k_total=1025, t_cap=131072, nc_cap=2048)
    assert rc_of(pl, big, FAKE, FAKE, 100, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 0) == sp.SPARDA_ERR_UNSUPPORTED


def test_status_strings(lib):
    assert sp.status_string(0) == "SPARDA_OK"
    assert sp.status_string(-4) == "SPARDA_ERR_HOST_NOT_MAPPED"
    assert sp.status_string(-99) == "SPARDA_ERR_UNKNOWN"


def test_indexer_kl_arguments(lib):
    kl = sp.sparda_indexer_kl
    sc = 1 / math.sqrt(128)
    g = dict(cmp_kernel=32, cmp_stride=16)
    s = shape(nc_cap=255, **g)
    args = lambda **kw: [kw.get("s", s), FAKE, FAKE, FAKE, FAKE, kw.get("n_q", 4), kw.get("q0", 4000), kw.get("sc", sc),
                         kw.get("k", 8), FAKE, FAKE, kw.get("ws", FAKE), kw.get("wsb", 1 << 40), 0]
    assert rc_of(kl, *args(sc=0.0)) == sp.SPARDA_ERR_INVALID_ARG
    assert rc_of(kl, *args(k=-1)) == sp.SPARDA_ERR_INVALID_ARG
    assert rc_of(kl, *args(k=4097)) == sp.SPARDA_ERR_INVALID_ARG
    assert rc_of(kl, *args(q0=10, n_q=4)) == sp.SPARDA_ERR_INVALID_ARG      # row 0 has no complete window
    assert rc_of(kl, *args(s=shape(nc_cap=200, **g))) == sp.SPARDA_ERR_INVALID_ARG  # window 248 beyond nc_cap
    need = sp.sparda_workspace_size(s, sp.SPARDA_OP_INDEXER_KL, 4, 4000)
    # the fine windows complete at the last row (p = 4003), then each row's weight of each of them
    assert need == 2 * 8 * 4003 * 128 * 2 + 2 * 8 * 4 * 4004 * 4
    assert rc_of(kl, *args(ws=None)) == sp.SPARDA_ERR_WORKSPACE
    assert rc_of(kl, *args(wsb=need - 2)) == sp.SPARDA_ERR_WORKSPACE
