"""GPU test of sparda_sparse_attn_noalloc: the attention variant that takes no workspace and keeps
its split partials in the library's static per-device scratch array.

Its output must equal sparda_sparse_attn's (same kernels, same inputs: bitwise), and both must
match the oracle within the attention bar.  Two calls in a row, the second with fewer rows and
fewer splits, check that the array's leftover contents from the first call do not leak into the
second.  A third call with 256 rows (no partials) and a G = 16 call cover the other launch shapes.
"""
import math
import sys

import numpy as np
import pytest
import torch

import oracle
import paper_2606_04511_amd.sparda as sp
from paper_2606_04511_amd import inputs
from parity import abs_bits, compare_attention

pytestmark = pytest.mark.gpu
SCALE = 1.0 / math.sqrt(128)


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def run_case(dev, B, H, G, T, k_total, seed, n_local=2):
    say(f"noalloc attention B{B} H{H} G{G} T{T} k{k_total}")
    w = inputs.Workload("noalloc", batch=B, seq_len=T, n_q=1, n_kv_heads=H, group_size=G, k_total=k_total,
                        n_local=n_local, seed=seed)
    case = inputs.make_case(w)
    nb = T // 64
    s = sp.SpardaShape(batch=B, n_kv_heads=H, group_size=G, k_total=k_total, t_cap=T, nc_cap=nb, n_local=n_local)
    o = oracle.Shape(batch=B, n_kv_heads=H, group_size=G, k_total=k_total, t_cap=T, nc_cap=nb, n_local=n_local)
    k16, v16, q16 = inputs.to_u16(case["k"]), inputs.to_u16(case["v"]), inputs.to_u16(case["q"])
    kc_ref = oracle.compress_keys(o, k16, T, 0, nb)
    sel, cnt = oracle.forecast_select(o, inputs.to_u16(case["f"]), 1, T - 1, kc_ref)
    q, k, v = case["q"].to(dev), case["k"].to(dev), case["v"].to(dev)
    sel_d, cnt_d = torch.from_numpy(sel).to(dev), torch.from_numpy(cnt).to(dev)
    need = sp.sparda_workspace_size(s, sp.SPARDA_OP_SPARSE_ATTN, 1, T - 1)
    out_ws = torch.full((B, H * G, 1, 128), float("nan"), dtype=torch.bfloat16, device=dev)
    sp.sparda_sparse_attn(s, q, 1, T - 1, k, v, 0, sel_d, cnt_d, SCALE, out_ws,
                          torch.empty(max(need, 16), dtype=torch.uint8, device=dev))
    out_na = torch.full_like(out_ws, float("nan"))
    sp.sparda_sparse_attn_noalloc(s, q, 1, T - 1, k, v, 0, sel_d, cnt_d, SCALE, out_na)
    torch.cuda.synchronize()
    a = inputs.to_u16(out_ws)
    b = inputs.to_u16(out_na)
    assert np.array_equal(a, b), f"noalloc output differs from the workspace call in {int((a != b).sum())} values"
    ref = oracle.sparse_attn(o, q16, 1, T - 1, k16, v16, 0, sel, cnt, SCALE)
    wab = oracle.sparse_attn(o, q16, 1, T - 1, k16, abs_bits(v16), 0, sel, cnt, SCALE)
    worst = compare_attention(out_na.float().cpu().numpy(), ref, "noalloc attention", wab)
    say(f"  partials {need} bytes, bitwise equal to the workspace call, max |o - oracle| {worst:.3g}")
    return need


def test_noalloc_matches_workspace_call_twice_then_smaller():
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a GPU")
    sp.load()
    dev = torch.device("cuda:0")
    first = run_case(dev, 8, 8, 4, 32768, 64, 7100)   # 64 rows, 4 splits per row
    second = run_case(dev, 1, 8, 4, 4096, 16, 7101)   # 8 rows, 2 splits: a smaller input
    assert 0 < second < first
    assert run_case(dev, 32, 8, 4, 8192, 64, 7102) == 0  # 256 rows: no partials, scratch unused
    assert run_case(dev, 2, 2, 16, 16384, 96, 7103, n_local=32) > 0  # G = 16 (the wide kernel)
