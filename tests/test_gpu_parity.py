"""GPU parity: the HIP library (through the C ABI) against the CPU oracle on the same seeded inputs.

Every test is marked `gpu`.  Inputs come from paper_2606_04511_amd.inputs; expected values come
only from the oracle.  Attention is always checked on the oracle's attended sets, uploaded to the
GPU.  Small cases compare every output; the full-size workloads compare sampled rows.
"""
import math
import os
import sys

import numpy as np
import pytest
import torch

import oracle
import paper_2606_04511_amd.sparda as sp
from paper_2606_04511_amd import hostmem, inputs
from parity import abs_bits, compare_attention, compare_multihead_selection, compare_selection

pytestmark = pytest.mark.gpu
SCALE = 1.0 / math.sqrt(128)


@pytest.fixture(scope="module")
def dev():
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a GPU")
    sp.load()  # the in-tree libsparda.so; there is no fallback
    return torch.device("cuda:0")


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def shapes(B, H, G, k_total, t_cap, nc_cap, n_init=1, n_local=2, lw=64, sw=64):
    s = sp.SpardaShape(batch=B, n_kv_heads=H, group_size=G, k_total=k_total, t_cap=t_cap, nc_cap=nc_cap,
                       n_init=n_init, n_local=n_local, cmp_kernel=lw, cmp_stride=sw)
    o = oracle.Shape(batch=B, n_kv_heads=H, group_size=G, k_total=k_total, t_cap=t_cap, nc_cap=nc_cap,
                     n_init=n_init, n_local=n_local, cmp_kernel=lw, cmp_stride=sw)
    return s, o


def ws(shape, op, n_q, q_pos0, dev):
    n = sp.sparda_workspace_size(shape, op, n_q, q_pos0)
    return torch.empty(max(n, 16), dtype=torch.uint8, device=dev)


def gpu_compress(s, k_dev, t_ctx, nb, nc_cap, dev):
    kc = torch.zeros(s.batch, s.n_kv_heads, nc_cap, 128, dtype=torch.bfloat16, device=dev)
    sp.sparda_compress_keys(s, k_dev, t_ctx, 0, nb, kc)
    return kc


def gpu_select(s, f_dev, n_q, q_pos0, kc_dev, dev):
    sel = torch.full((s.batch, s.n_kv_heads, n_q, s.k_total), 777, dtype=torch.int16, device=dev)
    cnt = torch.full((s.batch, s.n_kv_heads, n_q), 777, dtype=torch.int16, device=dev)
    sp.sparda_forecast_select(s, f_dev, n_q, q_pos0, kc_dev, sel, cnt, ws(s, sp.SPARDA_OP_FORECAST_SELECT, n_q,
                                                                          q_pos0, dev))
    torch.cuda.synchronize()
    # every row's count is written (777 exceeds every k_total here): no slice or unit is skipped,
    # whichever rows the comparisons sample
    assert not bool((cnt == 777).any()), f"{int((cnt == 777).sum())} rows left without a selection"
    return sel, cnt


def gpu_attend(s, q_dev, n_q, q_pos0, k_dev, v_dev, kv_mode, sel_dev, cnt_dev, dev):
    o = torch.full((s.batch, s.n_q_heads, n_q, 128), float("nan"), dtype=torch.bfloat16, device=dev)
    sp.sparda_sparse_attn(s, q_dev, n_q, q_pos0, k_dev, v_dev, kv_mode, sel_dev, cnt_dev, SCALE, o,
                          ws(s, sp.SPARDA_OP_SPARSE_ATTN, n_q, q_pos0, dev))
    torch.cuda.synchronize()
    # every output row is written (it starts as NaN, and finite inputs give finite outputs),
    # whichever rows the oracle comparisons sample
    assert not bool(torch.isnan(o).any()), f"{int(torch.isnan(o).sum())} output elements left unwritten"
    return o


def gpu_step(s, f_dev, q_pos, kc_dev, q_dev, k_dev, v_dev, dev):
    """sparda_decode_step: the sets and the attention output of one decode step."""
    sel = torch.full((s.batch, s.n_kv_heads, 1, s.k_total), 777, dtype=torch.int16, device=dev)
    cnt = torch.full((s.batch, s.n_kv_heads, 1), 777, dtype=torch.int16, device=dev)
    o = torch.full((s.batch, s.n_q_heads, 1, 128), float("nan"), dtype=torch.bfloat16, device=dev)
    sp.sparda_decode_step(s, f_dev, q_pos, kc_dev, q_dev, k_dev, v_dev, SCALE, sel, cnt, o,
                          ws(s, sp.SPARDA_OP_DECODE_STEP, 1, q_pos, dev))
    torch.cuda.synchronize()
    return sel, cnt, o


def make(B, H, G, T, n_q, k_total, seed, t_cap=None, n_init=1, n_local=2):
    w = inputs.Workload("t", batch=B, seq_len=T, n_q=n_q, n_kv_heads=H, group_size=G, k_total=k_total,
                        n_init=n_init, n_local=n_local, seed=seed)
    t_cap = -(-T // 64) * 64 if t_cap is None else t_cap
    return w, inputs.make_case(w, t_cap=t_cap)


# ----------------------------------------------------------------------------- compress

@pytest.mark.parametrize("B,H,T,t_cap", [(1, 8, 4096, 4096), (2, 2, 1000, 1024), (3, 1, 64, 128), (2, 3, 8192, 8192)])
def test_compress_bitwise(dev, B, H, T, t_cap):
    say(f"compress B{B} H{H} T{T}")
    w, case = make(B, H, 4, T, 1, 8, 2000 + T, t_cap=t_cap)
    nb = T // 64
    s, o = shapes(B, H, 4, 8, t_cap, max(nb, 1))
    kc = gpu_compress(s, case["k"].to(dev), T, nb, max(nb, 1), dev)
    torch.cuda.synchronize()
    ref = oracle.compress_keys(o, inputs.to_u16(case["k"]), T, 0, nb)
    assert np.array_equal(inputs.to_u16(kc), ref)


def test_compress_incremental_equals_full(dev):
    say("compress incremental")
    w, case = make(2, 2, 4, 2048, 1, 8, 2100)
    s, _ = shapes(2, 2, 4, 8, 2048, 32)
    k = case["k"].to(dev)
    full = gpu_compress(s, k, 2048, 32, 32, dev)
    inc = torch.zeros_like(full)
    for t in range(64, 2049, 64):
        sp.sparda_compress_keys(s, k, t, t // 64 - 1, t // 64, inc)
    torch.cuda.synchronize()
    assert torch.equal(full.view(torch.int16), inc.view(torch.int16))


# ----------------------------------------------------------------------------- selection

DECODE_SELECT = [
    # B, H, G, T, k_total, n_init, n_local
    (1, 8, 4, 4096, 16, 1, 2),
    (2, 2, 4, 65, 3, 1, 2),
    (2, 8, 4, 1000, 5, 1, 2),
    (3, 2, 4, 8192, 64, 1, 2),
    (1, 4, 1, 32768, 64, 1, 2),
    (1, 2, 4, 131072, 64, 1, 2),
    (2, 2, 4, 20000, 40, 0, 3),
    (1, 2, 16, 50000, 96, 1, 32),
    (1, 2, 4, 600000, 64, 1, 2),  # 9372 candidates: 5 chunks of the workgroup top-k
]


@pytest.mark.parametrize("B,H,G,T,k_total,n_init,n_local", DECODE_SELECT)
def test_decode_select(dev, B, H, G, T, k_total, n_init, n_local):
    say(f"decode select B{B} H{H} T{T} k{k_total} init{n_init} local{n_local}")
    w, case = make(B, H, G, T, 1, k_total, 3000 + T, n_init=n_init, n_local=n_local)
    nb = T // 64
    s, o = shapes(B, H, G, k_total, case["t_cap"], max(nb, 1), n_init, n_local)
    kc_ref = oracle.compress_keys(o, inputs.to_u16(case["k"]), T, 0, nb)
    kc_dev = inputs.from_u16(kc_ref, dev)  # the oracle's K~ as input: this test isolates selection
    sel, cnt = gpu_select(s, case["f"].to(dev), 1, T - 1, kc_dev, dev)
    rows = [(b, m, 0) for b in range(B) for m in range(H)]
    n, swaps = compare_selection(o, inputs.to_u16(case["f"]), kc_ref, 1, T - 1, sel.cpu().numpy(), cnt.cpu().numpy(),
                                 rows)
    say(f"  rows {n}, tie swaps {swaps}")


PREFILL_SELECT = [
    # B, H, T, n_q, q_pos0, k_total   (rows at positions q_pos0 .. q_pos0 + n_q - 1)
    (1, 2, 4096, 4096, 0, 16),
    (2, 1, 5000, 5000, 0, 8),
    (1, 2, 8192, 700, 3000, 64),
    (1, 1, 32768, 2048, 30720, 64),
    (1, 1, 40000, 37, 39963, 64),  # > 512 candidates per row: row-wise path, MFMA window scores
    (2, 2, 70000, 300, 69650, 64),  # 1089 candidates, 300 rows over 6 blocks: ragged first and last units
    (1, 1, 40000, 9, 39990, 64),  # fewer rows than the MFMA scorer takes: the per-row score kernel
]


@pytest.mark.parametrize("B,H,T,n_q,q_pos0,k_total", PREFILL_SELECT)
def test_prefill_select(dev, B, H, T, n_q, q_pos0, k_total):
    say(f"prefill select B{B} H{H} T{T} n_q{n_q} q_pos0 {q_pos0} k{k_total}")
    w, case = make(B, H, 4, T, n_q, k_total, 4000 + T)
    t_cap = -(-T // 64) * 64
    nb = T // 64
    s, o = shapes(B, H, 4, k_total, t_cap, max(nb, 1))
    kc_ref = oracle.compress_keys(o, inputs.to_u16(case["k"]), T, 0, nb)
    f_u16 = inputs.to_u16(case["f"])
    sel, cnt = gpu_select(s, case["f"].to(dev), n_q, q_pos0, inputs.from_u16(kc_ref, dev), dev)
    rng = np.random.default_rng(0)
    rr = sorted(set(rng.integers(0, n_q, size=min(n_q, 600)).tolist()) | {0, n_q - 1})
    rows = [(b, m, r) for b in range(B) for m in range(H) for r in rr]
    n, swaps = compare_selection(o, f_u16, kc_ref, n_q, q_pos0, sel.cpu().numpy(), cnt.cpu().numpy(), rows)
    say(f"  rows {n}, tie swaps {swaps}")


PREFILL_SELECT_WINDOWS = [
    # B, H, T, n_q, q_pos0, k_total, n_init, n_local
    (1, 1, 20000, 1000, 18991, 100, 1, 2),  # odd start, larger budget, a single group
    (3, 1, 2000, 2000, 0, 4, 1, 2),  # one chosen block per row
    (1, 2, 9000, 9000, 0, 40, 0, 3),  # no initial block
    (1, 1, 30000, 3000, 27000, 64, 4, 16),  # 4 initial blocks, a 16-block local window
    (1, 1, 2048, 2048, 0, 20, 1, 1),  # few candidates: lane groups past the last candidate
]


@pytest.mark.parametrize("B,H,T,n_q,q_pos0,k_total,n_init,n_local", PREFILL_SELECT_WINDOWS)
def test_prefill_select_windows(dev, B, H, T, n_q, q_pos0, k_total, n_init, n_local):
    say(f"prefill select B{B} H{H} T{T} n_q{n_q} q_pos0 {q_pos0} k{k_total} init {n_init} local {n_local}")
    w, case = make(B, H, 4, T, n_q, k_total, 4500 + T, n_init=n_init, n_local=n_local)
    t_cap = -(-T // 64) * 64
    nb = T // 64
    s, o = shapes(B, H, 4, k_total, t_cap, max(nb, 1), n_init=n_init, n_local=n_local)
    kc_ref = oracle.compress_keys(o, inputs.to_u16(case["k"]), T, 0, nb)
    f_u16 = inputs.to_u16(case["f"])
    sel, cnt = gpu_select(s, case["f"].to(dev), n_q, q_pos0, inputs.from_u16(kc_ref, dev), dev)
    rng = np.random.default_rng(1)
    rr = sorted(set(rng.integers(0, n_q, size=min(n_q, 500)).tolist()) | {0, n_q - 1})
    rows = [(b, m, r) for b in range(B) for m in range(H) for r in rr]
    n, swaps = compare_selection(o, f_u16, kc_ref, n_q, q_pos0, sel.cpu().numpy(), cnt.cpu().numpy(), rows)
    say(f"  rows {n}, tie swaps {swaps}")


def test_select_is_deterministic(dev):
    say("select determinism")
    w, case = make(1, 2, 4, 32768, 32768, 64, 4100)
    s, o = shapes(1, 2, 4, 64, 32768, 512)
    kc = gpu_compress(s, case["k"].to(dev), 32768, 512, 512, dev)
    f = case["f"].to(dev)
    a, ca = gpu_select(s, f, 32768, 0, kc, dev)
    b, cb = gpu_select(s, f, 32768, 0, kc, dev)
    assert torch.equal(a, b) and torch.equal(ca, cb)


# ----------------------------------------------------------------------------- attention

ATTN = [
    # B, H, G, T, n_q, k_total
    (1, 8, 4, 4096, 1, 16),
    (2, 2, 4, 1000, 1, 5),
    (2, 2, 4, 32768, 1, 64),
    (1, 2, 1, 8192, 1, 32),
    (1, 2, 8, 8192, 1, 32),
    (1, 1, 16, 8192, 1, 32),
    (1, 1, 4, 77, 1, 3),
    (1, 2, 5, 8192, 1, 32),
    (1, 2, 6, 8192, 1, 32),
    (1, 1, 12, 8192, 1, 32),
    (1, 2, 4, 640, 640, 4),
    (1, 1, 4, 8192, 300, 16),
    # multi-row calls on the tiled kernel (256/G rows per tile): every G it takes, ragged last
    # tiles, chunks that start off a block boundary, the 16-row threshold, one block only
    (1, 2, 1, 4096, 600, 16),
    (1, 2, 2, 2048, 2048, 8),
    (2, 1, 8, 3000, 130, 16),
    (1, 1, 16, 1024, 40, 6),
    (1, 1, 4, 64, 64, 3),
    (1, 2, 4, 5000, 16, 16),
    (1, 2, 4, 20000, 700, 64),
    # multi-row, G does not divide 16: the per-row kernels (VALU P V at 3 heads, MFMA at 6)
    (1, 2, 3, 2048, 100, 8),
    (1, 2, 6, 2048, 100, 8),
]


@pytest.mark.parametrize("B,H,G,T,n_q,k_total", ATTN)
def test_attention_on_oracle_sets(dev, B, H, G, T, n_q, k_total):
    say(f"attention B{B} H{H} G{G} T{T} n_q{n_q} k{k_total}")
    w, case = make(B, H, G, T, n_q, k_total, 5000 + T + G)
    t_cap = -(-T // 64) * 64
    nb = max(T // 64, 1)
    s, o = shapes(B, H, G, k_total, t_cap, nb)
    q_pos0 = T - n_q
    k16, v16, q16 = inputs.to_u16(case["k"]), inputs.to_u16(case["v"]), inputs.to_u16(case["q"])
    kc_ref = oracle.compress_keys(o, k16, T, 0, T // 64)
    sel, cnt = oracle.forecast_select(o, inputs.to_u16(case["f"]), n_q, q_pos0, kc_ref)
    out = gpu_attend(s, case["q"].to(dev), n_q, q_pos0, case["k"].to(dev), case["v"].to(dev), 0,
                     torch.from_numpy(sel).to(dev), torch.from_numpy(cnt).to(dev), dev)
    ref = oracle.sparse_attn(o, q16, n_q, q_pos0, k16, v16, 0, sel, cnt, SCALE)
    wab = oracle.sparse_attn(o, q16, n_q, q_pos0, k16, abs_bits(v16), 0, sel, cnt, SCALE)
    worst = compare_attention(out.float().cpu().numpy(), ref, "attention", wab)
    say(f"  max err {worst:.3g} ({compare_attention.last_tight_ratio:.3f} of the tight bar)")


def test_attention_staging_mode(dev):
    say("attention staging mode")
    B, H, G, T, k_total = 2, 2, 4, 8192, 16
    w, case = make(B, H, G, T, 1, k_total, 5100)
    s, o = shapes(B, H, G, k_total, T, T // 64)
    k16, v16 = inputs.to_u16(case["k"]), inputs.to_u16(case["v"])
    kc_ref = oracle.compress_keys(o, k16, T, 0, T // 64)
    sel, cnt = oracle.forecast_select(o, inputs.to_u16(case["f"]), 1, T - 1, kc_ref)
    st_k, st_v = oracle.gather_blocks(o, k16, v16, sel[:, :, 0], cnt[:, :, 0])
    out = gpu_attend(s, case["q"].to(dev), 1, T - 1, inputs.from_u16(st_k, dev), inputs.from_u16(st_v, dev), 1,
                     torch.from_numpy(sel).to(dev), torch.from_numpy(cnt).to(dev), dev)
    ref = oracle.sparse_attn(o, inputs.to_u16(case["q"]), 1, T - 1, k16, v16, 0, sel, cnt, SCALE)
    wab = oracle.sparse_attn(o, inputs.to_u16(case["q"]), 1, T - 1, k16, abs_bits(v16), 0, sel, cnt, SCALE)
    compare_attention(out.float().cpu().numpy(), ref, "staging", wab)


def test_attention_order_invariance_and_skips(dev):
    say("attention order invariance")
    B, H, G, T, k_total = 2, 2, 4, 8192, 16
    w, case = make(B, H, G, T, 1, k_total, 5200)
    s, o = shapes(B, H, G, k_total, T, T // 64)
    k16 = inputs.to_u16(case["k"])
    kc_ref = oracle.compress_keys(o, k16, T, 0, T // 64)
    sel, cnt = oracle.forecast_select(o, inputs.to_u16(case["f"]), 1, T - 1, kc_ref)
    rng = np.random.default_rng(1)
    perm = sel.copy()
    for b in range(B):
        for m in range(H):
            perm[b, m, 0, :cnt[b, m, 0]] = rng.permutation(perm[b, m, 0, :cnt[b, m, 0]])
    args = (case["q"].to(dev), 1, T - 1, case["k"].to(dev), case["v"].to(dev), 0)
    a = gpu_attend(s, *args, torch.from_numpy(sel).to(dev), torch.from_numpy(cnt).to(dev), dev)
    b_ = gpu_attend(s, *args, torch.from_numpy(perm).to(dev), torch.from_numpy(cnt).to(dev), dev)
    assert (a.float() - b_.float()).abs().max().item() <= 2e-2
    # entries outside [0, blk(p)] are skipped
    s2, o2 = shapes(B, H, G, k_total + 2, T, T // 64)
    sel2 = np.concatenate([sel, np.array([-3, 30000], np.int16)[None, None, None].repeat(B, 0).repeat(H, 1)], axis=-1)
    c = gpu_attend(s2, *args, torch.from_numpy(np.ascontiguousarray(sel2)).to(dev),
                   torch.from_numpy(cnt + 2).to(dev), dev)
    assert (a.float() - c.float()).abs().max().item() <= 2e-2


@pytest.mark.parametrize("n_q", [1, 200])
def test_attention_duplicate_entries_attended_once(dev, n_q):
    say(f"attention duplicates n_q={n_q}")
    B, H, G, T, k_total = 1, 2, 4, 6144, 12
    extra = 4
    w, case = make(B, H, G, T, n_q, k_total, 5250 + n_q)
    s, o = shapes(B, H, G, k_total, T, T // 64)
    q_pos0 = T - n_q
    k16, v16 = inputs.to_u16(case["k"]), inputs.to_u16(case["v"])
    kc_ref = oracle.compress_keys(o, k16, T, 0, T // 64)
    sel, cnt = oracle.forecast_select(o, inputs.to_u16(case["f"]), n_q, q_pos0, kc_ref)
    rng = np.random.default_rng(11)
    dup = np.concatenate([sel, sel[..., :extra]], axis=-1)
    dup = np.ascontiguousarray(np.take_along_axis(dup, rng.permuted(
        np.tile(np.arange(dup.shape[-1]), dup.shape[:-1] + (1,)), axis=-1), axis=-1))
    s2, o2 = shapes(B, H, G, k_total + extra, T, T // 64)
    cnt2 = np.full(cnt.shape, k_total + extra, np.int16)
    out = gpu_attend(s2, case["q"].to(dev), n_q, q_pos0, case["k"].to(dev), case["v"].to(dev), 0,
                     torch.from_numpy(dup).to(dev), torch.from_numpy(cnt2).to(dev), dev)
    ref = oracle.sparse_attn(o, inputs.to_u16(case["q"]), n_q, q_pos0, k16, v16, 0, sel, cnt, SCALE)
    wab = oracle.sparse_attn(o, inputs.to_u16(case["q"]), n_q, q_pos0, k16, abs_bits(v16), 0, sel, cnt, SCALE)
    compare_attention(out.float().cpu().numpy(), ref, "duplicates", wab)


# ----------------------------------------------------------------------------- gather

def test_gather_bitwise_and_host_checks(dev):
    say("gather")
    B, H, G, T, k_total = 2, 2, 4, 8192, 16
    w, case = make(B, H, G, T, 1, k_total, 5300)
    s, o = shapes(B, H, G, k_total, T, T // 64)
    k16, v16 = inputs.to_u16(case["k"]), inputs.to_u16(case["v"])
    kc_ref = oracle.compress_keys(o, k16, T, 0, T // 64)
    sel, cnt = oracle.forecast_select(o, inputs.to_u16(case["f"]), 1, T - 1, kc_ref)
    hk = case["k"].pin_memory()
    hv = case["v"].pin_memory()
    ref_k, ref_v = oracle.gather_blocks(o, k16, v16, sel[:, :, 0], cnt[:, :, 0])
    sel_d = torch.from_numpy(np.ascontiguousarray(sel[:, :, 0])).to(dev)
    cnt_d = torch.from_numpy(np.ascontiguousarray(cnt[:, :, 0])).to(dev)
    for nwg in (1, 7, 64):
        st_k = torch.zeros(B, H, k_total, 64, 128, dtype=torch.bfloat16, device=dev)
        st_v = torch.zeros_like(st_k)
        side = torch.cuda.Stream()
        sp.sparda_gather_blocks(s, hk, hv, sel_d, cnt_d, st_k, st_v, nwg, side)
        side.synchronize()
        assert np.array_equal(inputs.to_u16(st_k), ref_k) and np.array_equal(inputs.to_u16(st_v), ref_v)
    with pytest.raises(sp.SpardaError) as ei:
        sp.sparda_gather_blocks(s, case["k"], case["v"], sel_d, cnt_d, st_k, st_v, 8)  # pageable memory
    assert ei.value.status == sp.SPARDA_ERR_HOST_NOT_MAPPED
    # pools shorter than the [B][Hkv][t_cap][D] layout are refused before any launch: one 16-byte
    # piece short, and a pointer 4 KiB into an allocation of exactly the layout's size
    need = B * H * T * 128 * 2
    short = hostmem.PinnedBuffer(need - 16)
    exact = hostmem.PinnedBuffer(need)
    for hk_bad, hv_ok in ((short.ptr, hv), (hk, short.ptr), (exact.ptr + 4096, hv)):
        with pytest.raises(sp.SpardaError) as ei:
            sp.sparda_gather_blocks(s, hk_bad, hv_ok, sel_d, cnt_d, st_k, st_v, 8)
        assert ei.value.status == sp.SPARDA_ERR_INVALID_ARG, ei.value
    with pytest.raises(sp.SpardaError) as ei:
        sp.sparda_writeback_kv(s, st_k, st_v, 1, T - 1, short.ptr, hv, 8)
    assert ei.value.status == sp.SPARDA_ERR_INVALID_ARG
    sp.sparda_gather_blocks(s, exact.ptr, hv, sel_d, cnt_d, st_k, st_v, 8)  # exactly the layout: accepted
    torch.cuda.synchronize()
    short.free()
    exact.free()


@pytest.mark.parametrize("K,p", [(16, 4095), (64, 3000), (100, 64 * 70)])
def test_stage_append_bitwise(dev, K, p):
    """The decoded token into the staged copy of its own block, bitwise against the oracle: rows
    listing the block once, twice (k > 64: the second listing past entry 64), or not at all, and a
    row whose count leaves it out; every other staged byte unchanged."""
    say(f"stage append K{K} p{p}")
    B, H, T = 3, 2, 8192
    s, o = shapes(B, H, 4, K, T, T // 64)
    rng = np.random.default_rng(K + p)
    j = p // 64
    sel = np.full((B, H, K), -1, np.int16)
    cnt = np.zeros((B, H), np.int16)
    for b in range(B):
        for m in range(H):
            n = int(rng.integers(1, K + 1))
            blocks = rng.choice(j + 1, size=n, replace=n > j + 1).astype(np.int16)
            case = (b * H + m) % 4
            if case == 1:
                blocks[int(rng.integers(n))] = j
            elif case == 2 and n >= 2:
                blocks[0] = j
                blocks[n - 1] = j
            elif case == 3:
                blocks[blocks == j] = max(j - 1, 0)
            sel[b, m, :n] = blocks
            cnt[b, m] = n
    sel[0, 0, :] = j  # every slot holds the block, but the count covers only the first three
    cnt[0, 0] = 3
    stage_k = rng.integers(0, 0x7F00, size=(B, H, K, 64, 128), dtype=np.uint16)
    stage_v = rng.integers(0, 0x7F00, size=(B, H, K, 64, 128), dtype=np.uint16)
    k_new = rng.integers(0, 0x7F00, size=(B, H, 128), dtype=np.uint16)
    v_new = rng.integers(0, 0x7F00, size=(B, H, 128), dtype=np.uint16)
    want_k, want_v = oracle.stage_append_kv(o, k_new, v_new, p, sel, cnt, stage_k, stage_v)
    sk, sv = inputs.from_u16(stage_k, dev), inputs.from_u16(stage_v, dev)
    sp.sparda_stage_append_kv(s, inputs.from_u16(k_new, dev), inputs.from_u16(v_new, dev), p,
                              torch.from_numpy(sel).to(dev), torch.from_numpy(cnt).to(dev), sk, sv)
    torch.cuda.synchronize()
    assert np.array_equal(inputs.to_u16(sk), want_k) and np.array_equal(inputs.to_u16(sv), want_v)
    assert not np.array_equal(want_k, stage_k)  # something was appended


@pytest.mark.parametrize("n_new,pos0,nwg", [(1, 8191, 16), (1, 4000, 1), (300, 1000, 7), (64, 0, 64)])
def test_writeback_bitwise_and_host_checks(dev, n_new, pos0, nwg):
    say(f"write-back n_new {n_new} pos0 {pos0} workgroups {nwg}")
    B, H, T = 2, 3, 8192
    s, o = shapes(B, H, 4, 16, T, T // 64)
    pool_k = inputs.normal_bf16((B, H, T, 128), 5400, 1).pin_memory()
    pool_v = inputs.normal_bf16((B, H, T, 128), 5400, 2).pin_memory()
    new_k = inputs.normal_bf16((B, H, n_new, 128), 5400 + n_new, 3)
    new_v = inputs.normal_bf16((B, H, n_new, 128), 5400 + n_new, 4)
    ref_k, ref_v = oracle.writeback_kv(o, inputs.to_u16(new_k), inputs.to_u16(new_v), n_new, pos0,
                                       inputs.to_u16(pool_k), inputs.to_u16(pool_v))
    side = torch.cuda.Stream()
    sp.sparda_writeback_kv(s, new_k.to(dev), new_v.to(dev), n_new, pos0, pool_k, pool_v, nwg, side)
    side.synchronize()
    assert np.array_equal(inputs.to_u16(pool_k), ref_k) and np.array_equal(inputs.to_u16(pool_v), ref_v)
    with pytest.raises(sp.SpardaError) as ei:  # pageable host memory is refused
        sp.sparda_writeback_kv(s, new_k.to(dev), new_v.to(dev), n_new, pos0, torch.empty(pool_k.shape, dtype=torch.bfloat16),
                               pool_v, nwg, side)
    assert ei.value.status == sp.SPARDA_ERR_HOST_NOT_MAPPED


# ----------------------------------------------------------------------------- full-size workloads

def _decode_full(dev, name, n_sample_rows, n_sample_heads):
    w = inputs.WORKLOADS[name]
    T, nb = w.seq_len, w.n_blocks
    say(f"full workload {name}: generating on the GPU")
    case = inputs.make_case(w, device=dev)
    s, o = shapes(w.batch, w.n_kv_heads, w.group_size, w.k_total, T, nb)
    kc = gpu_compress(s, case["k"], T, nb, nb, dev)
    sel, cnt = gpu_select(s, case["f"], 1, T - 1, kc, dev)
    rng = np.random.default_rng(7)
    pairs = sorted({(int(rng.integers(w.batch)), int(rng.integers(w.n_kv_heads))) for _ in range(n_sample_rows)})
    sel_mixed = sel.clone()
    sel_np, cnt_np = sel.cpu().numpy(), cnt.cpu().numpy()
    _, o1 = shapes(1, 1, w.group_size, w.k_total, T, nb)
    swaps = 0
    for (b, m) in pairs:
        k16 = inputs.to_u16(case["k"][b:b + 1, m:m + 1])
        kc_ref = oracle.compress_keys(o1, k16, T, 0, nb)
        assert np.array_equal(inputs.to_u16(kc[b:b + 1, m:m + 1]), kc_ref), f"K~ of {(b, m)}"
        f16 = inputs.to_u16(case["f"][b:b + 1, m:m + 1])
        _, sw = compare_selection(o1, f16, kc_ref, 1, T - 1, sel_np[b:b + 1, m:m + 1], cnt_np[b:b + 1, m:m + 1],
                                  [(0, 0, 0)])
        swaps += sw
        ref_sel, ref_cnt, _ = oracle.select_row(o1, f16, 1, T - 1, kc_ref, 0, 0, 0)
        sel_mixed[b, m, 0] = torch.from_numpy(ref_sel)
        # planted blocks are all chosen (5% planted <= top-k slots)
        planted = set(case["plants"][b, m].tolist())
        chosen = set(ref_sel[:ref_cnt].tolist()) - {0, nb - 2, nb - 1}
        if len(planted) <= w.k_total - 3:
            assert planted <= chosen, "every planted block is selected"
        else:
            assert chosen <= planted, "every selected candidate is a planted block"
    out = gpu_attend(s, case["q"], 1, T - 1, case["k"], case["v"], 0, sel_mixed, cnt, dev)
    worst = 0.0
    for (b, m) in pairs[:n_sample_heads]:
        k16 = inputs.to_u16(case["k"][b:b + 1, m:m + 1])
        v16 = inputs.to_u16(case["v"][b:b + 1, m:m + 1])
        q16 = inputs.to_u16(case["q"][b:b + 1, m * w.group_size:(m + 1) * w.group_size])
        ssel = sel_mixed[b:b + 1, m:m + 1].cpu().numpy()
        scnt = cnt[b:b + 1, m:m + 1].cpu().numpy()
        ref = oracle.sparse_attn(o1, q16, 1, T - 1, k16, v16, 0, ssel, scnt, SCALE)
        wab = oracle.sparse_attn(o1, q16, 1, T - 1, k16, abs_bits(v16), 0, ssel, scnt, SCALE)
        got = out[b:b + 1, m * w.group_size:(m + 1) * w.group_size].float().cpu().numpy()
        worst = max(worst, compare_attention(got, ref, f"{name} {(b, m)}", wab))
    say(f"  sampled {len(pairs)} rows, tie swaps {swaps}, attention max err {worst:.3g}")
    # the fused decode step on the same inputs: the same sets, and the same output bit for bit as
    # the attention call over those sets
    sel2, cnt2, out2 = gpu_step(s, case["f"], T - 1, kc, case["q"], case["k"], case["v"], dev)
    assert torch.equal(sel2, sel) and torch.equal(cnt2, cnt)
    out_own = gpu_attend(s, case["q"], 1, T - 1, case["k"], case["v"], 0, sel, cnt, dev)
    assert torch.equal(out2.view(torch.int16), out_own.view(torch.int16))


def test_full_decode_b1_t4k_all_rows(dev):
    _decode_full(dev, "decode_b1_t4k", 64, 64)


def test_full_decode_b8_t32k_samples(dev):
    _decode_full(dev, "decode_b8_t32k", 24, 12)


def test_full_decode_b32_t128k_samples(dev):
    _decode_full(dev, "decode_b32_t128k", 16, 8)


def test_full_prefill_t32k_samples(dev):
    w = inputs.WORKLOADS["prefill_b1_t32k"]
    T, nb = w.seq_len, w.n_blocks
    say("full workload prefill_b1_t32k: generating on the GPU")
    case = inputs.make_case(w, device=dev)
    s, o = shapes(w.batch, w.n_kv_heads, w.group_size, w.k_total, T, nb)
    kc = gpu_compress(s, case["k"], T, nb, nb, dev)
    sel, cnt = gpu_select(s, case["f"], T, 0, kc, dev)
    rng = np.random.default_rng(9)
    ms = [int(x) for x in rng.integers(0, w.n_kv_heads, size=3)]
    rows_r = sorted(set(int(x) for x in rng.integers(0, T, size=40)) | {0, 63, 64, 4095, 4096, T - 1})
    _, o1 = shapes(1, 1, w.group_size, w.k_total, T, nb)
    sel_np, cnt_np = sel.cpu().numpy(), cnt.cpu().numpy()
    sel_mixed = sel.clone()
    swaps = 0
    for m in ms:
        k16 = inputs.to_u16(case["k"][0:1, m:m + 1])
        kc_ref = oracle.compress_keys(o1, k16, T, 0, nb)
        f16 = inputs.to_u16(case["f"][0:1, m:m + 1])
        _, sw = compare_selection(o1, f16, kc_ref, T, 0, sel_np[0:1, m:m + 1], cnt_np[0:1, m:m + 1],
                                  [(0, 0, r) for r in rows_r])
        swaps += sw
        for r in rows_r:
            ref_sel, _, _ = oracle.select_row(o1, f16, T, 0, kc_ref, 0, 0, r)
            sel_mixed[0, m, r] = torch.from_numpy(ref_sel)
    out = gpu_attend(s, case["q"], T, 0, case["k"], case["v"], 0, sel_mixed, cnt, dev)
    worst = 0.0
    for m in ms[:2]:
        G = w.group_size
        k16 = inputs.to_u16(case["k"][0:1, m:m + 1])
        v16 = inputs.to_u16(case["v"][0:1, m:m + 1])
        q16 = inputs.to_u16(case["q"][0:1, m * G:(m + 1) * G])
        ssel = sel_mixed[0:1, m:m + 1].cpu().numpy()
        scnt = cnt[0:1, m:m + 1].cpu().numpy()
        for r in rows_r[::3]:
            for h in range(G):
                ref = oracle.attend_row(o1, q16, T, 0, k16, v16, 0, ssel, scnt, SCALE, 0, h, r)
                wab = oracle.attend_row(o1, q16, T, 0, k16, abs_bits(v16), 0, ssel, scnt, SCALE, 0, h, r)
                got = out[0, m * G + h, r].float().cpu().numpy()
                worst = max(worst, compare_attention(got, ref, f"prefill {(m, h, r)}", wab))
    say(f"  sampled {len(rows_r) * len(ms)} rows, tie swaps {swaps}, attention max err {worst:.3g}")


# Block-coded V (every token of block j holds a 0/1 code of j, see inputs.block_coded_values) at full
# size, in the launch configurations the benchmark times, checked on sampled rows against both
# attention bars.  On these values a kernel that attends one wrong block, drops one or counts one
# twice misses the tight bar by a factor of ten or more (tests/test_parity_bars.py shows it on the
# CPU for every attended block of rows of the same shapes).
BLOCK_CODED = [
    # name, B, Hkv, G, T, n_q, k_total, n_local, sampled (b, m) pairs or rows
    ("decode B32 128K k64 (one workgroup per row)", 32, 8, 4, 131072, 1, 64, 2, 12),
    ("decode B8 32K k64 (split rows + combine)", 8, 8, 4, 32768, 1, 64, 2, 12),
    ("decode B32 128K k96 (entries past 64 in the repeat scan)", 32, 8, 4, 131072, 1, 96, 2, 8),
    ("decode B32 128K Hkv2 G16 k96 local 32 (paper layout, split, P V on MFMA)", 32, 2, 16, 131072, 1, 96, 32, 8),
    ("decode B128 32K Hkv2 G16 k64 (one workgroup per row, P V on MFMA)", 128, 2, 16, 32768, 1, 64, 2, 8),
    ("prefill 32K k64 (tiles of 64 rows)", 1, 8, 4, 32768, 32768, 64, 2, 24),
    ("prefill 32K Hkv2 G16 k96 local 32 (tiles of 16 rows)", 1, 2, 16, 32768, 32768, 96, 32, 24),
]


@pytest.mark.parametrize("name,B,H,G,T,n_q,k_total,n_local,n_sample", BLOCK_CODED)
def test_block_coded_attention_full_size(dev, name, B, H, G, T, n_q, k_total, n_local, n_sample):
    say(f"block-coded V: {name}: generating on the GPU")
    w = inputs.Workload("blockcoded", batch=B, seq_len=T, n_q=n_q, n_kv_heads=H, group_size=G, k_total=k_total,
                        n_local=n_local, seed=8800 + T // 1024 + G + k_total)
    nb = T // 64
    q = inputs.normal_bf16((B, H * G, n_q, 128), w.seed, 0, dev)
    f = inputs.normal_bf16((B, H, n_q, 128), w.seed, 1, dev)
    k = inputs.keys_with_plants(w, f[:, :, -1, :], T, dev, seed=w.seed)
    v = inputs.block_coded_values(B, H, T, dev)
    s, _ = shapes(B, H, G, k_total, T, nb, 1, n_local)
    kc = gpu_compress(s, k, T, nb, nb, dev)
    q_pos0 = T - n_q
    sel, cnt = gpu_select(s, f, n_q, q_pos0, kc, dev)
    out = gpu_attend(s, q, n_q, q_pos0, k, v, 0, sel, cnt, dev)
    _, o1 = shapes(1, 1, G, k_total, T, nb, 1, n_local)
    rng = np.random.default_rng(13)
    if n_q == 1:
        picks = sorted({(int(rng.integers(B)), int(rng.integers(H)), 0) for _ in range(n_sample)})
    else:
        rows = sorted(set(int(x) for x in rng.integers(4096, T, size=n_sample)) | {4096, T - 1})
        picks = [(0, int(rng.integers(H)), r) for r in rows]
    sel_np, cnt_np = sel.cpu().numpy(), cnt.cpu().numpy()
    worst = ratio = 0.0
    cache = {}
    for (b, m, r) in picks:
        if (b, m) not in cache:
            cache[(b, m)] = (inputs.to_u16(k[b:b + 1, m:m + 1]), inputs.to_u16(v[b:b + 1, m:m + 1]))
        k16, v16 = cache[(b, m)]
        q16 = inputs.to_u16(q[b:b + 1, m * G:(m + 1) * G, r:r + 1])
        p = q_pos0 + r
        ssel = sel_np[b:b + 1, m:m + 1, r:r + 1]
        scnt = cnt_np[b:b + 1, m:m + 1, r:r + 1]
        assert int(scnt[0, 0, 0]) >= 1
        ref = oracle.sparse_attn(o1, q16, 1, p, k16, v16, 0, ssel, scnt, SCALE)
        wab = oracle.sparse_attn(o1, q16, 1, p, k16, abs_bits(v16), 0, ssel, scnt, SCALE)
        got = out[b:b + 1, m * G:(m + 1) * G, r:r + 1].float().cpu().numpy()
        worst = max(worst, compare_attention(got, ref, f"{name} {(b, m, r)}", wab))
        ratio = max(ratio, compare_attention.last_tight_ratio)
    say(f"  {len(picks)} rows: max |o - oracle| {worst:.3g}, at most {ratio:.3f} of the tight bar")


def test_paper_configuration_prefill_samples(dev):
    """The paper's model configuration at full size, chunked prefill: 32K, all rows, 32 query /
    2 KV heads (G = 16), k = 96 with a 32-block local window, keys on the (32, 16) grid, in the
    launch configuration the benchmark times; sampled rows of the selection of both groups, and
    of the attention over the oracle's sets."""
    w = inputs.WORKLOADS["paper_prefill_b1_t32k"]
    T, G = w.seq_len, w.group_size
    nw = n_windows(T)
    say("paper configuration prefill: generating on the GPU")
    case = inputs.make_case(w, device=dev)
    s, _ = shapes(w.batch, w.n_kv_heads, G, w.k_total, T, nw, w.n_init, w.n_local, lw=32, sw=16)
    kc = gpu_compress(s, case["k"], T, nw, nw, dev)
    sel, cnt = gpu_select(s, case["f"], T, 0, kc, dev)
    _, o1 = shapes(1, 1, G, w.k_total, T, nw, w.n_init, w.n_local, lw=32, sw=16)
    rng = np.random.default_rng(41)
    rows_r = sorted(set(int(x) for x in rng.integers(0, T, size=30)) | {0, 2047, 2048, 2111, 6143, 6144, T - 1})
    sel_np, cnt_np = sel.cpu().numpy(), cnt.cpu().numpy()
    sel_mixed = sel.clone()
    swaps = 0
    for m in range(w.n_kv_heads):
        kc_ref = oracle.compress_keys(o1, inputs.to_u16(case["k"][0:1, m:m + 1]), T, 0, nw)
        assert np.array_equal(inputs.to_u16(kc[0:1, m:m + 1]), kc_ref)
        f16 = inputs.to_u16(case["f"][0:1, m:m + 1])
        _, sw = compare_selection(o1, f16, kc_ref, T, 0, sel_np[0:1, m:m + 1], cnt_np[0:1, m:m + 1],
                                  [(0, 0, r) for r in rows_r])
        swaps += sw
        for r in rows_r:
            ref_sel, _, _ = oracle.select_row(o1, f16, T, 0, kc_ref, 0, 0, r)
            sel_mixed[0, m, r] = torch.from_numpy(ref_sel)
    out = gpu_attend(s, case["q"], T, 0, case["k"], case["v"], 0, sel_mixed, cnt, dev)
    worst = 0.0
    for m in range(w.n_kv_heads):
        k16 = inputs.to_u16(case["k"][0:1, m:m + 1])
        v16 = inputs.to_u16(case["v"][0:1, m:m + 1])
        q16 = inputs.to_u16(case["q"][0:1, m * G:(m + 1) * G])
        ssel = sel_mixed[0:1, m:m + 1].cpu().numpy()
        scnt = cnt[0:1, m:m + 1].cpu().numpy()
        for r in rows_r[::3]:
            for h in range(0, G, 5):
                ref = oracle.attend_row(o1, q16, T, 0, k16, v16, 0, ssel, scnt, SCALE, 0, h, r)
                wab = oracle.attend_row(o1, q16, T, 0, k16, abs_bits(v16), 0, ssel, scnt, SCALE, 0, h, r)
                got = out[0, m * G + h, r].float().cpu().numpy()
                worst = max(worst, compare_attention(got, ref, f"paper prefill {(m, h, r)}", wab))
    say(f"  sampled {len(rows_r) * w.n_kv_heads} rows, tie swaps {swaps}, attention max err {worst:.3g}")


# ----------------------------------------------------------------------------- score contraction alone

SCORE_MAX = [
    # B, H, T, n_q, q_pos0, n_init, n_local
    (1, 8, 4096, 4096, 0, 1, 2),  # a whole 4K prefill (persistent form): rows without candidates
    (2, 3, 5000, 700, 4300, 1, 2),  # an unaligned, ragged chunk; 6 (batch, group) pairs
    (1, 2, 20000, 1000, 18991, 0, 3),  # odd start, no initial block
    (1, 1, 100, 100, 0, 1, 2),  # no row has a candidate
    (1, 1, 70000, 130, 69870, 1, 2),  # 1089 candidates: the general kernel, 35 M-tiles
    (2, 2, 40000, 300, 39700, 1, 2),  # 617 candidates: the general kernel, ragged chunk
    (1, 2, 32768, 4096, 28672, 1, 2),  # 509 candidates at the end: the persistent form, 8 slots
    (1, 4, 8192, 1, 8191, 4, 16),  # one row, 4 initial blocks, a 16-block local window
]


def gpu_score_max(s, f_dev, n_q, q_pos0, kc_dev, dev):
    out = torch.full((s.batch, s.n_kv_heads, n_q), float("nan"), dtype=torch.float32, device=dev)
    sp.sparda_forecast_score_max(s, f_dev, n_q, q_pos0, kc_dev, out)
    torch.cuda.synchronize()
    return out.cpu().numpy()


def check_score_max(got, want, f_u16, kc_u16, q_pos0, n_init, n_local, label):
    """Rows without candidates must be -inf on both sides; elsewhere the float32 maximum may differ
    from the float64 one by the a-priori bound of a 128-term float32 dot product, gamma_128 times
    the largest sum of |F_d K~_d| over the row's candidates."""
    u = 2.0 ** -24
    gamma = 128 * u / (1 - 128 * u)
    to64 = lambda a: np.abs((np.ascontiguousarray(a).astype(np.uint32) << 16).view(np.float32).astype(np.float64))
    fa, ka = to64(f_u16), to64(kc_u16)
    B, H, n_q = want.shape
    worst = 0.0
    for b in range(B):
        for m in range(H):
            for r in range(n_q):
                hi = (q_pos0 + r) // 64 - n_local
                if hi < n_init:
                    assert want[b, m, r] == -np.inf and got[b, m, r] == -np.inf, (label, b, m, r)
                    continue
                bound = gamma * float((ka[b, m, n_init:hi + 1] @ fa[b, m, r]).max()) + 1e-6
                err = abs(float(got[b, m, r]) - want[b, m, r])
                assert err <= bound, (label, b, m, r, float(got[b, m, r]), want[b, m, r], bound)
                worst = max(worst, err / bound)
    return worst


@pytest.mark.parametrize("B,H,T,n_q,q_pos0,n_init,n_local", SCORE_MAX)
def test_score_max_matches_oracle(dev, B, H, T, n_q, q_pos0, n_init, n_local):
    say(f"score max B{B} H{H} T{T} n_q{n_q} q_pos0 {q_pos0} init {n_init} local {n_local}")
    w, case = make(B, H, 4, T, n_q, n_init + n_local + 1, 5000 + T, n_init=n_init, n_local=n_local)
    t_cap = -(-T // 64) * 64
    nb = max(T // 64, 1)
    s, o = shapes(B, H, 4, n_init + n_local + 1, t_cap, nb, n_init=n_init, n_local=n_local)
    kc_ref = oracle.compress_keys(o, inputs.to_u16(case["k"]), T, 0, T // 64)
    f_u16 = inputs.to_u16(case["f"])
    got = gpu_score_max(s, case["f"].to(dev), n_q, q_pos0, inputs.from_u16(kc_ref, dev), dev)
    want = oracle.forecast_score_max(o, f_u16, n_q, q_pos0, kc_ref)
    worst = check_score_max(got, want, f_u16, kc_ref, q_pos0, n_init, n_local, "score max")
    say(f"  worst error / bound {worst:.3g}")


def test_score_max_full_prefill_t32k(dev):
    """The 32K prefill workload at full size, in the launch the benchmark times; every row of two
    groups against the oracle."""
    w = inputs.WORKLOADS["prefill_b1_t32k"]
    T, nb = w.seq_len, w.n_blocks
    say("full workload prefill_b1_t32k (score max): generating on the GPU")
    case = inputs.make_case(w, device=dev)
    s, _ = shapes(w.batch, w.n_kv_heads, w.group_size, w.k_total, T, nb)
    kc = gpu_compress(s, case["k"], T, nb, nb, dev)
    got = gpu_score_max(s, case["f"], T, 0, kc, dev)
    _, o1 = shapes(1, 1, w.group_size, w.k_total, T, nb)
    worst = 0.0
    for m in (0, w.n_kv_heads - 1):
        kc_ref = oracle.compress_keys(o1, inputs.to_u16(case["k"][0:1, m:m + 1]), T, 0, nb)
        f16 = inputs.to_u16(case["f"][0:1, m:m + 1])
        want = oracle.forecast_score_max(o1, f16, T, 0, kc_ref)
        worst = max(worst, check_score_max(got[0:1, m:m + 1], want, f16, kc_ref, 0, w.n_init, w.n_local, f"m{m}"))
    say(f"  2 x {T} rows, worst error / bound {worst:.3g}")


def test_split_attention_workspace_needs_no_clearing(dev):
    """With fewer rows than CUs the attention splits each row's blocks over workgroups whose
    partials go through the workspace.  A workspace full of arbitrary bytes, and the same
    workspace used again and again, give the same output bit for bit, equal to the oracle's
    within the tight bar."""
    say("split attention: arbitrary workspace bytes, repeated calls")
    B, H, G, T, k_total = 1, 2, 4, 8192, 32
    w, case = make(B, H, G, T, 1, k_total, 7100)
    s, o = shapes(B, H, G, k_total, T, T // 64)
    q, k, v = (case[x].to(dev) for x in ("q", "k", "v"))
    kc_ref = oracle.compress_keys(o, inputs.to_u16(case["k"]), T, 0, T // 64)
    sel, cnt = gpu_select(s, case["f"].to(dev), 1, T - 1, inputs.from_u16(kc_ref, dev), dev)
    n = sp.sparda_workspace_size(s, sp.SPARDA_OP_SPARSE_ATTN, 1, T - 1)
    assert n > 0
    g = torch.Generator(device="cpu").manual_seed(5)
    outs = []
    for fill in ("random", "same", "same", "ones", "same"):
        if fill == "random":
            wsb = torch.randint(0, 256, (n,), dtype=torch.uint8, generator=g).to(dev)
        elif fill == "ones":
            wsb.fill_(255)
        o_dev = torch.full((B, H * G, 1, 128), float("nan"), dtype=torch.bfloat16, device=dev)
        sp.sparda_sparse_attn(s, q, 1, T - 1, k, v, 0, sel, cnt, SCALE, o_dev, wsb)
        torch.cuda.synchronize()
        outs.append(o_dev.clone())
    for x in outs[1:]:
        assert torch.equal(x.view(torch.int16), outs[0].view(torch.int16))
    for (b, m) in ((0, 0), (0, 1)):
        k16 = inputs.to_u16(case["k"][b:b + 1, m:m + 1])
        v16 = inputs.to_u16(case["v"][b:b + 1, m:m + 1])
        q16 = inputs.to_u16(case["q"][b:b + 1, m * G:(m + 1) * G])
        _, o1 = shapes(1, 1, G, k_total, T, T // 64)
        ssel = sel[b:b + 1, m:m + 1].cpu().numpy()
        scnt = cnt[b:b + 1, m:m + 1].cpu().numpy()
        ref = oracle.sparse_attn(o1, q16, 1, T - 1, k16, v16, 0, ssel, scnt, SCALE)
        wab = oracle.sparse_attn(o1, q16, 1, T - 1, k16, abs_bits(v16), 0, ssel, scnt, SCALE)
        compare_attention(outs[0][b:b + 1, m * G:(m + 1) * G].float().cpu().numpy(), ref, f"split {(b, m)}", wab)


# ----------------------------------------------------------------------------- decode step

DECODE_STEP = [
    # B, H, G, T, k_total, lw, sw, n_local: G != 6 on a decode select path runs one kernel per row
    # and attention split (the split select path after its scoring launch), the others the two
    # calls
    (64, 4, 4, 8192, 64, 64, 64, 2),
    (32, 8, 1, 4096, 16, 64, 64, 2),
    (128, 2, 2, 6000, 40, 64, 64, 2),  # ragged last block
    (86, 3, 3, 3000, 24, 64, 64, 2),   # 258 rows
    (64, 4, 5, 4096, 32, 64, 64, 2),
    (64, 4, 4, 8192, 96, 32, 16, 2),   # the paper's (32, 16) grid: window scores max-pooled in LDS
    (64, 4, 4, 200, 16, 64, 64, 2),    # fewer candidates than slots: every candidate is taken
    (4, 8, 4, 8192, 64, 64, 64, 2),    # 32 rows: 8 splits per row, each split's workgroup selects
    (1, 2, 4, 4096, 16, 64, 64, 2),    # 2 rows, 2 splits
    (3, 8, 4, 20000, 200, 64, 64, 2),  # 24 rows, k = 200: splits of 25 blocks
    (1, 2, 4, 131072, 64, 64, 64, 2),  # 2 rows of 2045 candidates: the split select path
    (64, 4, 8, 4096, 32, 64, 64, 2),   # 8 heads: the MFMA P V attention
    (8, 2, 16, 16384, 64, 64, 64, 2),  # 16 heads, 16 rows: splits
    (4, 2, 12, 8192, 32, 32, 16, 2),   # 12 heads on the (32, 16) grid
    (32, 2, 16, 32768, 96, 32, 16, 32),  # the paper's head layout: split select path, 16 heads
    # 200 rows x 2 splits on the split select path: more workgroups than CUs, so some read their
    # row's window scores after others have written attention partials (separate workspace parts)
    (100, 2, 4, 16448, 64, 32, 16, 2),
    (64, 4, 6, 4096, 32, 64, 64, 2),   # 6 heads: the MFMA P V attention
]


@pytest.mark.parametrize("B,H,G,T,k_total,lw,sw,n_local", DECODE_STEP)
def test_decode_step_matches_separate_calls(dev, B, H, G, T, k_total, lw, sw, n_local):
    """sparda_decode_step writes the sets of sparda_forecast_select and the output of
    sparda_sparse_attn over them, bit for bit; a few rows are checked against the oracle too."""
    say(f"decode step B{B} H{H} G{G} T{T} k{k_total} grid ({lw}, {sw})")
    w = inputs.Workload("t", batch=B, seq_len=T, n_q=1, n_kv_heads=H, group_size=G, k_total=k_total, n_init=1,
                        n_local=n_local, seed=6100 + T + G)
    t_cap = -(-T // 64) * 64
    case = inputs.make_case(w, t_cap=t_cap, device=dev)
    nw = (T - lw) // sw + 1
    s, o = shapes(B, H, G, k_total, t_cap, nw, 1, n_local, lw=lw, sw=sw)
    f, q, k, v = (case[x] for x in ("f", "q", "k", "v"))
    kc = gpu_compress(s, k, T, nw, nw, dev)
    sel, cnt = gpu_select(s, f, 1, T - 1, kc, dev)
    out = gpu_attend(s, q, 1, T - 1, k, v, 0, sel, cnt, dev)
    sel2, cnt2, out2 = gpu_step(s, f, T - 1, kc, q, k, v, dev)
    assert torch.equal(cnt2, cnt)
    assert torch.equal(sel2, sel)
    assert torch.equal(out2.view(torch.int16), out.view(torch.int16))
    rows = [(0, 0, 0), (B - 1, H - 1, 0), (B // 2, H // 2, 0)]
    kc16 = inputs.to_u16(kc)
    n, swaps = compare_selection(o, inputs.to_u16(case["f"]), kc16, 1, T - 1, sel2.cpu().numpy(), cnt2.cpu().numpy(),
                                 rows)
    _, o1 = shapes(1, 1, G, k_total, t_cap, nw, 1, n_local, lw=lw, sw=sw)
    for (b, m, _) in rows:
        k16 = inputs.to_u16(case["k"][b:b + 1, m:m + 1])
        v16 = inputs.to_u16(case["v"][b:b + 1, m:m + 1])
        q16 = inputs.to_u16(case["q"][b:b + 1, m * G:(m + 1) * G])
        ssel = sel2[b:b + 1, m:m + 1].cpu().numpy()
        scnt = cnt2[b:b + 1, m:m + 1].cpu().numpy()
        ref = oracle.sparse_attn(o1, q16, 1, T - 1, k16, v16, 0, ssel, scnt, SCALE)
        wab = oracle.sparse_attn(o1, q16, 1, T - 1, k16, abs_bits(v16), 0, ssel, scnt, SCALE)
        compare_attention(out2[b:b + 1, m * G:(m + 1) * G].float().cpu().numpy(), ref, f"step {(b, m)}", wab)
    say(f"  rows {n}, tie swaps {swaps}")


# ----------------------------------------------------------------------------- exact ties

@pytest.mark.parametrize("B,T,n_q,k_total,spread", [
    (1, 8192, 1, 16, 1), (1, 8192, 1024, 16, 1), (1, 32768, 2048, 64, 1), (1, 65536, 3, 64, 1), (1, 40000, 1, 200, 1),
    # integers in [-8, 8]: scores spread over about 2000 values, so the bin that holds the k-th
    # score mixes distinct values and exact ties (decode: split path below 256 rows, fused above)
    (1, 131072, 1, 64, 8), (128, 131072, 1, 64, 8), (128, 32768, 1, 96, 8), (1, 65536, 3, 64, 8),
    (1, 8192, 1024, 16, 8)])
def test_select_exact_ties_take_lowest_index(dev, B, T, n_q, k_total, spread):
    """F and K~ hold small integers, so every score is an exact integer in fp32 and in fp64 and
    many candidates tie; the GPU must break ties by the lower block index exactly as the oracle."""
    say(f"exact ties B{B} T{T} n_q{n_q} k{k_total} spread {spread}")
    H = 2
    nb = T // 64
    t_cap = -(-T // 64) * 64
    s, o = shapes(B, H, 4, k_total, t_cap, nb)
    g = torch.Generator().manual_seed(T + n_q + (B - 1) + 1000 * (spread - 1))
    f = torch.randint(-spread, spread + 1, (B, H, n_q, 128), generator=g).to(torch.bfloat16)
    kc = torch.randint(-spread, spread + 1, (B, H, nb, 128), generator=g).to(torch.bfloat16)
    m3 = nb // 3
    kc[:, :, 0:3 * m3:3] = kc[:, :, 1:3 * m3:3]  # duplicated K~ rows: exact score ties
    q_pos0 = T - n_q
    sel, cnt = gpu_select(s, f.to(dev), n_q, q_pos0, kc.to(dev), dev)
    ref_sel, ref_cnt = oracle.forecast_select(o, inputs.to_u16(f), n_q, q_pos0, inputs.to_u16(kc))
    assert np.array_equal(cnt.cpu().numpy(), ref_cnt)
    assert np.array_equal(sel.cpu().numpy(), ref_sel)


@pytest.mark.parametrize("B,T,n_q,k_total,zero", [
    (1, 8192, 4096, 16, True), (1, 20000, 3000, 100, True), (1, 16384, 4096, 16, False),
    # decode rows: one workgroup per row over 2048-candidate chunks (1 chunk at 128K, 4 at 400K,
    # 8 at 1M), fused (>= 256 rows) and split (fewer rows) paths
    (1, 131072, 1, 64, True), (1, 131072, 1, 64, False), (1, 400000, 1, 64, False), (1, 1048000, 1, 96, True),
    (128, 131072, 1, 64, False), (128, 400000, 1, 64, True), (128, 400000, 1, 64, False)])
def test_select_flat_and_clustered_scores(dev, B, T, n_q, k_total, zero):
    """Score distributions far from the normal model the selection's first threshold guess is
    drawn from: F = 0 (every score of a row is 0: every row takes its lowest candidates), and
    K~ built from 3 distinct rows (each row's scores take 3 values with many ties, so brackets
    collapse onto single values).  Sets must equal the oracle's exactly."""
    say(f"flat/clustered B{B} T{T} n_q{n_q} k{k_total} zero {zero}")
    H = 2
    nb = T // 64
    t_cap = -(-T // 64) * 64
    s, o = shapes(B, H, 4, k_total, t_cap, nb)
    g = torch.Generator().manual_seed(T + 7 + B)
    f = torch.randn((B, H, n_q, 128), generator=g).to(torch.bfloat16)
    if zero:
        f.zero_()
        kc = torch.randn((B, H, nb, 128), generator=g).to(torch.bfloat16)
    else:
        kc = torch.randn((1, 1, 3, 128), generator=g).to(torch.bfloat16)
        kc = kc[:, :, torch.randint(0, 3, (nb,), generator=g)].expand(B, H, nb, 128).contiguous()
    q_pos0 = T - n_q
    sel, cnt = gpu_select(s, f.to(dev), n_q, q_pos0, kc.to(dev), dev)
    ref_sel, ref_cnt = oracle.forecast_select(o, inputs.to_u16(f), n_q, q_pos0, inputs.to_u16(kc))
    assert np.array_equal(cnt.cpu().numpy(), ref_cnt)
    assert np.array_equal(sel.cpu().numpy(), ref_sel)


# ----------------------------------------------------------------------------- the paper's (32, 16) grid

def n_windows(T, lw=32, sw=16):
    return (T - lw) // sw + 1


@pytest.mark.parametrize("B,H,T,t_cap", [(1, 8, 4096, 4096), (2, 2, 1000, 1024), (2, 3, 8192, 8192)])
def test_grid_compress_bitwise(dev, B, H, T, t_cap):
    say(f"grid compress B{B} H{H} T{T}")
    w, case = make(B, H, 4, T, 1, 16, 5100 + T, t_cap=t_cap)
    nw = n_windows(T)
    s, o = shapes(B, H, 4, 16, t_cap, nw, lw=32, sw=16)
    ref = oracle.compress_keys(o, inputs.to_u16(case["k"]), T, 0, nw)
    got = gpu_compress(s, case["k"].to(dev), T, nw, nw, dev)
    assert np.array_equal(inputs.to_u16(got), ref)
    # incremental: the windows completed by each new 16 tokens, as a decode loop would
    inc = torch.zeros_like(got)
    done = 0
    for t in range(16, T + 1, 16 * 7):
        n_now = n_windows(t) if t >= 32 else 0
        if n_now > done:
            sp.sparda_compress_keys(s, case["k"].to(dev), t, done, n_now, inc)
            done = n_now
    if nw > done:
        sp.sparda_compress_keys(s, case["k"].to(dev), T, done, nw, inc)
    torch.cuda.synchronize()
    assert torch.equal(inc, got)


GRID_DECODE = [
    # B, H, T, k_total, n_init, n_local
    (1, 8, 4096, 16, 1, 2),
    (2, 2, 32768, 64, 1, 2),
    (1, 2, 5000, 16, 0, 3),
    (2, 2, 8200, 24, 1, 1),  # one local block: the last candidate's edge window is still open (p % 64 = 7)
    (2, 1, 8255, 24, 1, 1),  # ... and complete (p % 64 = 62)
    (1, 2, 131072, 64, 1, 2),
]


@pytest.mark.parametrize("B,H,T,k_total,n_init,n_local", GRID_DECODE)
def test_grid_decode_select(dev, B, H, T, k_total, n_init, n_local):
    say(f"grid decode select B{B} H{H} T{T} k{k_total} init {n_init} local {n_local}")
    w, case = make(B, H, 4, T, 1, k_total, 5200 + T, n_init=n_init, n_local=n_local)
    t_cap = -(-T // 64) * 64
    nw = n_windows(T)
    s, o = shapes(B, H, 4, k_total, t_cap, nw, n_init, n_local, lw=32, sw=16)
    kc_ref = oracle.compress_keys(o, inputs.to_u16(case["k"]), T, 0, nw)
    sel, cnt = gpu_select(s, case["f"].to(dev), 1, T - 1, inputs.from_u16(kc_ref, dev), dev)
    rows = [(b, m, 0) for b in range(B) for m in range(H)]
    n, swaps = compare_selection(o, inputs.to_u16(case["f"]), kc_ref, 1, T - 1, sel.cpu().numpy(),
                                 cnt.cpu().numpy(), rows)
    say(f"  rows {n}, tie swaps {swaps}")
    if T >= 4096 and n_local == 2:
        sel_np, cnt_np = sel.cpu().numpy(), cnt.cpu().numpy()
        for b in range(B):
            for m in range(H):
                chosen = set(sel_np[b, m, 0, : cnt_np[b, m, 0]].tolist())
                planted = set(int(j) for j in case["plants"][b, m])
                n_sel = k_total - n_init - n_local
                if len(planted) <= n_sel:
                    assert planted <= chosen, "every planted block is selected on the paper's grid too"


GRID_PREFILL = [
    # B, H, T, n_q, q_pos0, k_total, n_local, n_init
    (1, 2, 4096, 4096, 0, 16, 2, 1),        # fused tile kernel, sets staged in LDS
    (2, 1, 3000, 700, 2300, 12, 2, 1),      # chunk off a block boundary, ragged last slice
    (1, 2, 6000, 333, 5601, 20, 1, 1),      # one local block: edge windows hidden until complete
    (1, 1, 5000, 1000, 4000, 16, 1, 0),     # no initial block: block 0 has no window 4b - 1
    (1, 2, 8192, 2000, 6192, 96, 2, 1),     # sets longer than 64 entries: assembled in the chunk buffers
    (1, 2, 20000, 500, 19500, 256, 2, 1),   # the longest sets assembled in the chunk buffers
    (1, 2, 32960, 300, 32660, 300, 2, 1),   # sets past 256 entries: written straight to the output
    (1, 2, 32960, 500, 32460, 64, 2, 1),    # the last row has 512 candidates: the tile kernel's maximum
    (1, 2, 36000, 200, 35800, 64, 2, 1),    # more candidates: the row-wise path (MFMA window scores)
    (1, 1, 70000, 130, 69870, 40, 1, 1),    # 2176 windows per row, one local block: edge windows
    (1, 2, 21000, 19000, 2000, 64, 2, 1),   # 297 slice groups on 256 units: a partial second sweep
]


@pytest.mark.parametrize("B,H,T,n_q,q_pos0,k_total,n_local,n_init", GRID_PREFILL)
def test_grid_prefill_select(dev, B, H, T, n_q, q_pos0, k_total, n_local, n_init):
    say(f"grid prefill select B{B} H{H} T{T} n_q{n_q} q_pos0 {q_pos0} k{k_total} local {n_local} init {n_init}")
    w, case = make(B, H, 4, T, n_q, k_total, 5300 + T, n_init=n_init, n_local=n_local)
    t_cap = -(-T // 64) * 64
    nw = n_windows(T)
    s, o = shapes(B, H, 4, k_total, t_cap, nw, n_init, n_local, lw=32, sw=16)
    kc_ref = oracle.compress_keys(o, inputs.to_u16(case["k"]), T, 0, nw)
    f_u16 = inputs.to_u16(case["f"])
    sel, cnt = gpu_select(s, case["f"].to(dev), n_q, q_pos0, inputs.from_u16(kc_ref, dev), dev)
    rng = np.random.default_rng(2)
    rr = sorted(set(rng.integers(0, n_q, size=min(n_q, 400)).tolist()) | {0, n_q - 1})
    rows = [(b, m, r) for b in range(B) for m in range(H) for r in rr]
    n, swaps = compare_selection(o, f_u16, kc_ref, n_q, q_pos0, sel.cpu().numpy(), cnt.cpu().numpy(), rows)
    say(f"  rows {n}, tie swaps {swaps}")


def test_grid_prefill_full_t32k_samples(dev):
    """The 32K prefill on the (32, 16) grid, all rows selected by the fused kernel; sampled rows
    of three groups against the oracle."""
    w = inputs.WORKLOADS["prefill_b1_t32k"]
    T = w.seq_len
    nw = n_windows(T)
    say("full workload prefill_b1_t32k on the (32, 16) grid: generating on the GPU")
    case = inputs.make_case(w, device=dev)
    s, _ = shapes(w.batch, w.n_kv_heads, w.group_size, w.k_total, T, nw, lw=32, sw=16)
    kc = gpu_compress(s, case["k"], T, nw, nw, dev)
    sel, cnt = gpu_select(s, case["f"], T, 0, kc, dev)
    rng = np.random.default_rng(19)
    ms = [int(x) for x in rng.integers(0, w.n_kv_heads, size=3)]
    rows_r = sorted(set(int(x) for x in rng.integers(0, T, size=40)) | {0, 63, 64, 4095, 4096, 4160, T - 1})
    _, o1 = shapes(1, 1, w.group_size, w.k_total, T, nw, lw=32, sw=16)
    sel_np, cnt_np = sel.cpu().numpy(), cnt.cpu().numpy()
    swaps = 0
    for m in ms:
        kc_ref = oracle.compress_keys(o1, inputs.to_u16(case["k"][0:1, m:m + 1]), T, 0, nw)
        assert np.array_equal(inputs.to_u16(kc[0:1, m:m + 1]), kc_ref)
        f16 = inputs.to_u16(case["f"][0:1, m:m + 1])
        _, sw = compare_selection(o1, f16, kc_ref, T, 0, sel_np[0:1, m:m + 1], cnt_np[0:1, m:m + 1],
                                  [(0, 0, r) for r in rows_r])
        swaps += sw
    say(f"  sampled {len(rows_r) * len(ms)} rows, tie swaps {swaps}")


@pytest.mark.parametrize("T,n_q,k_total,n_local", [(8192, 1024, 16, 2), (20000, 700, 64, 1), (20000, 700, 128, 2),
                                                   (20000, 1, 64, 2)])
def test_grid_select_exact_ties_take_lowest_index(dev, T, n_q, k_total, n_local):
    """Integer F and window keys: every window score, and so every pooled block score, is an exact
    integer on both sides, and duplicated windows make many blocks tie; the GPU must take the
    lower block index exactly as the oracle, in the fused prefill kernel and in decode."""
    say(f"grid exact ties T{T} n_q{n_q} k{k_total} local {n_local}")
    B, H = 1, 2
    nw = n_windows(T)
    t_cap = -(-T // 64) * 64
    s, o = shapes(B, H, 4, k_total, t_cap, nw, 1, n_local, lw=32, sw=16)
    g = torch.Generator().manual_seed(T + n_q + 7)
    f = torch.randint(-1, 2, (B, H, n_q, 128), generator=g).to(torch.bfloat16)
    kc = torch.randint(-1, 2, (B, H, nw, 128), generator=g).to(torch.bfloat16)
    m8 = nw // 8
    kc[:, :, 0:8 * m8:8] = kc[:, :, 4:8 * m8:8]  # window 8i equals window 8i + 4: blocks 2i and 2i + 1 tie often
    q_pos0 = T - n_q
    sel, cnt = gpu_select(s, f.to(dev), n_q, q_pos0, kc.to(dev), dev)
    ref_sel, ref_cnt = oracle.forecast_select(o, inputs.to_u16(f), n_q, q_pos0, inputs.to_u16(kc))
    assert np.array_equal(cnt.cpu().numpy(), ref_cnt)
    assert np.array_equal(sel.cpu().numpy(), ref_sel)


# ----------------------------------------------------------------------------- InfLLM-V2 multi-head selector

def gpu_multihead(s, q_dev, n_q, q_pos0, kc_dev, dev):
    sel = torch.full((s.batch, s.n_kv_heads, n_q, s.k_total), 777, dtype=torch.int16, device=dev)
    cnt = torch.full((s.batch, s.n_kv_heads, n_q), 777, dtype=torch.int16, device=dev)
    sp.sparda_multihead_select(s, q_dev, n_q, q_pos0, kc_dev, SCALE, sel, cnt,
                               ws(s, sp.SPARDA_OP_MULTIHEAD_SELECT, n_q, q_pos0, dev))
    torch.cuda.synchronize()
    return sel, cnt


MULTIHEAD = [
    # B, H, G, T, n_q, k_total, n_init, n_local, grid (lw, sw)
    (2, 2, 4, 4096, 1, 16, 1, 2, (64, 64)),      # fused decode
    (1, 2, 1, 8192, 1, 16, 1, 2, (64, 64)),      # fused, one head: ranks like the dot-product selector
    (1, 1, 2, 20000, 1, 64, 0, 1, (32, 16)),     # fused, (32, 16), no initial block, one local block
    (2, 2, 4, 32768, 1, 64, 1, 2, (32, 16)),     # fused, (32, 16)
    (1, 1, 8, 40000, 1, 32, 1, 3, (32, 16)),     # fused, G = 8
    (1, 2, 3, 9000, 1, 24, 1, 2, (32, 16)),      # G = 3: two-pass fused (MFMA scores)
    (1, 1, 16, 12000, 1, 40, 1, 2, (32, 16)),    # G = 16: two-pass fused
    (2, 2, 16, 131072, 1, 64, 1, 2, (32, 16)),   # G = 16 at 128K: two-pass fused
    (1, 2, 4, 200000, 1, 64, 0, 1, (32, 16)),    # G = 4 past one pass's LDS: two-pass fused
    (1, 1, 4, 524288, 1, 64, 1, 2, (32, 16)),    # 32767 windows: row-wise decode
    (1, 2, 4, 5000, 300, 12, 1, 2, (64, 64)),    # multi-row MFMA tiles, chunk off a block boundary
    (1, 1, 4, 6000, 333, 20, 1, 1, (32, 16)),    # multi-row tiles, (32, 16), one local block
    (1, 1, 16, 9000, 130, 24, 1, 2, (32, 16)),   # tiles of 4 rows x 16 heads, ragged last unit
    (2, 1, 2, 3000, 77, 10, 0, 2, (64, 64)),     # tiles of 32 rows x 2 heads, no initial block
    (1, 2, 8, 7000, 40, 16, 1, 2, (32, 16)),     # tiles of 8 rows x 8 heads
    (1, 1, 1, 4500, 100, 12, 1, 2, (32, 16)),    # tiles of 64 rows x 1 head
    (1, 2, 4, 5000, 9, 12, 1, 2, (32, 16)),      # fewer rows than the tiles take: per-row kernels
    (1, 1, 3, 5000, 50, 12, 1, 2, (32, 16)),     # G = 3 (does not divide 64): per-row kernels
]


@pytest.mark.parametrize("B,H,G,T,n_q,k_total,n_init,n_local,grid", MULTIHEAD)
def test_multihead_select(dev, B, H, G, T, n_q, k_total, n_init, n_local, grid):
    lw, sw = grid
    say(f"multihead select B{B} H{H} G{G} T{T} n_q{n_q} k{k_total} init {n_init} local {n_local} grid {grid}")
    w, case = make(B, H, G, T, n_q, k_total, 6100 + T + G, n_init=n_init, n_local=n_local)
    t_cap = -(-T // 64) * 64
    nw = (T - lw) // sw + 1
    s, o = shapes(B, H, G, k_total, t_cap, nw, n_init, n_local, lw=lw, sw=sw)
    kc_ref = oracle.compress_keys(o, inputs.to_u16(case["k"]), T, 0, nw)
    q_u16 = inputs.to_u16(case["q"])
    q_pos0 = T - n_q
    sel, cnt = gpu_multihead(s, case["q"].to(dev), n_q, q_pos0, inputs.from_u16(kc_ref, dev), dev)
    rng = np.random.default_rng(3)
    rr = sorted(set(rng.integers(0, n_q, size=min(n_q, 60)).tolist()) | {0, n_q - 1})
    rows = [(b, m, r) for b in range(B) for m in range(H) for r in rr]
    n, swaps = compare_multihead_selection(o, q_u16, kc_ref, n_q, q_pos0, SCALE, sel.cpu().numpy(),
                                           cnt.cpu().numpy(), rows)
    say(f"  rows {n}, tie swaps {swaps}")


@pytest.mark.parametrize("T,n_q,G,grid", [(8192, 1, 4, (32, 16)), (8192, 1, 8, (64, 64)), (3000, 200, 4, (32, 16)),
                                          (5000, 1, 3, (64, 64))])
def test_multihead_zero_query_ties_take_lowest_index(dev, T, n_q, G, grid):
    """q = 0: every head's softmax is exactly uniform on both sides, every candidate ties, and the
    lowest indices must win on the fused and row-wise paths alike."""
    lw, sw = grid
    B, H, k_total = 1, 2, 16
    nw = (T - lw) // sw + 1
    t_cap = -(-T // 64) * 64
    s, o = shapes(B, H, G, k_total, t_cap, nw, 1, 2, lw=lw, sw=sw)
    g = torch.Generator().manual_seed(T)
    kc = torch.randn((B, H, nw, 128), generator=g).to(torch.bfloat16)
    q = torch.zeros((B, H * G, n_q, 128), dtype=torch.bfloat16)
    sel, cnt = gpu_multihead(s, q.to(dev), n_q, T - n_q, kc.to(dev), dev)
    ref_sel, ref_cnt = oracle.multihead_select(o, inputs.to_u16(q), n_q, T - n_q, inputs.to_u16(kc), SCALE)
    assert np.array_equal(cnt.cpu().numpy(), ref_cnt)
    assert np.array_equal(sel.cpu().numpy(), ref_sel)


def test_multihead_full_decode_t128k_samples(dev):
    """The 128K, batch-32 decode layer on the (32, 16) grid, selected by the multi-head selector from
    the attention queries; sampled rows against the oracle."""
    w = inputs.WORKLOADS["decode_b32_t128k"]
    T = w.seq_len
    nw = (T - 32) // 16 + 1
    say("multihead full decode_b32_t128k: generating on the GPU")
    case = inputs.make_case(w, device=dev)
    s, _ = shapes(w.batch, w.n_kv_heads, w.group_size, w.k_total, T, nw, lw=32, sw=16)
    kc = gpu_compress(s, case["k"], T, nw, nw, dev)
    sel, cnt = gpu_multihead(s, case["q"], 1, T - 1, kc, dev)
    _, o1 = shapes(1, 1, w.group_size, w.k_total, T, nw, lw=32, sw=16)
    sel_np, cnt_np = sel.cpu().numpy(), cnt.cpu().numpy()
    rng = np.random.default_rng(21)
    swaps = 0
    pairs = sorted(set((int(b), int(m)) for b, m in zip(rng.integers(0, w.batch, 6), rng.integers(0, w.n_kv_heads, 6))))
    for b, m in pairs:
        kc_ref = oracle.compress_keys(o1, inputs.to_u16(case["k"][b:b + 1, m:m + 1]), T, 0, nw)
        assert np.array_equal(inputs.to_u16(kc[b:b + 1, m:m + 1]), kc_ref)
        q16 = inputs.to_u16(case["q"][b:b + 1, m * w.group_size:(m + 1) * w.group_size])
        _, sw_ = compare_multihead_selection(o1, q16, kc_ref, 1, T - 1, SCALE, sel_np[b:b + 1, m:m + 1],
                                             cnt_np[b:b + 1, m:m + 1], [(0, 0, 0)])
        swaps += sw_
    say(f"  sampled {len(pairs)} rows, tie swaps {swaps}")


# ----------------------------------------------------------------------------- step-to-step reuse of staging

def _plan_run(dev, B, H, K, p0, steps, seed):
    """GPU plan vs oracle plan, bit for bit, over a decode run with drifting sets of varying size."""
    from test_oracle_pins import _random_set
    s, o = shapes(B, H, 4, K, 64 * 1024, 1024)
    rng = np.random.default_rng(seed)
    blk_o = np.full((B, H, K), -1, np.int16)
    len_o = np.zeros((B, H, K), np.int16)
    blk_d = torch.full((B, H, K), -1, dtype=torch.int16, device=dev)
    len_d = torch.zeros((B, H, K), dtype=torch.int16, device=dev)
    fetch_d = torch.empty((B, H, K), dtype=torch.int16, device=dev)
    staged_d = torch.empty((B, H, K), dtype=torch.int16, device=dev)
    scnt_d = torch.empty((B, H), dtype=torch.int16, device=dev)
    nf_d = torch.empty((B, H), dtype=torch.int32, device=dev)
    prev = [[None] * H for _ in range(B)]
    p = p0
    total_fetch = total_sel = 0
    for step in range(steps):
        p += 1 if step % 5 else 40
        sel = np.full((B, H, K), -1, np.int16)
        cnt = np.zeros((B, H), np.int16)
        for b in range(B):
            for m in range(H):
                sel[b, m], cnt[b, m] = _random_set(rng, p, K, prev[b][m], vary=True)
                prev[b][m] = sel[b, m, :cnt[b, m]].tolist()
        fetch, staged, n_fetch = oracle.plan_staging(o, sel, cnt, p, blk_o, len_o)
        sp.sparda_plan_staging(s, torch.from_numpy(sel).to(dev), torch.from_numpy(cnt).to(dev), p, blk_d, len_d,
                               fetch_d, staged_d, scnt_d, nf_d)
        torch.cuda.synchronize()
        assert np.array_equal(fetch_d.cpu().numpy(), fetch), f"step {step}: fetch"
        assert np.array_equal(staged_d.cpu().numpy(), staged), f"step {step}: sel_staged"
        assert np.array_equal(nf_d.cpu().numpy(), n_fetch), f"step {step}: n_fetch"
        assert np.array_equal(blk_d.cpu().numpy(), blk_o) and np.array_equal(len_d.cpu().numpy(), len_o)
        assert np.all(scnt_d.cpu().numpy() == K)
        total_fetch += int(n_fetch.sum())
        total_sel += int(cnt.sum())
    return total_fetch, total_sel


@pytest.mark.parametrize("B,H,K,p0,steps", [(2, 3, 12, 1500, 150), (1, 4, 64, 9000, 120), (1, 2, 200, 30000, 60)])
def test_plan_staging_matches_oracle(dev, B, H, K, p0, steps):
    say(f"plan staging B{B} H{H} K{K} p0 {p0} steps {steps}")
    fetched, selected = _plan_run(dev, B, H, K, p0, steps, 77 + K)
    say(f"  fetched {fetched} of {selected} selected blocks")
    assert fetched < selected


def test_reuse_pipeline_attends_exact_tokens(dev):
    """A 45-step decode crossing block boundaries: the host pool receives each token only when it
    is decoded (later tokens hold a sentinel), the plan decides the fetches, the gather copies only
    them, and the staged attention must equal the oracle's attention over the true K/V."""
    from test_oracle_pins import _random_set
    B, H, G, K = 1, 2, 4, 16
    T = 64 * 64
    p0 = 64 * 50 - 20
    w, case = make(B, H, G, T, 1, K, 8100)
    s, o = shapes(B, H, G, K, T, T // 64)
    k16, v16 = inputs.to_u16(case["k"]), inputs.to_u16(case["v"])
    hk = torch.full_like(case["k"], 7.0).pin_memory()  # tokens not yet decoded: a sentinel
    hv = torch.full_like(case["v"], -7.0).pin_memory()
    hk[:, :, :p0] = case["k"][:, :, :p0]
    hv[:, :, :p0] = case["v"][:, :, :p0]
    st_k = torch.zeros(B, H, K, 64, 128, dtype=torch.bfloat16, device=dev)
    st_v = torch.zeros_like(st_k)
    blk_d = torch.full((B, H, K), -1, dtype=torch.int16, device=dev)
    len_d = torch.zeros((B, H, K), dtype=torch.int16, device=dev)
    fetch_d = torch.empty((B, H, K), dtype=torch.int16, device=dev)
    staged_d = torch.empty((B, H, K), dtype=torch.int16, device=dev)
    scnt_d = torch.empty((B, H), dtype=torch.int16, device=dev)
    nf_d = torch.empty((B, H), dtype=torch.int32, device=dev)
    rng = np.random.default_rng(5)
    prev = [None] * H
    worst, fetched, selected = 0.0, 0, 0
    for step in range(45):
        p = p0 + step
        hk[:, :, p] = case["k"][:, :, p]  # the decoded token's K/V reach the host pool
        hv[:, :, p] = case["v"][:, :, p]
        sel = np.full((B, H, K), -1, np.int16)
        cnt = np.zeros((B, H), np.int16)
        for m in range(H):
            sel[0, m], cnt[0, m] = _random_set(rng, p, K, prev[m], keep=0.8)
            prev[m] = sel[0, m, :cnt[0, m]].tolist()
        sp.sparda_plan_staging(s, torch.from_numpy(sel).to(dev), torch.from_numpy(cnt).to(dev), p, blk_d, len_d,
                               fetch_d, staged_d, scnt_d, nf_d)
        sp.sparda_gather_blocks(s, hk, hv, fetch_d, scnt_d, st_k, st_v, 8)
        q = case["q"][:, :, 0:1].to(dev)
        out = gpu_attend(s, q, 1, p, st_k, st_v, 1, staged_d, scnt_d, dev)
        fetched += int(nf_d.sum().item())
        selected += int(cnt.sum())
        q16 = inputs.to_u16(case["q"][:, :, 0:1])
        for h in range(H * G):
            ref = oracle.attend_row(o, q16, 1, p, k16, v16, 0, sel[:, :, None], cnt[:, :, None], SCALE, 0, h, 0)
            wab = oracle.attend_row(o, q16, 1, p, k16, abs_bits(v16), 0, sel[:, :, None], cnt[:, :, None], SCALE,
                                    0, h, 0)
            worst = max(worst, compare_attention(out[0, h, 0].float().cpu().numpy(), ref, f"step {step} head {h}",
                                                 wab))
    say(f"  fetched {fetched} of {selected} selected blocks, attention max err {worst:.3g}")
    assert fetched < selected


# ----------------------------------------------------------------------------- indexer-training loss (Eq. 6-7)

KL_CASES = [
    # B, H, G, T, n_q, k_top, n_init, n_local, grid
    (1, 2, 4, 2048, 48, 16, 1, 2, (32, 16)),
    (1, 1, 16, 3000, 20, 30, 1, 1, (32, 16)),
    (2, 1, 4, 1500, 16, 0, 0, 2, (32, 16)),      # k_top = 0: only the rest bucket, loss 0
    (1, 1, 4, 1200, 10, 4096, 1, 2, (32, 16)),   # k_top beyond the candidates: all of them
    (1, 2, 2, 4096, 12, 12, 1, 2, (64, 64)),     # block-granular prediction grid
    (1, 1, 4, 16384, 6, 64, 1, 2, (32, 16)),     # 1022 positions, 16K fine windows
    (1, 2, 8, 5000, 37, 20, 1, 2, (32, 16)),     # G = 8: units of 8 rows, ragged last unit
    (1, 1, 1, 3000, 70, 10, 1, 2, (64, 64)),     # G = 1: units of 64 rows, two units
    (1, 1, 3, 2500, 9, 12, 1, 2, (32, 16)),      # G = 3: the target computed inside the row kernel
]


@pytest.mark.parametrize("B,H,G,T,n_q,k_top,n_init,n_local,grid", KL_CASES)
def test_indexer_kl_matches_oracle(dev, B, H, G, T, n_q, k_top, n_init, n_local, grid):
    """Loss and gradient per row against the oracle.  The kernels accumulate every softmax and
    bucket sum in float32 as per-lane partial sums of at most a few hundred terms merged in a tree,
    so each normalised weight carries a relative error of order 100 ulps (1e-5) at most; the loss
    is a difference of cross-entropy terms of size ~1-10 with weights summing to 1 and the gradient
    a weighted sum of the compressed keys, hence the bars
        |loss - ref| <= 4e-6 + 1e-5 |ref|,   |dF - ref| <= 1e-5 (|ref| + max |ref|) + 2e-8,
    where 2e-8 covers rows whose exact gradient vanishes (k_top = 0: float32 leaves a residue of a
    few ulps of the bucket weights times sm_scale |K~|).  The largest errors measured over these
    cases were 2.4e-7 (loss, rows with loss 0.005-0.2) and 1.7e-9 (gradient, max |dF| 2e-4 to 1e-2),
    about 20 times inside the bars."""
    lw, sw = grid
    say(f"indexer kl B{B} H{H} G{G} T{T} n_q{n_q} k{k_top} init {n_init} local {n_local} grid {grid}")
    w, case = make(B, H, G, T, n_q, 8, 9100 + T + G, n_init=n_init, n_local=n_local)
    t_cap = -(-T // 64) * 64
    nw = (T - lw) // sw + 1
    s, o = shapes(B, H, G, 8, t_cap, nw, n_init, n_local, lw=lw, sw=sw)
    k16 = inputs.to_u16(case["k"])
    kcp = oracle.compress_keys(o, k16, T, 0, nw)
    q_pos0 = T - n_q
    ofine = oracle.Shape(**{**o.__dict__, "nc_cap": T - 1, "cmp_kernel": 2, "cmp_stride": 1})
    kct = oracle.compress_keys(ofine, k16, T, 0, T - 1)
    loss = torch.full((B, H, n_q), float("nan"), dtype=torch.float32, device=dev)
    dF = torch.full((B, H, n_q, 128), float("nan"), dtype=torch.float32, device=dev)
    wsb = sp.sparda_workspace_size(s, sp.SPARDA_OP_INDEXER_KL, n_q, q_pos0)
    wst = torch.empty(wsb, dtype=torch.uint8, device=dev)
    sp.sparda_indexer_kl(s, case["q"].to(dev), case["k"].to(dev), case["f"].to(dev), inputs.from_u16(kcp, dev), n_q,
                         q_pos0, SCALE, k_top, loss, dF, wst)
    torch.cuda.synchronize()
    loss_g, dF_g = loss.cpu().numpy(), dF.cpu().numpy()
    q16, f16 = inputs.to_u16(case["q"]), inputs.to_u16(case["f"])
    worst_l = worst_d = ratio_l = ratio_d = 0.0
    for b in range(B):
        for m in range(H):
            for r in range(n_q):
                ref, dref, _, _ = oracle.indexer_kl_row(o, q16, kct, 2, 1, f16, kcp, n_q, q_pos0, SCALE, k_top, b, m, r)
                gl = float(loss_g[b, m, r])
                bar_l = 4e-6 + 1e-5 * abs(ref)
                assert abs(gl - ref) <= bar_l, f"row {(b, m, r)}: loss {gl} vs {ref}"
                tol = 1e-5 * (np.abs(dref) + np.abs(dref).max()) + 2e-8
                err_d = np.abs(dF_g[b, m, r] - dref)
                assert np.all(err_d <= tol), f"row {(b, m, r)}: gradient off by {float(err_d.max()):.3g}"
                worst_l = max(worst_l, abs(gl - ref))
                worst_d = max(worst_d, float(err_d.max()))
                ratio_l = max(ratio_l, abs(gl - ref) / bar_l)
                ratio_d = max(ratio_d, float((err_d / tol).max()))
    say(f"  worst |loss - ref| {worst_l:.3g} ({ratio_l:.3f} of its bar), worst |dF - ref| {worst_d:.3g} "
        f"({ratio_d:.3f} of its bar)")


def test_paper_configuration_decode_samples(dev):
    """The paper's model configuration at full size: decode at 128K, B32, 32 query / 2 KV heads,
    k = 96 with a 32-block local window, keys on the (32, 16) grid; sampled rows of the selection
    and of the attention over the oracle's sets."""
    w = inputs.WORKLOADS["paper_decode_b32_t128k"]
    T, G = w.seq_len, w.group_size
    nw = (T - 32) // 16 + 1
    say("paper configuration decode: generating on the GPU")
    case = inputs.make_case(w, device=dev)
    s, _ = shapes(w.batch, w.n_kv_heads, G, w.k_total, T, nw, w.n_init, w.n_local, lw=32, sw=16)
    kc = gpu_compress(s, case["k"], T, nw, nw, dev)
    sel, cnt = gpu_select(s, case["f"], 1, T - 1, kc, dev)
    _, o1 = shapes(1, 1, G, w.k_total, T, nw, w.n_init, w.n_local, lw=32, sw=16)
    sel_np, cnt_np = sel.cpu().numpy(), cnt.cpu().numpy()
    rng = np.random.default_rng(31)
    pairs = sorted(set((int(b), int(m)) for b, m in zip(rng.integers(0, w.batch, 5), rng.integers(0, w.n_kv_heads, 5))))
    sel_mixed = sel.clone()
    swaps = 0
    for b, m in pairs:
        k16 = inputs.to_u16(case["k"][b:b + 1, m:m + 1])
        kc_ref = oracle.compress_keys(o1, k16, T, 0, nw)
        assert np.array_equal(inputs.to_u16(kc[b:b + 1, m:m + 1]), kc_ref)
        f16 = inputs.to_u16(case["f"][b:b + 1, m:m + 1])
        _, sw_ = compare_selection(o1, f16, kc_ref, 1, T - 1, sel_np[b:b + 1, m:m + 1], cnt_np[b:b + 1, m:m + 1],
                                   [(0, 0, 0)])
        swaps += sw_
        ref_sel, _, _ = oracle.select_row(o1, f16, 1, T - 1, kc_ref, 0, 0, 0)
        sel_mixed[b, m, 0] = torch.from_numpy(ref_sel)
    out = gpu_attend(s, case["q"], 1, T - 1, case["k"], case["v"], 0, sel_mixed, cnt, dev)
    worst = 0.0
    for b, m in pairs[:3]:
        k16 = inputs.to_u16(case["k"][b:b + 1, m:m + 1])
        v16 = inputs.to_u16(case["v"][b:b + 1, m:m + 1])
        q16 = inputs.to_u16(case["q"][b:b + 1, m * G:(m + 1) * G])
        ssel = sel_mixed[b:b + 1, m:m + 1].cpu().numpy()
        scnt = cnt[b:b + 1, m:m + 1].cpu().numpy()
        for h in range(0, G, 5):
            ref = oracle.attend_row(o1, q16, 1, T - 1, k16, v16, 0, ssel, scnt, SCALE, 0, h, 0)
            wab = oracle.attend_row(o1, q16, 1, T - 1, k16, abs_bits(v16), 0, ssel, scnt, SCALE, 0, h, 0)
            worst = max(worst, compare_attention(out[b, m * G + h, 0].float().cpu().numpy(), ref, f"{(b, m, h)}",
                                                 wab))
    say(f"  sampled {len(pairs)} rows, tie swaps {swaps}, attention max err {worst:.3g}")
