"""Pins of the CPU oracle against things other than itself.

Each function of the oracle is checked against an independent brute force (dense numpy/torch
algebra, full sorts), closed forms, the invariants the paper states, and the block budget the
paper prints.  test_oracle_mutants.py plants mistakes in copies of the oracle to show that the
pins notice them.
"""
import json
import math
import os

import numpy as np
import pytest
import torch

import brute
from paper_2606_04511_amd import inputs

pytestmark = pytest.mark.filterwarnings("ignore::RuntimeWarning")

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def rnd_u16(shape, seed, tid):
    return inputs.to_u16(inputs.normal_bf16(shape, seed, tid))


def shape_for(oracle, B, H, G, T, k_total, n_init=1, n_local=2, D=128, t_cap=None, nc_cap=None):
    t_cap = T if t_cap is None else t_cap
    return oracle.Shape(batch=B, n_kv_heads=H, group_size=G, head_dim=D, block_size=64, n_init=n_init,
                        n_local=n_local, k_total=k_total, t_cap=t_cap,
                        nc_cap=max(t_cap // 64, 1) if nc_cap is None else nc_cap)


# ----------------------------------------------------------------------------- bf16 rounding

def test_bf16_rounding_matches_torch_on_float32_values(oracle_lib):
    x = torch.randn(4000, generator=torch.Generator().manual_seed(5), dtype=torch.float32) * 37.0
    want = x.to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    got = np.array([oracle_lib.f64_to_bf16(float(v)) for v in x.tolist()], np.uint16)
    assert np.array_equal(got, want)


def test_bf16_rounding_is_direct_not_double():
    """1 + 2^-8 + 2^-30 is just above a bf16 midpoint; rounding through float32 first lands on the
    midpoint and ties down to 1.0.  Direct rounding must go up."""
    import oracle
    x = 1.0 + 2.0 ** -8 + 2.0 ** -30
    assert oracle.f64_to_bf16(x) == 0x3F81
    assert oracle.f64_to_bf16(1.0 + 2.0 ** -8) == 0x3F80          # exact tie -> even
    assert oracle.f64_to_bf16(1.0 + 3 * 2.0 ** -8) == 0x3F82      # exact tie -> even (up)
    assert oracle.f64_to_bf16(-2.5) == 0xC020
    assert oracle.f64_to_bf16(0.0) == 0x0000 and oracle.f64_to_bf16(-0.0) == 0x8000
    # the independent integer rounding of the brute force agrees on random float64 values
    rng = np.random.default_rng(3)
    vals = rng.standard_normal(3000) * 10.0
    got = np.array([oracle.f64_to_bf16(float(v)) for v in vals], np.uint16)
    assert np.array_equal(got, brute.f64_to_bf16_bits(vals))


# ----------------------------------------------------------------------------- compress (Eq. 2)

def test_compress_constant_keys_give_that_key(oracle_lib):
    s = shape_for(oracle_lib, 1, 2, 4, 256, 16)
    row = rnd_u16((2, 1, 128), 7, 0)
    k = np.broadcast_to(row, (1, 2, 256, 128)).copy()
    kc = oracle_lib.compress_keys(s, k, 256, 0, 4)
    assert np.array_equal(kc, np.broadcast_to(row, (1, 2, 4, 128)))


def test_compress_ramp_closed_form(oracle_lib):
    """K[t][d] = t (exact in bf16 for t < 256): the block mean is 64 j + 31.5."""
    s = shape_for(oracle_lib, 1, 1, 1, 256, 16)
    t = np.arange(256, dtype=np.float32)
    kf = np.broadcast_to(t[:, None], (256, 128))
    k = torch.from_numpy(np.ascontiguousarray(kf)).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    kc = oracle_lib.compress_keys(s, k.reshape(1, 1, 256, 128), 256, 0, 4)
    for j in range(4):
        want = torch.tensor(64.0 * j + 31.5, dtype=torch.float64).to(torch.float32).to(torch.bfloat16)
        assert kc[0, 0, j, 0] == int(want.view(torch.int16).item()) & 0xFFFF


def test_compress_matches_bruteforce(oracle_lib):
    s = shape_for(oracle_lib, 2, 3, 4, 448, 16)
    k = rnd_u16((2, 3, 448, 128), 11, 2)
    kc = oracle_lib.compress_keys(s, k, 448, 0, 7)
    assert np.array_equal(kc, brute.compress(k, 7))


def test_compress_incremental_equals_full(oracle_lib):
    s = shape_for(oracle_lib, 1, 2, 4, 640, 16)
    k = rnd_u16((1, 2, 640, 128), 12, 2)
    full = oracle_lib.compress_keys(s, k, 640, 0, 10)
    inc = np.zeros_like(full)
    for t_ctx in range(64, 641, 64):  # a block is compressed once it is complete
        oracle_lib.compress_keys(s, k, t_ctx, t_ctx // 64 - 1, t_ctx // 64, inc)
    assert np.array_equal(full, inc)


def test_compress_rejects_incomplete_block(oracle_lib):
    s = shape_for(oracle_lib, 1, 1, 1, 128, 16)
    k = rnd_u16((1, 1, 128, 128), 1, 2)
    with pytest.raises(oracle_lib.OracleError):
        oracle_lib.compress_keys(s, k, 100, 0, 2)


# ----------------------------------------------------------------------------- select (Eq. 1, Eq. 4)

@pytest.mark.parametrize("T,k_total,n_init,n_local,G", [
    (1, 3, 1, 2, 4), (63, 3, 1, 2, 4), (64, 3, 1, 2, 4), (65, 4, 1, 2, 1), (128, 3, 1, 1, 16),
    (191, 5, 0, 3, 4), (192, 4, 1, 2, 4), (257, 4, 1, 1, 4), (640, 6, 1, 2, 4), (1280, 7, 1, 3, 4),
    (1280, 22, 1, 2, 4), (4096, 16, 1, 2, 4),
])
def test_select_matches_bruteforce(oracle_lib, T, k_total, n_init, n_local, G):
    H, D = 2, 128
    n_q = min(T, 70)
    q_pos0 = T - n_q
    nc = max((T - 1) // 64, 1)
    s = shape_for(oracle_lib, 1, H, G, T, k_total, n_init, n_local, t_cap=max(64, -(-T // 64) * 64), nc_cap=nc)
    f = rnd_u16((1, H, n_q, D), 100 + T, 1)
    kc = rnd_u16((1, H, nc, D), 100 + T, 4)
    sel, cnt = oracle_lib.forecast_select(s, f, n_q, q_pos0, kc)
    bsel, bcnt, _ = brute.select_rows(f, kc, q_pos0, k_total, n_init, n_local)
    assert np.array_equal(cnt, bcnt)
    assert np.array_equal(sel, bsel)


def test_select_forced_blocks_and_count(oracle_lib):
    T, H, k_total = 2048, 3, 9
    s = shape_for(oracle_lib, 2, H, 4, T, k_total)
    f = rnd_u16((2, H, T, 128), 21, 1)
    kc = rnd_u16((2, H, 32, 128), 21, 4)
    sel, cnt = oracle_lib.forecast_select(s, f, T, 0, kc)
    for r in range(0, T, 37):
        blk = r // 64
        for b in range(2):
            for m in range(H):
                row = sel[b, m, r]
                n = int(cnt[b, m, r])
                assert n == min(k_total, blk + 1)
                valid = row[:n]
                assert np.all(np.diff(valid) > 0) and np.all(row[n:] == -1)
                assert 0 in valid and blk in valid and (blk - 1 in valid or blk == 0)
                assert valid.max() <= blk


def test_select_takes_every_causal_block_when_k_covers(oracle_lib):
    T = 1024
    s = shape_for(oracle_lib, 1, 2, 4, T, 40)
    f = rnd_u16((1, 2, T, 128), 22, 1)
    kc = rnd_u16((1, 2, 16, 128), 22, 4)
    sel, cnt = oracle_lib.forecast_select(s, f, T, 0, kc)
    for r in range(T):
        blk = r // 64
        assert list(sel[0, 0, r, : cnt[0, 0, r]]) == list(range(blk + 1))


def test_select_ignores_initial_and_local_keys(oracle_lib):
    """Selection excludes the initial and local blocks, so it cannot depend on their keys
    (Sec. 4.1: the next layer's newly appended keys do not change the selection)."""
    T, nb = 4096, 64
    s = shape_for(oracle_lib, 1, 2, 4, T, 16)
    f = rnd_u16((1, 2, 1, 128), 23, 1)
    kc = rnd_u16((1, 2, nb, 128), 23, 4)
    sel, cnt = oracle_lib.forecast_select(s, f, 1, T - 1, kc)
    kc2 = kc.copy()
    noise = rnd_u16((1, 2, 3, 128), 24, 4)
    kc2[:, :, [0, nb - 2, nb - 1]] = noise  # the initial block and both local blocks
    sel2, cnt2 = oracle_lib.forecast_select(s, f, 1, T - 1, kc2)
    assert np.array_equal(sel, sel2) and np.array_equal(cnt, cnt2)


@pytest.mark.parametrize("name", ["decode_b1_t4k", "decode_b8_t32k"])
def test_select_planted_recall(oracle_lib, name):
    w = inputs.WORKLOADS[name]
    if name == "decode_b8_t32k":
        w = inputs.Workload(w.name, batch=2, seq_len=w.seq_len, n_q=1, k_total=w.k_total, seed=w.seed)
    case = inputs.make_case(w)
    s = shape_for(oracle_lib, w.batch, w.n_kv_heads, w.group_size, w.seq_len, w.k_total)
    k = inputs.to_u16(case["k"])
    kc = oracle_lib.compress_keys(s, k, w.seq_len, 0, w.n_blocks)
    sel, cnt = oracle_lib.forecast_select(s, inputs.to_u16(case["f"]), 1, w.seq_len - 1, kc)
    plants = case["plants"]
    n_sel = w.k_total - 3
    assert plants.shape[2] <= n_sel
    for b in range(w.batch):
        for m in range(w.n_kv_heads):
            chosen = set(sel[b, m, 0, : cnt[b, m, 0]].tolist())
            assert set(plants[b, m].tolist()) <= chosen


def test_decode_equals_prefill_row(oracle_lib):
    """A decode step at position i selects what row i of a prefill selects."""
    T = 1536
    s = shape_for(oracle_lib, 1, 2, 4, T, 8)
    f = rnd_u16((1, 2, T, 128), 25, 1)
    kc = rnd_u16((1, 2, 24, 128), 25, 4)
    sel, cnt = oracle_lib.forecast_select(s, f, T, 0, kc)
    for i in (0, 63, 64, 200, 777, 1535):
        d_sel, d_cnt = oracle_lib.forecast_select(s, np.ascontiguousarray(f[:, :, i:i + 1]), 1, i, kc)
        assert np.array_equal(d_sel[:, :, 0], sel[:, :, i]) and np.array_equal(d_cnt[:, :, 0], cnt[:, :, i])


def test_select_worked_example_with_tie(oracle_lib):
    """Hand-worked case, D = 2, decode at p = 447 (block 6), one initial and two local blocks:
    forced = {0, 5, 6}, candidates = {1, 2, 3, 4}.  With F = (1, 0.5):
      s1 = 1, s2 = 2, s3 = 2 - 1 = 1, s4 = -1.
    k_total = 5 leaves two top-k slots: block 2, then the tie s1 = s3 goes to the lower index 1."""
    s = oracle_lib.Shape(batch=1, n_kv_heads=1, group_size=1, head_dim=2, n_init=1, n_local=2, k_total=5,
                         t_cap=448, nc_cap=7)
    to = lambda a: torch.tensor(a, dtype=torch.float32).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    f = to([[[[1.0, 0.5]]]])
    kc = to([[[[9, 9], [1, 0], [0, 4], [2, -2], [-1, 0], [9, 9], [9, 9]]]])
    sel, cnt, scores = oracle_lib.select_row(s, f, 1, 447, kc, 0, 0, 0)
    assert cnt == 5 and list(sel) == [0, 1, 2, 5, 6]
    assert np.isnan(scores[0]) and np.isnan(scores[5]) and np.isnan(scores[6])
    assert list(scores[1:5]) == [1.0, 2.0, 1.0, -1.0]


# ----------------------------------------------------------------------------- the paper's (32, 16) grid

def grid_shape(oracle, B, H, T, k_total, lw=32, sw=16, n_init=1, n_local=2, D=128):
    return oracle.Shape(batch=B, n_kv_heads=H, group_size=4, head_dim=D, block_size=64, n_init=n_init,
                        n_local=n_local, k_total=k_total, t_cap=T, nc_cap=(T - lw) // sw + 1, cmp_kernel=lw,
                        cmp_stride=sw)


@pytest.mark.parametrize("lw,sw", [(32, 16), (16, 16), (64, 32), (32, 32)])
def test_compress_windows_match_bruteforce(oracle_lib, lw, sw):
    T = 640
    s = grid_shape(oracle_lib, 2, 2, T, 8, lw, sw)
    k = rnd_u16((2, 2, T, 128), 71, 0)
    got = oracle_lib.compress_keys(s, k, T, 0, s.nc_cap)
    assert np.array_equal(got, brute.compress_windows(k, s.nc_cap, lw, sw))


def test_compress_windows_incremental_and_bounds(oracle_lib):
    """Compressing the windows completed by each 16-token step equals one full pass; a window that
    reaches past t_ctx is refused."""
    import oracle
    T = 512
    s = grid_shape(oracle_lib, 1, 2, T, 8)
    k = rnd_u16((1, 2, T, 128), 72, 0)
    full = oracle_lib.compress_keys(s, k, T, 0, s.nc_cap)
    inc = np.zeros_like(full)
    done = 0
    for t in range(16, T + 1, 16):
        n_now = (t - 32) // 16 + 1 if t >= 32 else 0
        if n_now > done:
            oracle_lib.compress_keys(s, k, t, done, n_now, inc)
            done = n_now
    assert np.array_equal(inc, full)
    with pytest.raises(oracle.OracleError):
        oracle_lib.compress_keys(s, k, 300, 0, 18)  # window 17 ends at token 304 > 300


@pytest.mark.parametrize("T,n_q,k_total,n_init,n_local,lw,sw", [
    (1024, 1, 6, 1, 2, 32, 16), (1024, 200, 6, 1, 2, 32, 16), (2000, 300, 9, 0, 3, 32, 16),
    (1500, 260, 7, 2, 1, 32, 16), (1280, 150, 5, 1, 2, 64, 32), (1280, 150, 5, 1, 1, 16, 8)])
def test_select_pooled_matches_bruteforce(oracle_lib, T, n_q, k_total, n_init, n_local, lw, sw):
    s = grid_shape(oracle_lib, 1, 2, T, k_total, lw, sw, n_init, n_local)
    f = rnd_u16((1, 2, n_q, 128), 73, 1)
    k = rnd_u16((1, 2, T, 128), 73, 2)
    kc = oracle_lib.compress_keys(s, k, T, 0, s.nc_cap)
    q_pos0 = T - n_q
    sel, cnt = oracle_lib.forecast_select(s, f, n_q, q_pos0, kc)
    bsel, bcnt, pooled = brute.select_rows_pooled(f, kc, q_pos0, k_total, n_init, n_local, lw, sw)
    assert np.array_equal(cnt, bcnt)
    assert np.array_equal(sel, bsel)
    for r in (0, n_q // 2, n_q - 1):
        _, _, scores, wins = oracle_lib.select_row_windows(s, f, n_q, q_pos0, kc, 0, 1, r)
        cand = ~np.isnan(scores)
        assert np.allclose(scores[cand], pooled[0, 1, r, : len(scores)][cand], rtol=0, atol=1e-12)
        # the reported window gives exactly the block's score
        f64, k64 = brute.bf16_bits_to_f64(f), brute.bf16_bits_to_f64(kc)
        for j in np.flatnonzero(cand):
            assert abs(float(f64[0, 1, r] @ k64[0, 1, wins[j]]) - scores[j]) <= 1e-12


def test_select_pooled_closed_form_block_constant_keys(oracle_lib):
    """Keys constant within each 64-token block: the windows inside block j equal K_j and the window
    straddling j and j+1 is (K_j + K_{j+1}) / 2 (exact in bf16 for these values), so the pooled
    score of block j is max(s_j, (s_{j-1} + s_j) / 2, (s_j + s_{j+1}) / 2) with s_j = F . K_j."""
    T, D = 640, 2
    s = oracle_lib.Shape(batch=1, n_kv_heads=1, group_size=1, head_dim=D, block_size=64, n_init=1, n_local=2,
                         k_total=10, t_cap=T, nc_cap=(T - 32) // 16 + 1, cmp_kernel=32, cmp_stride=16)
    to = lambda a: np.array(a, np.float32).view(np.uint32).__rshift__(16).astype(np.uint16)
    blockv = [[0, 0], [1, 0], [3, 1], [-2, 0], [0, 2], [5, -1], [1, 1], [2, 2], [0, 0], [0, 0]]
    k = to([[np.repeat(np.array(blockv, np.float32), 64, axis=0)]])
    kc = oracle_lib.compress_keys(s, k, T, 0, s.nc_cap)
    f = to([[[[1.0, 0.5]]]])
    _, _, scores = oracle_lib.select_row(s, f, 1, T - 1, kc, 0, 0, 0)
    sb = [1.0 * a + 0.5 * b for a, b in blockv]
    for j in range(1, 8):  # candidates [1, 9 - 2] = [1, 7]
        want = max(sb[j], (sb[j - 1] + sb[j]) / 2, (sb[j] + sb[j + 1]) / 2)
        assert scores[j] == want, (j, scores[j], want)
    assert np.isnan(scores[0]) and np.isnan(scores[8]) and np.isnan(scores[9])


@pytest.mark.parametrize("T,n_q,n_init,n_local,lw,sw", [
    (1280, 300, 1, 2, 64, 64), (1000, 1000, 0, 3, 64, 64), (1024, 200, 1, 2, 32, 16), (777, 97, 2, 1, 32, 16)])
def test_score_max_matches_bruteforce(oracle_lib, T, n_q, n_init, n_local, lw, sw):
    """Each row's largest candidate score against dense numpy scores, the explicit (block, window)
    overlap mask of the brute-force selection, and the candidate range [n_init, blk - n_local]."""
    s = grid_shape(oracle_lib, 2, 2, T, n_init + n_local + 3, lw, sw, n_init, n_local)
    f = rnd_u16((2, 2, n_q, 128), 75, 1)
    k = rnd_u16((2, 2, T, 128), 75, 2)
    kc = oracle_lib.compress_keys(s, k, T, 0, s.nc_cap)
    q_pos0 = T - n_q
    got = oracle_lib.forecast_score_max(s, f, n_q, q_pos0, kc)
    _, _, pooled = brute.select_rows_pooled(f, kc, q_pos0, s.k_total, n_init, n_local, lw, sw)
    for r in range(n_q):
        hi = (q_pos0 + r) // 64 - n_local
        if hi < n_init:
            assert np.all(got[:, :, r] == -np.inf)
            continue
        want = pooled[:, :, r, n_init: hi + 1].max(axis=-1)
        assert np.allclose(got[:, :, r], want, rtol=1e-12, atol=1e-12), r


def test_score_max_closed_form_skips_forced_blocks(oracle_lib):
    """One key per block with known scores (F = e0): the maximum is the largest score among the
    candidates; larger keys planted in the initial and local blocks never count, and rows whose
    candidate range is empty get -inf."""
    T, D = 640, 2
    s = oracle_lib.Shape(batch=1, n_kv_heads=1, group_size=1, head_dim=D, block_size=64, n_init=1, n_local=2,
                         k_total=4, t_cap=T, nc_cap=10)
    to = lambda a: np.array(a, np.float32).view(np.uint32).__rshift__(16).astype(np.uint16)
    val = [50.0, 3.0, -1.0, 7.0, 2.0, -4.0, 6.0, 1.0, 40.0, 60.0]  # blocks 0, 8, 9 are forced at p = 639
    kc = to([[[[v, 0.0] for v in val]]])
    pos = [0, 100, 191, 192, 300, 320, 450, 512, 575, 576, 639]
    f = to([[[[1.0, 0.0]] * len(pos)]])
    for i, p in enumerate(pos):
        got = oracle_lib.forecast_score_max(s, np.ascontiguousarray(f[:, :, i:i + 1]), 1, p, kc)[0, 0, 0]
        hi = p // 64 - 2
        want = max(val[1: hi + 1]) if hi >= 1 else -np.inf
        assert got == want, (p, got, want)


def test_select_pooled_window_visibility_at_the_local_edge(oracle_lib):
    """With one local block the last candidate j = blk - 1 has a window reaching 16 tokens into the
    query's own block; it counts only once those tokens exist (p >= 64 (j + 1) + 15)."""
    T, D = 512, 2
    s = oracle_lib.Shape(batch=1, n_kv_heads=1, group_size=1, head_dim=D, block_size=64, n_init=1, n_local=1,
                         k_total=3, t_cap=T, nc_cap=(T - 32) // 16 + 1, cmp_kernel=32, cmp_stride=16)
    to = lambda a: np.array(a, np.float32).view(np.uint32).__rshift__(16).astype(np.uint16)
    kf = np.zeros((T, D), np.float32)
    kf[4 * 64:4 * 64 + 16, 0] = 1.0   # block 4's first 16 keys: only windows 15 and 16 see them
    k = to([[kf]])
    kc = oracle_lib.compress_keys(s, k, T, 0, s.nc_cap)
    f = to([[[[1.0, 0.0]]]])
    # query in block 4: candidates [1, 3]; window 15 = tokens [240, 272) straddles blocks 3 and 4
    for p, want in [(4 * 64 + 14, 0.0), (4 * 64 + 15, 0.5), (4 * 64 + 40, 0.5)]:
        _, _, scores = oracle_lib.select_row(s, f, 1, p, kc, 0, 0, 0)
        assert scores[3] == want, (p, scores[3])
        assert scores[1] == 0.0 and scores[2] == 0.0


def test_select_pooled_planted_recall_and_decode_equals_prefill(oracle_lib):
    """Planted blocks carry the full shift in their inner windows, so the paper's grid still finds
    them all; decode at position p selects what prefill row p selects."""
    T = 4096
    w = inputs.Workload("g", batch=1, seq_len=T, n_q=64, n_kv_heads=2, group_size=4, k_total=16, seed=77)
    case = inputs.make_case(w)
    s = grid_shape(oracle_lib, 1, 2, T, 16)
    k = inputs.to_u16(case["k"])
    kc = oracle_lib.compress_keys(s, k, T, 0, s.nc_cap)
    f_last = inputs.to_u16(case["f"])[:, :, -1:]
    sel, cnt = oracle_lib.forecast_select(s, f_last, 1, T - 1, kc)
    for m in range(2):
        chosen = set(sel[0, m, 0, : cnt[0, m, 0]].tolist())
        planted = set(int(j) for j in case["plants"][0, m])
        assert planted <= chosen, (planted - chosen)
    f = inputs.to_u16(case["f"])
    selp, cntp = oracle_lib.forecast_select(s, f, 64, T - 64, kc)
    for r in (0, 17, 63):
        seld, cntd = oracle_lib.forecast_select(s, np.ascontiguousarray(f[:, :, r:r + 1]), 1, T - 64 + r, kc)
        assert np.array_equal(seld[:, :, 0], selp[:, :, r]) and np.array_equal(cntd[:, :, 0], cntp[:, :, r])


def test_grid_shapes_outside_the_family_are_refused(oracle_lib):
    import oracle
    k = np.zeros((1, 1, 256, 128), np.uint16)
    for lw, sw in [(128, 64), (32, 48), (48, 20), (16, 32)]:
        s = grid_shape(oracle_lib, 1, 1, 256, 4, lw, sw)
        with pytest.raises(oracle.OracleError) as e:
            oracle_lib.compress_keys(s, k, 256, 0, 1)
        assert e.value.rc == oracle.ERR_UNSUPPORTED


def test_select_block_budget_from_paper(oracle_lib):
    """The paper's MiniCPM settings: 64-token blocks, 1 initial block, a 2048-token (32-block)
    local window and one overall budget of 96 blocks.  Read with k counting the forced blocks,
    a 128K decode attends exactly 96 blocks, 63 of them chosen by score."""
    with open(os.path.join(GOLDEN, "paper_block_budget.json")) as fh:
        g = json.load(fh)
    n_local = g["local_window_tokens"] // g["block_size_tokens"]
    T = 131072
    nb = T // g["block_size_tokens"]
    s = oracle_lib.Shape(batch=1, n_kv_heads=1, group_size=1, head_dim=128, n_init=g["initial_blocks"],
                         n_local=n_local, k_total=g["overall_block_budget"], t_cap=T, nc_cap=nb)
    f = rnd_u16((1, 1, 1, 128), 26, 1)
    kc = rnd_u16((1, 1, nb, 128), 26, 4)
    sel, cnt, scores = oracle_lib.select_row(s, f, 1, T - 1, kc, 0, 0, 0)
    assert cnt == 96
    chosen = [j for j in sel[:cnt] if g["initial_blocks"] <= j < nb - n_local]
    assert len(chosen) == 96 - 1 - 32
    cand_scores = scores[~np.isnan(scores)]
    kth = np.sort(cand_scores)[::-1][len(chosen) - 1]
    assert all(scores[j] >= kth for j in chosen)


# ----------------------------------------------------------------------------- attention (Eq. 1, Eq. 5)

def _attn_case(oracle_lib, T, n_q, k_total, G=4, H=2, B=1, seed=30, n_local=2):
    D = 128
    s = shape_for(oracle_lib, B, H, G, T, k_total, 1, n_local, t_cap=-(-T // 64) * 64)
    tc = s.t_cap
    q = rnd_u16((B, H * G, n_q, D), seed, 0)
    k = rnd_u16((B, H, tc, D), seed, 2)
    v = rnd_u16((B, H, tc, D), seed, 3)
    f = rnd_u16((B, H, n_q, D), seed, 1)
    nb = max((T - 1) // 64, 1)
    kc = oracle_lib.compress_keys(shape_for(oracle_lib, B, H, G, T, k_total, 1, n_local, t_cap=tc, nc_cap=nb),
                                  k, T, 0, T // 64 if T // 64 <= nb else nb)
    s = shape_for(oracle_lib, B, H, G, T, k_total, 1, n_local, t_cap=tc, nc_cap=nb)
    sel, cnt = oracle_lib.forecast_select(s, f, n_q, T - n_q, kc)
    return s, q, k, v, sel, cnt


@pytest.mark.parametrize("T,n_q,k_total", [(4096, 1, 16), (1000, 1, 5), (640, 130, 4), (130, 130, 3), (64, 64, 3)])
def test_attend_matches_dense_masked(oracle_lib, T, n_q, k_total):
    s, q, k, v, sel, cnt = _attn_case(oracle_lib, T, n_q, k_total)
    scale = 1.0 / math.sqrt(128)
    got = oracle_lib.sparse_attn(s, q, n_q, T - n_q, k, v, 0, sel, cnt, scale)
    want = brute.attend_dense_masked(q, k[:, :, :T], v[:, :, :T], sel, cnt, T - n_q, 4, scale)
    np.testing.assert_allclose(got, want, rtol=0, atol=1e-12)


def test_attend_is_invariant_to_selection_order(oracle_lib):
    T = 4096
    s, q, k, v, sel, cnt = _attn_case(oracle_lib, T, 1, 16, B=2)
    scale = 1.0 / math.sqrt(128)
    base = oracle_lib.sparse_attn(s, q, 1, T - 1, k, v, 0, sel, cnt, scale)
    rng = np.random.default_rng(0)
    perm = sel.copy()
    for b in range(2):
        for m in range(2):
            n = cnt[b, m, 0]
            perm[b, m, 0, :n] = rng.permutation(perm[b, m, 0, :n])
    got = oracle_lib.sparse_attn(s, q, 1, T - 1, k, v, 0, perm, cnt, scale)
    np.testing.assert_allclose(got, base, rtol=0, atol=1e-13)


def test_attend_equals_causal_sdpa_when_k_covers_all(oracle_lib):
    """With every causal block attended, sparse attention is dense causal attention; the library
    routine is torch's scaled_dot_product_attention in float64 with GQA expansion."""
    T, G, H = 320, 4, 2
    s, q, k, v, sel, cnt = _attn_case(oracle_lib, T, T, 8, G=G, H=H)
    assert np.all(cnt[0, :, T - 1] == T // 64)
    scale = 1.0 / math.sqrt(128)
    got = oracle_lib.sparse_attn(s, q, T, 0, k, v, 0, sel, cnt, scale)
    qt = torch.from_numpy(brute.bf16_bits_to_f64(q))
    kt = torch.from_numpy(brute.bf16_bits_to_f64(k)).repeat_interleave(G, dim=1)
    vt = torch.from_numpy(brute.bf16_bits_to_f64(v)).repeat_interleave(G, dim=1)
    want = torch.nn.functional.scaled_dot_product_attention(qt, kt, vt, is_causal=True, scale=scale).numpy()
    np.testing.assert_allclose(got, want, rtol=0, atol=1e-12)


def test_attend_zero_query_is_mean_of_attended_values(oracle_lib):
    T = 1000
    s, q, k, v, sel, cnt = _attn_case(oracle_lib, T, 1, 5)
    q[:] = 0
    got = oracle_lib.sparse_attn(s, q, 1, T - 1, k, v, 0, sel, cnt, 0.0883883)
    vv = brute.bf16_bits_to_f64(v)
    for h in range(8):
        m = h // 4
        toks = [t for j in sel[0, m, 0, : cnt[0, m, 0]] for t in range(64 * j, 64 * j + 64) if t <= T - 1]
        np.testing.assert_allclose(got[0, h, 0], vv[0, m, toks].mean(axis=0), rtol=0, atol=1e-12)


def test_attend_single_hot_key_closed_form(oracle_lib):
    """D = 2, sm_scale = 1, decode at p = 100 over blocks {0, 1} (tokens 0..100).  All keys are 0
    except K[5] = (2, 0); Q = (1, 0); V[t] = (t, 1).  Then
      o_0 = (5 e^2 + (5050 - 5)) / (e^2 + 100),  o_1 = 1."""
    s = oracle_lib.Shape(batch=1, n_kv_heads=1, group_size=1, head_dim=2, n_init=1, n_local=1, k_total=2,
                         t_cap=128, nc_cap=2)
    to = lambda a: torch.tensor(a, dtype=torch.float32).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    kf = np.zeros((128, 2), np.float32)
    kf[5, 0] = 2.0
    vf = np.stack([np.arange(128, dtype=np.float32), np.ones(128, np.float32)], axis=1)
    q = to([[[[1.0, 0.0]]]])
    k = to(kf.reshape(1, 1, 128, 2))
    v = to(vf.reshape(1, 1, 128, 2))
    sel = np.array([[[[0, 1]]]], np.int16)
    cnt = np.array([[[2]]], np.int16)
    out = oracle_lib.attend_row(s, q, 1, 100, k, v, 0, sel, cnt, 1.0, 0, 0, 0)
    e2 = math.exp(2.0)
    assert abs(out[0] - (5 * e2 + 5045.0) / (e2 + 100.0)) < 1e-12
    assert abs(out[1] - 1.0) < 1e-15


def test_attend_constant_values(oracle_lib):
    T = 777
    s, q, k, v, sel, cnt = _attn_case(oracle_lib, T, 1, 6)
    v[:] = v[0, 0, 0, 0]
    got = oracle_lib.sparse_attn(s, q, 1, T - 1, k, v, 0, sel, cnt, 0.1)
    np.testing.assert_allclose(got, brute.bf16_bits_to_f64(v[0, 0, 0, :1])[0], rtol=0, atol=1e-13)


def test_staging_mode_matches_cache_mode_and_gather_is_bitwise(oracle_lib):
    T = 4096
    s, q, k, v, sel, cnt = _attn_case(oracle_lib, T, 1, 16, B=2)
    st_k, st_v = oracle_lib.gather_blocks(s, k, v, sel[:, :, 0], cnt[:, :, 0])
    for b in range(2):
        for m in range(2):
            for i in range(cnt[b, m, 0]):
                j = sel[b, m, 0, i]
                assert np.array_equal(st_k[b, m, i], k[b, m, 64 * j:64 * j + 64])
                assert np.array_equal(st_v[b, m, i], v[b, m, 64 * j:64 * j + 64])
    scale = 1.0 / math.sqrt(128)
    a = oracle_lib.sparse_attn(s, q, 1, T - 1, k, v, 0, sel, cnt, scale)
    b_ = oracle_lib.sparse_attn(s, q, 1, T - 1, st_k, st_v, 1, sel, cnt, scale)
    np.testing.assert_allclose(a, b_, rtol=0, atol=1e-13)


def test_out_of_range_entries_are_skipped(oracle_lib):
    T = 1000
    s, q, k, v, sel, cnt = _attn_case(oracle_lib, T, 1, 5)
    scale = 0.09
    base = oracle_lib.sparse_attn(s, q, 1, T - 1, k, v, 0, sel, cnt, scale)
    sel2 = np.concatenate([sel, np.full(sel.shape[:-1] + (2,), 99, np.int16)], axis=-1)
    sel2[..., -2] = -7
    s2 = oracle_lib.Shape(**{**s.__dict__, "k_total": s.k_total + 2})
    cnt2 = (cnt + 2).astype(np.int16)
    got = oracle_lib.sparse_attn(s2, q, 1, T - 1, k, v, 0, np.ascontiguousarray(sel2), cnt2, scale)
    np.testing.assert_allclose(got, base, rtol=0, atol=0)


def test_duplicate_entries_are_attended_once(oracle_lib):
    # The attended tokens are the union of the set's blocks (Eq. 1, Eq. 5): listing a block again
    # adds nothing.  Checked against the dense masked attention, whose mask is a set by
    # construction, on decode and multi-row cases.
    for T, n_q, k_total in ((4096, 1, 16), (640, 70, 6)):
        s, q, k, v, sel, cnt = _attn_case(oracle_lib, T, n_q, k_total)
        scale = 1.0 / math.sqrt(128)
        extra = 3
        sel2 = np.concatenate([sel, sel[..., :extra]], axis=-1)  # re-list the first three entries
        rng = np.random.default_rng(7)
        sel2 = np.take_along_axis(sel2, rng.permuted(np.tile(np.arange(sel2.shape[-1]), sel2.shape[:-1] + (1,)),
                                                      axis=-1), axis=-1)
        # rows whose count is below k_total hold -1 pads among the first entries; keep cnt = all slots
        s2 = oracle_lib.Shape(**{**s.__dict__, "k_total": s.k_total + extra})
        cnt2 = np.full(cnt.shape, s2.k_total, np.int16)
        got = oracle_lib.sparse_attn(s2, q, n_q, T - n_q, k, v, 0, np.ascontiguousarray(sel2), cnt2, scale)
        want = brute.attend_dense_masked(q, k[:, :, :T], v[:, :, :T], sel, cnt, T - n_q, 4, scale)
        np.testing.assert_allclose(got, want, rtol=0, atol=1e-12)


# ----------------------------------------------------------------------------- InfLLM-V2 multi-head selector

MH_SCALE = 1.0 / math.sqrt(128)


def mh_shape(oracle, B, H, G, T, k_total, lw=64, sw=64, n_init=1, n_local=2, D=128):
    return oracle.Shape(batch=B, n_kv_heads=H, group_size=G, head_dim=D, block_size=64, n_init=n_init,
                        n_local=n_local, k_total=k_total, t_cap=T, nc_cap=(T - lw) // sw + 1, cmp_kernel=lw,
                        cmp_stride=sw)


def test_multihead_worked_example(oracle_lib):
    with open(os.path.join(GOLDEN, "multihead_worked_example.json")) as fh:
        g = json.load(fh)
    to = lambda a: torch.tensor(a, dtype=torch.float32).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    kc = to([[g["k_cmp"]]])
    q = to([[[row] for row in g["q_heads"]]])  # [1][2 heads][1 row][2]
    for k_total, key in ((4, "k4"), (5, "k5")):
        s = oracle_lib.Shape(batch=1, n_kv_heads=1, group_size=2, head_dim=2, n_init=1, n_local=2, k_total=k_total,
                             t_cap=448, nc_cap=7)
        sel, cnt, scores, _ = oracle_lib.multihead_select_row(s, q, 1, g["query_position"], kc, math.log(2.0), 0, 0, 0)
        assert cnt == g["expected"][key]["cnt"]
        assert list(sel[:cnt]) == g["expected"][key]["sel"]
        for j, num in g["expected"]["block_scores_num_over_299"].items():
            assert scores[int(j)] == pytest.approx(num / 299, rel=1e-14)


@pytest.mark.parametrize("T,n_q,k_total,G,n_init,n_local,lw,sw", [
    (1024, 1, 6, 4, 1, 2, 64, 64), (1024, 200, 6, 4, 1, 2, 64, 64), (1500, 150, 7, 2, 0, 3, 64, 64),
    (1024, 1, 6, 4, 1, 2, 32, 16), (1500, 260, 7, 4, 2, 1, 32, 16), (1280, 150, 5, 3, 1, 2, 32, 16),
    (900, 90, 5, 16, 1, 1, 32, 16)])
def test_multihead_matches_bruteforce(oracle_lib, T, n_q, k_total, G, n_init, n_local, lw, sw):
    H = 2
    s = mh_shape(oracle_lib, 1, H, G, T, k_total, lw, sw, n_init, n_local)
    q = rnd_u16((1, H * G, n_q, 128), 81, G)
    k = rnd_u16((1, H, T, 128), 82, 0)
    kc = oracle_lib.compress_keys(s, k, T, 0, s.nc_cap)
    sel, cnt = oracle_lib.multihead_select(s, q, n_q, T - n_q, kc, MH_SCALE)
    bsel, bcnt, pooled = brute.multihead_select_rows(q, kc, T - n_q, k_total, n_init, n_local, G, MH_SCALE, lw, sw)
    assert np.array_equal(cnt, bcnt)
    assert np.array_equal(sel, bsel)
    for r in (0, n_q // 2, n_q - 1):
        _, _, sc, _ = oracle_lib.multihead_select_row(s, q, n_q, T - n_q, kc, MH_SCALE, 0, 1, r)
        ok = ~np.isnan(sc)
        np.testing.assert_allclose(sc[ok], pooled[0, 1, r, :len(sc)][ok], rtol=1e-12, atol=0)


@pytest.mark.parametrize("lw,sw", [(64, 64), (32, 16)])
def test_multihead_single_head_ranks_like_a_forecast_row(oracle_lib, lw, sw):
    """With one head per group the softmax is increasing in the score and the max-pool commutes
    with it, so the multi-head selector picks exactly what the plain dot-product selector picks
    when the Forecast row is that head's query."""
    T, n_q = 1500, 120
    s = mh_shape(oracle_lib, 2, 2, 1, T, 9, lw, sw)
    q = rnd_u16((2, 2, n_q, 128), 83, 0)
    k = rnd_u16((2, 2, T, 128), 83, 1)
    kc = oracle_lib.compress_keys(s, k, T, 0, s.nc_cap)
    sel, cnt = oracle_lib.multihead_select(s, q, n_q, T - n_q, kc, MH_SCALE)
    fsel, fcnt = oracle_lib.forecast_select(s, q, n_q, T - n_q, kc)
    assert np.array_equal(cnt, fcnt) and np.array_equal(sel, fsel)


def test_multihead_zero_query_is_uniform_and_takes_lowest_blocks(oracle_lib):
    """q = 0: every head's softmax is uniform, every candidate ties, the lowest indices win."""
    T, n_q, G = 2048, 40, 4
    s = mh_shape(oracle_lib, 1, 2, G, T, 8, 32, 16)
    q = np.zeros((1, 2 * G, n_q, 128), np.uint16)
    kc = oracle_lib.compress_keys(s, rnd_u16((1, 2, T, 128), 84, 0), T, 0, s.nc_cap)
    sel, cnt = oracle_lib.multihead_select(s, q, n_q, T - n_q, kc, MH_SCALE)
    for r in range(n_q):
        p = T - n_q + r
        blk = p // 64
        forced = {0, blk - 1, blk}
        want = sorted(forced | set(range(1, 1 + 8 - 3)))
        assert list(sel[0, 0, r, :cnt[0, 0, r]]) == want
        _, _, sc, _ = oracle_lib.multihead_select_row(s, q, n_q, T - n_q, kc, MH_SCALE, 0, 0, r)
        n_vis = (p + 1 - 32) // 16 + 1
        assert np.allclose(sc[1:blk - 1], G / n_vis, rtol=1e-14)


def test_multihead_head_order_and_decode_equals_prefill(oracle_lib):
    """Permuting the heads inside each group leaves the selection unchanged; a decode call at
    position p selects what row p of a multi-row call selects."""
    T, n_q, G = 1800, 64, 4
    s = mh_shape(oracle_lib, 1, 2, G, T, 7, 32, 16)
    q = rnd_u16((1, 2 * G, n_q, 128), 85, 0)
    kc = oracle_lib.compress_keys(s, rnd_u16((1, 2, T, 128), 85, 1), T, 0, s.nc_cap)
    sel, cnt = oracle_lib.multihead_select(s, q, n_q, T - n_q, kc, MH_SCALE)
    perm = np.concatenate([m * G + np.array([2, 0, 3, 1]) for m in range(2)])
    psel, pcnt = oracle_lib.multihead_select(s, np.ascontiguousarray(q[:, perm]), n_q, T - n_q, kc, MH_SCALE)
    assert np.array_equal(sel, psel) and np.array_equal(cnt, pcnt)
    for r in (0, 31, n_q - 1):
        dsel, dcnt = oracle_lib.multihead_select(s, np.ascontiguousarray(q[:, :, r:r + 1]), 1, T - n_q + r, kc,
                                                 MH_SCALE)
        assert np.array_equal(dsel[:, :, 0], sel[:, :, r]) and np.array_equal(dcnt[:, :, 0], cnt[:, :, r])


def test_multihead_needs_every_complete_window(oracle_lib):
    """The softmax runs over every key complete at the query, the local blocks' included, so the
    compressed-key capacity must hold them all."""
    import oracle
    T = 1024
    s = mh_shape(oracle_lib, 1, 1, 4, T, 6, 32, 16)
    short = oracle.Shape(**{**s.__dict__, "nc_cap": s.nc_cap - 1})
    q = rnd_u16((1, 4, 1, 128), 86, 0)
    kc = np.zeros((1, 1, s.nc_cap, 128), np.uint16)
    with pytest.raises(oracle.OracleError):
        oracle_lib.multihead_select(short, q, 1, T - 1, np.ascontiguousarray(kc[:, :, :-1]), MH_SCALE)
    with pytest.raises(oracle.OracleError):
        oracle_lib.multihead_select(s, q, 1, T - 1, kc, 0.0)


# ----------------------------------------------------------------------------- NOSI step reuse: staging plan

def _plan_shape(oracle, B=2, H=3, k_total=12, t_cap=64 * 200):
    return oracle.Shape(batch=B, n_kv_heads=H, group_size=4, head_dim=128, n_init=1, n_local=2, k_total=k_total,
                        t_cap=t_cap, nc_cap=t_cap // 64)


def _random_set(rng, p, k_total, prev=None, keep=0.7, vary=False):
    """An attended set for position p: initial block 0, the two local blocks, and top-k slots drawn
    from the candidates, keeping about `keep` of the previous step's choices.  With vary, the set
    sometimes leaves a few slots unused (the plan must handle any set, not only full ones)."""
    blk = p // 64
    forced = {0, blk - 1, blk}
    cand = list(range(1, blk - 1))
    n_sel = min(k_total - 3, len(cand))
    if vary:
        n_sel -= int(rng.integers(0, 4))
    chosen = set()
    if prev is not None:
        old = [j for j in prev if 1 <= j <= blk - 2]
        chosen = set(j for j in old if rng.random() < keep)
    rest = [j for j in cand if j not in chosen]
    rng.shuffle(rest)
    while len(chosen) < n_sel:
        chosen.add(rest.pop())
    chosen = set(sorted(chosen)[:n_sel])
    full = sorted(forced | chosen)
    sel = np.full(k_total, -1, np.int16)
    sel[:len(full)] = full
    return sel, len(full)


def test_writeback_places_new_rows_and_touches_nothing_else(oracle_lib):
    """The write-back is a placement: numpy slice assignment of the new rows at [pos0, pos0 + n)
    of every (batch, group) pool row; every other position keeps its bytes; a range past t_cap
    is refused."""
    s = shape_for(oracle_lib, 2, 3, 4, 640, 8)
    pool_k = rnd_u16((2, 3, 640, 128), 81, 1)
    pool_v = rnd_u16((2, 3, 640, 128), 81, 2)
    new_k = rnd_u16((2, 3, 5, 128), 81, 3)
    new_v = rnd_u16((2, 3, 5, 128), 81, 4)
    hk, hv = oracle_lib.writeback_kv(s, new_k, new_v, 5, 300, pool_k, pool_v)
    want_k, want_v = pool_k.copy(), pool_v.copy()
    want_k[:, :, 300:305] = new_k
    want_v[:, :, 300:305] = new_v
    assert np.array_equal(hk, want_k) and np.array_equal(hv, want_v)
    with pytest.raises(oracle_lib.OracleError):
        oracle_lib.writeback_kv(s, new_k, new_v, 5, 636, pool_k, pool_v)


def test_stage_append_completes_the_gather_of_the_appended_cache(oracle_lib):
    """Alg. 2 appends the decoded token to the cache.  Gathering a cache that does not hold the
    token yet and then appending the token to the staged copy of its block gives exactly the
    gather of the cache that holds it; a slot listing the block twice gets it twice, other slots
    keep their bytes, and a row whose set lacks the token's block is not written."""
    B, H, K, T = 2, 3, 6, 640
    s = shape_for(oracle_lib, B, H, 4, T, K)
    p = 64 * 7 + 21
    full_k = rnd_u16((B, H, T, 128), 91, 1)
    full_v = rnd_u16((B, H, T, 128), 91, 2)
    pool_k, pool_v = full_k.copy(), full_v.copy()
    pool_k[:, :, p:] = 0x7FC0  # not written back yet: a NaN pattern
    pool_v[:, :, p:] = 0x7FC0
    sel = np.full((B, H, K), -1, np.int16)
    cnt = np.zeros((B, H), np.int16)
    sets = {(0, 0): [0, 3, 6, 7], (0, 1): [7, 1, 7], (0, 2): [2, 5], (1, 0): [0, 7], (1, 1): [7], (1, 2): [0, 4, 6, 7]}
    for (b, m), blocks in sets.items():
        sel[b, m, :len(blocks)] = blocks
        cnt[b, m] = len(blocks)
    stage_k, stage_v = oracle_lib.gather_blocks(s, pool_k, pool_v, sel, cnt)
    sk, sv = oracle_lib.stage_append_kv(s, full_k[:, :, p], full_v[:, :, p], p, sel, cnt, stage_k, stage_v)
    want_k, want_v = oracle_lib.gather_blocks(s, full_k, full_v, sel, cnt, stage_k.copy(), stage_v.copy())
    for (b, m), blocks in sets.items():
        for slot, j in enumerate(blocks):
            if j == p // 64:  # the token's own block: equal to the appended cache up to p
                assert np.array_equal(sk[b, m, slot, :p % 64 + 1], want_k[b, m, slot, :p % 64 + 1])
                assert np.array_equal(sv[b, m, slot, :p % 64 + 1], want_v[b, m, slot, :p % 64 + 1])
                assert np.all(sk[b, m, slot, p % 64 + 1:] == 0x7FC0)  # later rows untouched
            else:
                assert np.array_equal(sk[b, m, slot], stage_k[b, m, slot])
                assert np.array_equal(sk[b, m, slot], want_k[b, m, slot])
    assert np.array_equal(sk[0, 2], stage_k[0, 2]) and np.array_equal(sv[0, 2], stage_v[0, 2])  # no own block
    with pytest.raises(oracle_lib.OracleError):
        oracle_lib.stage_append_kv(s, full_k[:, :, 0], full_v[:, :, 0], T, sel, cnt, stage_k, stage_v)


def test_plan_first_step_is_the_plain_gather_layout(oracle_lib):
    s = _plan_shape(oracle_lib)
    rng = np.random.default_rng(90)
    sel = np.full((2, 3, 12), -1, np.int16)
    cnt = np.zeros((2, 3), np.int16)
    for b in range(2):
        for m in range(3):
            sel[b, m], cnt[b, m] = _random_set(rng, 3000, 12)
    blk = np.full((2, 3, 12), -1, np.int16)
    ln = np.zeros((2, 3, 12), np.int16)
    fetch, staged, n_fetch = oracle_lib.plan_staging(s, sel, cnt, 3000, blk, ln)
    assert np.array_equal(fetch, sel) and np.array_equal(staged, sel) and np.array_equal(n_fetch, cnt)
    assert np.array_equal(blk, sel)
    # the open block 3000 // 64 = 46 holds tokens 2944 .. 3000: 57 of them; complete blocks 64
    want_len = np.where(sel == 46, 57, np.where(sel >= 0, 64, 0))
    assert np.array_equal(ln, want_len)


def test_plan_same_set_inside_a_block_fetches_only_the_open_block(oracle_lib):
    s = _plan_shape(oracle_lib, B=1, H=1)
    sel, n = _random_set(np.random.default_rng(91), 5000, 12)
    sel, cnt = sel[None, None], np.array([[n]], np.int16)
    blk = np.full((1, 1, 12), -1, np.int16)
    ln = np.zeros((1, 1, 12), np.int16)
    oracle_lib.plan_staging(s, sel, cnt, 5000, blk, ln)
    for p in (5001, 5002, 5003):  # same block 78, one more token each step
        fetch, staged, n_fetch = oracle_lib.plan_staging(s, sel, cnt, p, blk, ln)
        assert n_fetch[0, 0] == 1 and set(fetch[fetch >= 0].tolist()) == {5000 // 64}
        assert sorted(staged[staged >= 0].tolist()) == sorted(sel[0, 0, :n].tolist())


def test_plan_emulated_cache_serves_exact_tokens_with_minimal_fetches(oracle_lib):
    """A 300-step decode with drifting sets.  An emulated staging store records, per slot, the
    token values copied at fetch time (tokens after the fetch position read as unwritten).  Every
    step: the attended slots hold exactly the step's set, each of them holds every token its block
    contributes up to p, fetches land in the lowest free slots in ascending block order, and the
    number of fetches is |S| minus the blocks of S that the previous step attended with enough
    tokens (the NOSI rule)."""
    K = 12
    s = _plan_shape(oracle_lib, B=1, H=2, k_total=K)
    rng = np.random.default_rng(92)
    blk = np.full((1, 2, K), -1, np.int16)
    ln = np.zeros((1, 2, K), np.int16)
    store = [[None] * K for _ in range(2)]  # (block, tuple of token ids written when fetched)
    prev_sets = [None, None]
    prev_valid = [dict(), dict()]  # block -> tokens staged, for the previous step's attended slots
    p = 1500
    for step in range(300):
        p += 1 if step % 7 else 30  # mostly one token, sometimes a jump
        sel = np.full((1, 2, K), -1, np.int16)
        cnt = np.zeros((1, 2), np.int16)
        for m in range(2):
            sel[0, m], cnt[0, m] = _random_set(rng, p, K, prev_sets[m], vary=True)
        fetch, staged, n_fetch = oracle_lib.plan_staging(s, sel, cnt, p, blk, ln)
        for m in range(2):
            S = set(sel[0, m, :cnt[0, m]].tolist())
            # fetches copy the tokens written so far (<= p) of their block
            for t in range(K):
                j = int(fetch[0, m, t])
                if j >= 0:
                    store[m][t] = (j, tuple(x for x in range(64 * j, 64 * j + 64) if x <= p))
            att = {int(staged[0, m, t]): t for t in range(K) if staged[0, m, t] >= 0}
            assert set(att) == S and len(att) == len(S)
            for j, t in att.items():
                held_j, toks = store[m][t]
                assert held_j == j
                assert set(range(64 * j, min(64 * j + 64, p + 1))) <= set(toks), f"slot {t} stale for block {j}"
            need = lambda j: min(64, p + 1 - 64 * j)
            reusable = {j for j, n_tok in prev_valid[m].items() if j in S and n_tok >= need(j)}
            assert n_fetch[0, m] == len(S) - len(reusable)
            slots = [t for t in range(K) if fetch[0, m, t] >= 0]
            blocks = [int(fetch[0, m, t]) for t in slots]
            assert blocks == sorted(blocks)
            kept = {t for t in range(K) if staged[0, m, t] >= 0 and fetch[0, m, t] < 0}
            assert slots == [t for t in range(K) if t not in kept][:len(slots)]
            prev_valid[m] = {int(staged[0, m, t]): len(store[m][t][1]) for t in range(K) if staged[0, m, t] >= 0}
            prev_sets[m] = sorted(S)


# ----------------------------------------------------------------------------- indexer-training KL (Eq. 6-7)

def _kl_case(oracle, T, n_q, G, seed, n_init=1, n_local=2, D=128):
    """Synthetic tensors of one group: queries, fine (2, 1) and prediction (32, 16) compressed
    keys of the same random keys, Forecast rows."""
    s = oracle.Shape(batch=1, n_kv_heads=1, group_size=G, head_dim=D, block_size=64, n_init=n_init,
                     n_local=n_local, k_total=8, t_cap=T, nc_cap=(T - 32) // 16 + 1, cmp_kernel=32, cmp_stride=16)
    st_ = oracle.Shape(**{**s.__dict__, "nc_cap": T - 1, "cmp_kernel": 2, "cmp_stride": 1})
    k = rnd_u16((1, 1, T, D), seed, 0)
    kct = oracle.compress_keys(st_, k, T, 0, T - 1)
    kcp = oracle.compress_keys(s, k, T, 0, s.nc_cap)
    q = rnd_u16((1, G, n_q, D), seed, 1)
    f = rnd_u16((1, 1, n_q, D), seed, 2)
    return s, q, kct, f, kcp


@pytest.mark.parametrize("T,n_q,G,k_top,n_local", [(640, 3, 4, 6, 2), (1000, 2, 2, 10, 1), (777, 2, 16, 3, 3)])
def test_kl_matches_bruteforce_and_gradient_matches_finite_differences(oracle_lib, T, n_q, G, k_top, n_local):
    s, q, kct, f, kcp = _kl_case(oracle_lib, T, n_q, G, 95 + G, n_local=n_local)
    b64 = brute.bf16_bits_to_f64
    for r in range(n_q):
        p = T - n_q + r
        loss, dF, sel, n_sel = oracle_lib.indexer_kl_row(s, q, kct, 2, 1, f, kcp, n_q, T - n_q, MH_SCALE, k_top, 0, 0, r)
        qr, fr = b64(q[0, :, r]), b64(f[0, 0, r])
        bl, bS = brute.indexer_kl(qr, b64(kct[0, 0]), fr, b64(kcp[0, 0]), p, MH_SCALE, k_top, 1, n_local)
        assert loss == pytest.approx(bl, rel=1e-10, abs=1e-14)
        assert list(sel[:n_sel]) == list(bS)
        assert loss >= 0.0
        # central differences of the brute-force loss in every coordinate of the Forecast row
        eps = 1e-4
        fd = np.empty(128)
        for d in range(128):
            e = np.zeros(128)
            e[d] = eps
            lp_, _ = brute.indexer_kl(qr, b64(kct[0, 0]), fr + e, b64(kcp[0, 0]), p, MH_SCALE, k_top, 1, n_local)
            lm_, _ = brute.indexer_kl(qr, b64(kct[0, 0]), fr - e, b64(kcp[0, 0]), p, MH_SCALE, k_top, 1, n_local)
            fd[d] = (lp_ - lm_) / (2 * eps)
        np.testing.assert_allclose(dF, fd, rtol=1e-5, atol=1e-9)


def test_kl_uniform_closed_forms(oracle_lib):
    """q = 0 and F = 0: both distributions are uniform over the positions, the target's top-k is the
    lowest candidate positions, and the partitions agree exactly, so the loss and gradient vanish.
    k_top = 0 leaves only the rest bucket: loss 0 for any F."""
    T, G = 900, 4
    s, q, kct, f, kcp = _kl_case(oracle_lib, T, 1, G, 96)
    zq, zf = np.zeros_like(q), np.zeros_like(f)
    loss, dF, sel, n_sel = oracle_lib.indexer_kl_row(s, zq, kct, 2, 1, zf, kcp, 1, T - 1, MH_SCALE, 5, 0, 0, 0)
    assert loss == pytest.approx(0.0, abs=1e-15) and np.allclose(dF, 0.0, atol=1e-15)
    assert list(sel) == [4, 5, 6, 7, 8]  # positions 4.. start at token 64 (block 1, the first candidate)
    loss, dF, _, n_sel = oracle_lib.indexer_kl_row(s, q, kct, 2, 1, f, kcp, 1, T - 1, MH_SCALE, 0, 0, 0, 0)
    assert n_sel == 0 and loss == pytest.approx(0.0, abs=1e-15) and np.allclose(dF, 0.0, atol=1e-15)


def test_kl_head_order_does_not_matter(oracle_lib):
    T, G = 700, 4
    s, q, kct, f, kcp = _kl_case(oracle_lib, T, 2, G, 97)
    a = oracle_lib.indexer_kl_row(s, q, kct, 2, 1, f, kcp, 2, T - 2, MH_SCALE, 6, 0, 0, 1)
    qp = np.ascontiguousarray(q[:, [3, 1, 0, 2]])
    b = oracle_lib.indexer_kl_row(s, qp, kct, 2, 1, f, kcp, 2, T - 2, MH_SCALE, 6, 0, 0, 1)
    assert a[0] == pytest.approx(b[0], rel=1e-13) and np.allclose(a[1], b[1], rtol=1e-12, atol=1e-16)
    assert list(a[2]) == list(b[2])
