"""Comparison helpers for the GPU parity tests.

Selection: cnt must match exactly; the block sets must match, except that a block chosen by only
one side is accepted when the oracle's score of every such block lies within the tie window of
the oracle's k-th chosen score s_k.  The window is max(1e-3 |s_k|, gamma_128 * sum_d |F_d K~_id|),
with i the compressed key that gives block j its (max-pooled) score:
the relative window the acceptance bar states, floored by the a-priori float32 error bound of a
128-term dot product (gamma_n = n u / (1 - n u), u = 2^-24), which only matters when s_k ~ 0.
All scores and bounds here come from the oracle's inputs and the oracle's scores.

Attention: two bars, both against the oracle's float64 output on the same attended set.
  * the acceptance bar: |o_gpu - o_oracle| <= 2e-2 absolute (bf16 inputs, float32 accumulation);
  * a tight bar from the arithmetic, per output element: with w = sum_t p_t |v_t| / sum_t p_t
    (the oracle's attention over |V|, same set), a kernel that rounds P to bf16 before P V
    (relative 2^-8 per weight, in the numerator and the normaliser alike), sums at most 16384
    terms in float32 (gamma_n < 2^-10, which also covers the float32 logits, |dz| < 2^-14) and
    rounds the output to bf16 (2^-8 of |o|) stays within
        |o_gpu - o| <= (2^-8 + 2^-10) w + (2^-7 + 2^-10) |o|        (first order).
    Kernels that keep P in float32 sit far inside it.  On block-coded V (every token of block j
    holds a 0/1 code of j) w = |o|, so the bar is relative, about 1.4 % of each element, while
    leaving out or exchanging one attended block moves some element by all of that block's mass.
"""
from __future__ import annotations

import numpy as np

import brute
import oracle

ATTN_ATOL = 2e-2
TIGHT_W = 2.0 ** -8 + 2.0 ** -10
TIGHT_O = 2.0 ** -7 + 2.0 ** -10
REL_TIE = 1e-3
_U = 2.0 ** -24
GAMMA_128 = 128 * _U / (1 - 128 * _U)


def compare_selection(oshape, f_u16, kc_u16, n_q, q_pos0, gpu_sel, gpu_cnt, rows):
    """rows: iterable of (b, m, r).  Returns (n_rows, n_tie_swaps).  Raises AssertionError."""
    f64 = None
    n_rows = n_swaps = 0
    for (b, m, r) in rows:
        ref, cnt, scores, wins = oracle.select_row_windows(oshape, f_u16, n_q, q_pos0, kc_u16, b, m, r)
        g = gpu_sel[b, m, r]
        gc = int(gpu_cnt[b, m, r])
        assert gc == cnt, f"row {(b, m, r)}: cnt {gc} != oracle {cnt}"
        assert np.all(g[cnt:] == -1), f"row {(b, m, r)}: padding"
        gs = g[:cnt]
        assert np.all(np.diff(gs.astype(np.int64)) > 0), f"row {(b, m, r)}: not strictly ascending: {gs}"
        n_rows += 1
        if np.array_equal(gs, ref[:cnt]):
            continue
        A, R = set(gs.tolist()), set(ref[:cnt].tolist())
        only = (A - R) | (R - A)
        cand = ~np.isnan(scores)
        for j in only:
            assert 0 <= j < len(scores) and cand[j], f"row {(b, m, r)}: non-candidate block {j} differs"
        chosen_ref = [j for j in R if cand[j]]
        s_k = min(scores[j] for j in chosen_ref)
        if f64 is None:
            f64 = brute.bf16_bits_to_f64(f_u16)
            kc64 = brute.bf16_bits_to_f64(kc_u16)
        # the floor for block j uses the compressed key that gives j its (max-pooled) score
        absdot = lambda j: float(np.abs(f64[b, m, r] * kc64[b, m, wins[j]]).sum())
        for j in only:
            win = max(REL_TIE * abs(s_k), GAMMA_128 * absdot(j))
            assert abs(scores[j] - s_k) <= win, (
                f"row {(b, m, r)}: block {j} (score {scores[j]:.6g}) differs beyond the tie window "
                f"{win:.3g} of s_k = {s_k:.6g}")
        n_swaps += 1
    return n_rows, n_swaps


def compare_multihead_selection(oshape, q_u16, kc_u16, n_q, q_pos0, sm_scale, gpu_sel, gpu_cnt, rows):
    """The multi-head selector's sets against the oracle's.  Its block scores are sums of softmax
    weights, all > 0, computed on the GPU in float32 (exp2 domain) from float32 dot products, so
    a relative error of a few 1e-6 covers them; a block chosen by only one side is accepted when
    its oracle score lies within 1e-3 of s_k relatively.  Returns (n_rows, n_tie_swaps)."""
    n_rows = n_swaps = 0
    for (b, m, r) in rows:
        ref, cnt, scores, _ = oracle.multihead_select_row(oshape, q_u16, n_q, q_pos0, kc_u16, sm_scale, b, m, r)
        g = gpu_sel[b, m, r]
        gc = int(gpu_cnt[b, m, r])
        assert gc == cnt, f"row {(b, m, r)}: cnt {gc} != oracle {cnt}"
        assert np.all(g[cnt:] == -1), f"row {(b, m, r)}: padding"
        gs = g[:cnt]
        assert np.all(np.diff(gs.astype(np.int64)) > 0), f"row {(b, m, r)}: not strictly ascending: {gs}"
        n_rows += 1
        if np.array_equal(gs, ref[:cnt]):
            continue
        A, R = set(gs.tolist()), set(ref[:cnt].tolist())
        cand = ~np.isnan(scores)
        only = (A - R) | (R - A)
        for j in only:
            assert 0 <= j < len(scores) and cand[j], f"row {(b, m, r)}: non-candidate block {j} differs"
        s_k = min(scores[j] for j in R if cand[j])
        for j in only:
            assert abs(scores[j] - s_k) <= REL_TIE * s_k, (
                f"row {(b, m, r)}: block {j} (score {scores[j]:.6g}) differs beyond the tie window of "
                f"s_k = {s_k:.6g}")
        n_swaps += 1
    return n_rows, n_swaps


def abs_bits(v_u16):
    """|V| as bf16 bits (sign cleared): the oracle's attention over it gives the tight bar's w."""
    return np.asarray(v_u16, np.uint16) & np.uint16(0x7FFF)


def tight_bar(o_ref, w):
    return TIGHT_W * np.asarray(w, np.float64) + TIGHT_O * np.abs(o_ref)


def compare_attention(o_gpu, o_ref, what="", w=None):
    """Both bars (the tight one only when w, the oracle's attention over |V|, is given).  Returns
    the largest |o_gpu - o_ref|; compare_attention.last_tight_ratio holds the largest error over
    the tight bar (0 without w)."""
    o_gpu = np.asarray(o_gpu, np.float64)
    err = np.abs(o_gpu - o_ref)
    worst = float(err.max()) if err.size else 0.0
    assert np.all(np.isfinite(o_gpu)), f"{what}: non-finite output"
    assert worst <= ATTN_ATOL, f"{what}: max |o - oracle| = {worst:.3g} > {ATTN_ATOL}"
    compare_attention.last_tight_ratio = 0.0
    if w is not None:
        bar = tight_bar(o_ref, w)
        over = err > bar
        if np.any(over):
            i = np.unravel_index(int(np.argmax(err - bar)), err.shape)
            raise AssertionError(f"{what}: {int(over.sum())} elements beyond the tight bar, e.g. at {i}: "
                                 f"|{o_gpu[i]:.6g} - {o_ref[i]:.6g}| > {bar[i]:.3g}")
        nz = bar > 0
        compare_attention.last_tight_ratio = float((err[nz] / bar[nz]).max()) if np.any(nz) else 0.0
    return worst


compare_attention.last_tight_ratio = 0.0
