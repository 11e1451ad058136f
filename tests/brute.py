"""Brute-force numpy/torch references used only to pin the oracle on tiny inputs.

These are written independently of the C oracle: vectorised dense algebra, a full sort instead
of a partial selection, dense attention with the complement of the attended set masked to -inf,
and an integer bit-manipulation bf16 rounding instead of frexp/nearbyint.
"""
from __future__ import annotations

import numpy as np
import torch

BLOCK = 64


def bf16_bits_to_f64(a: np.ndarray) -> np.ndarray:
    return (a.astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def f64_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float64 -> bf16 (nearest, ties to even) with integer arithmetic on the float64 bits.
    Normal-range finite values only (enough for the pins)."""
    x = np.asarray(x, np.float64)
    bits = x.view(np.uint64).astype(np.uint64)
    sign = (bits >> np.uint64(63)).astype(np.uint64)
    exp = ((bits >> np.uint64(52)) & np.uint64(0x7FF)).astype(np.int64)
    man = (bits & np.uint64((1 << 52) - 1)).astype(np.uint64)
    out = np.zeros(x.shape, np.uint16)
    zero = (exp == 0) & (man == 0)
    normal = ~zero
    # keep 7 explicit mantissa bits, 45 bits are rounded away
    keep = man >> np.uint64(45)
    rest = man & np.uint64((1 << 45) - 1)
    half = np.uint64(1 << 44)
    round_up = (rest > half) | ((rest == half) & ((keep & np.uint64(1)) == np.uint64(1)))
    keep = keep + round_up.astype(np.uint64)
    e = exp - 1023 + 127
    carry = keep == np.uint64(128)
    keep = np.where(carry, np.uint64(0), keep)
    e = np.where(carry, e + 1, e)
    assert np.all((e[normal] > 0) & (e[normal] < 255)), "pins use normal-range values only"
    val = (sign << np.uint64(15)) | (e.astype(np.uint64) << np.uint64(7)) | keep
    out[normal] = val[normal].astype(np.uint16)
    out[zero] = (sign[zero] << np.uint64(15)).astype(np.uint16)
    return out


def compress(k_bits: np.ndarray, n_blocks: int) -> np.ndarray:
    """k: uint16 [B][H][T][D] -> uint16 [B][H][n_blocks][D]."""
    k = bf16_bits_to_f64(k_bits[:, :, : n_blocks * BLOCK])
    B, H, _, D = k.shape
    mean = k.reshape(B, H, n_blocks, BLOCK, D).mean(axis=3)
    return f64_to_bf16_bits(mean)


def compress_windows(k_bits: np.ndarray, n_win: int, lw: int, sw: int) -> np.ndarray:
    """Windows of lw keys at stride sw: k uint16 [B][H][T][D] -> uint16 [B][H][n_win][D]."""
    k = bf16_bits_to_f64(k_bits)
    idx = np.arange(n_win)[:, None] * sw + np.arange(lw)[None, :]  # [n_win][lw] token indices
    mean = k[:, :, idx, :].mean(axis=3)
    return f64_to_bf16_bits(mean)


def select_rows_pooled(f_bits, kc_bits, q_pos0, k_total, n_init, n_local, lw, sw):
    """Dense window scores, a max over the windows that overlap each block and are complete at the
    row's position (an explicit mask over all (block, window) pairs), then a full lexsort.
    kc: [B][H][n_win][D] windows.  Returns sel, cnt and the pooled block scores (NaN where a
    block has no visible window)."""
    f = bf16_bits_to_f64(f_bits)
    kc = bf16_bits_to_f64(kc_bits)
    wsc = np.einsum("bhqd,bhid->bhqi", f, kc)
    return _pool_and_select(wsc, q_pos0, k_total, n_init, n_local, lw, sw)


def multihead_select_rows(q_bits, kc_bits, q_pos0, k_total, n_init, n_local, G, scale, lw=64, sw=64):
    """The InfLLM-V2 multi-head selector by brute force: dense scaled scores of every query head
    against every window, -inf on windows not complete at the row's position, scipy's softmax
    over the windows, the sum over each group's G heads, then the same dense max-pool mask and
    lexsort as select_rows_pooled.  q: [B][Hq][n_q][D], kc: [B][Hkv][n_win][D]."""
    from scipy.special import softmax
    q = bf16_bits_to_f64(q_bits)
    kc = bf16_bits_to_f64(kc_bits)
    B, Hq, n_q, D = q.shape
    Hkv, n_win = kc.shape[1], kc.shape[2]
    assert Hq == Hkv * G
    kc_h = np.repeat(kc, G, axis=1)  # query head h reads KV head h // G
    z = scale * np.einsum("bhqd,bhid->bhqi", q, kc_h)
    start = np.arange(n_win) * sw
    pos = q_pos0 + np.arange(n_q)
    visible = (start[None, :] + lw) <= (pos[:, None] + 1)  # [n_q][n_win]
    z = np.where(visible[None, None], z, -np.inf)
    a = np.zeros_like(z)
    for r in range(n_q):
        if visible[r].any():
            a[:, :, r, :] = softmax(z[:, :, r, :], axis=-1)
    shared = a.reshape(B, Hkv, G, n_q, n_win).sum(axis=2)
    return _pool_and_select(shared, q_pos0, k_total, n_init, n_local, lw, sw)


def _pool_and_select(wsc, q_pos0, k_total, n_init, n_local, lw, sw):
    B, H, n_q, n_win = wsc.shape
    start = np.arange(n_win) * sw
    sel = np.full((B, H, n_q, k_total), -1, np.int16)
    cnt = np.zeros((B, H, n_q), np.int16)
    n_blk = (q_pos0 + n_q - 1) // BLOCK + 1
    pooled = np.full((B, H, n_q, n_blk), np.nan)
    for r in range(n_q):
        p = q_pos0 + r
        blk = p // BLOCK
        for j in range(blk + 1):
            overl = (start < (j + 1) * BLOCK) & (start + lw > j * BLOCK) & (start + lw <= p + 1)
            if overl.any():
                pooled[:, :, r, j] = wsc[:, :, r, overl].max(axis=-1)
        forced = set(range(0, min(n_init, blk + 1))) | set(range(max(0, blk - n_local + 1), blk + 1))
        cand = np.array([j for j in range(blk + 1) if j not in forced and j >= n_init and j <= blk - n_local],
                        np.int64)
        n_take = min(k_total - len(forced), len(cand))
        for b in range(B):
            for h in range(H):
                if len(cand):
                    s = pooled[b, h, r, cand]
                    order = np.lexsort((cand, -s))
                    chosen = set(cand[order[:n_take]].tolist())
                else:
                    chosen = set()
                full = sorted(forced | chosen)
                sel[b, h, r, : len(full)] = full
                cnt[b, h, r] = len(full)
    return sel, cnt, pooled


def select_rows(f_bits, kc_bits, q_pos0, k_total, n_init, n_local):
    """Dense scores + full lexsort.  f: [B][H][n_q][D], kc: [B][H][nc][D].
    Returns sel [B][H][n_q][k_total] (ascending, -1 padded), cnt [B][H][n_q], scores [B][H][n_q][nc]."""
    f = bf16_bits_to_f64(f_bits)
    kc = bf16_bits_to_f64(kc_bits)
    scores = np.einsum("bhqd,bhjd->bhqj", f, kc)
    B, H, n_q, _ = f.shape
    nc = kc.shape[2]
    sel = np.full((B, H, n_q, k_total), -1, np.int16)
    cnt = np.zeros((B, H, n_q), np.int16)
    for r in range(n_q):
        p = q_pos0 + r
        blk = p // BLOCK
        forced = set(range(0, min(n_init, blk + 1))) | set(range(max(0, blk - n_local + 1), blk + 1))
        cand = np.array([j for j in range(blk + 1) if j not in forced and j >= n_init and j <= blk - n_local],
                        np.int64)
        n_take = min(k_total - len(forced), len(cand))
        for b in range(B):
            for h in range(H):
                if len(cand):
                    s = scores[b, h, r, cand]
                    order = np.lexsort((cand, -s))  # primary: -score, secondary: index
                    chosen = set(cand[order[:n_take]].tolist())
                else:
                    chosen = set()
                full = sorted(forced | chosen)
                sel[b, h, r, : len(full)] = full
                cnt[b, h, r] = len(full)
    del nc
    return sel, cnt, scores


def attend_dense_masked(q_bits, k_bits, v_bits, sel, cnt, q_pos0, group_size, sm_scale):
    """Dense attention over all T tokens with every token outside the attended set masked.
    q: [B][Hq][n_q][D]; k, v: [B][Hkv][T][D]; returns float64 [B][Hq][n_q][D]."""
    q = torch.from_numpy(bf16_bits_to_f64(q_bits))
    k = torch.from_numpy(bf16_bits_to_f64(k_bits))
    v = torch.from_numpy(bf16_bits_to_f64(v_bits))
    B, Hq, n_q, D = q.shape
    T = k.shape[2]
    kx = k.repeat_interleave(group_size, dim=1)
    vx = v.repeat_interleave(group_size, dim=1)
    logits = torch.einsum("bhqd,bhtd->bhqt", q, kx) * sm_scale
    allowed = torch.zeros(B, Hq, n_q, T, dtype=torch.bool)
    tok = torch.arange(T)
    for b in range(B):
        for h in range(Hq):
            m = h // group_size
            for r in range(n_q):
                p = q_pos0 + r
                blocks = [int(j) for j in sel[b, m, r, : int(cnt[b, m, r])] if 0 <= int(j) <= p // BLOCK]
                if blocks:
                    in_set = torch.zeros(T, dtype=torch.bool)
                    for j in blocks:
                        in_set[j * BLOCK:(j + 1) * BLOCK] = True
                    allowed[b, h, r] = in_set & (tok <= p)
    logits = logits.masked_fill(~allowed, float("-inf"))
    w = torch.softmax(logits, dim=-1)
    w = torch.nan_to_num(w, nan=0.0)
    return torch.einsum("bhqt,bhtd->bhqd", w, vx).numpy()


def indexer_kl(q_rows, kct, f_row, kcp, p, sm_scale, k_top, n_init, n_local, lt=2, st=1, lp=32, sp=16):
    """The indexer-training KL of one query row, densely: q_rows [G][D], kct [n_t][D] and kcp
    [n_p][D] as float64 arrays (compressed keys), f_row [D] float64 (a real vector, so that the
    loss can be differentiated numerically).  Target: scipy softmax per head over the fine windows
    complete at p, summed, then a dense (position, window) containment mask and a max; prediction:
    scipy softmax over the positions complete at p; the top-k by a lexsort over the positions
    inside candidate blocks; the (k+1)-bucket KL.  Returns (loss, sorted selected positions)."""
    from scipy.special import softmax
    n_pos = (p + 1 - lp) // sp + 1 if p + 1 >= lp else 0
    n_tw = (p + 1 - lt) // st + 1 if p + 1 >= lt else 0
    a = softmax(sm_scale * (q_rows @ kct[:n_tw].T), axis=-1).sum(axis=0)  # [n_tw]
    i = np.arange(n_tw)
    w = np.arange(n_pos)
    inside = (i[None, :] * st >= w[:, None] * sp) & (i[None, :] * st + lt <= w[:, None] * sp + lp)
    T = np.where(inside, a[None, :], 0.0).max(axis=1)
    P = softmax(sm_scale * (kcp[:n_pos] @ f_row))
    blk = p // 64
    cand = (w * sp >= n_init * 64) & (w * sp + lp <= (blk - n_local + 1) * 64)
    cw = w[cand]
    order = np.lexsort((cw, -T[cw]))
    S = np.sort(cw[order[:k_top]])
    t = T / T.sum()
    mask = np.zeros(n_pos, bool)
    mask[S] = True
    t_rest, R = t[~mask].sum(), P[~mask].sum()
    kl = float(np.sum(t[mask] * np.log(t[mask] / P[mask])))
    if t_rest > 0:
        kl += float(t_rest * np.log(t_rest / R))
    return kl, S
