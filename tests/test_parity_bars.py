"""The attention parity bars can see a wrong block (CPU, oracle only).

On block-coded V (inputs.block_coded_values) and rows shaped like every block-coded GPU case
(same context, set size, group size and local window), leaving out any one attended block, or
exchanging it for a causal block the row does not attend, moves some output element by more
than ten times the tight bar of tests/parity.py.  A kernel that reads one wrong block, skips one
or counts one twice therefore fails the GPU comparison.  On the N(0, 1) values of the other
fixtures the same perturbation is checked against the 2e-2 acceptance bar for contrast (it can
hide there, which is why the block-coded fixtures exist).
"""
import math

import numpy as np
import pytest

import oracle
from paper_2606_04511_amd import inputs
from parity import abs_bits, tight_bar

SCALE = 1.0 / math.sqrt(128)

# T, G, k_total, n_local, positions (decode form: one row at each position)
CASES = [
    (131072, 4, 64, 2, [131071]),
    (32768, 4, 64, 2, [32767]),
    (131072, 4, 96, 2, [131071]),
    (131072, 16, 96, 32, [131071]),
    (32768, 16, 64, 2, [32767]),
    (32768, 4, 64, 2, [4096, 20000]),
    (32768, 16, 96, 32, [4096, 27001]),
]


def _row_inputs(T, G, k_total, n_local, seed):
    w = inputs.Workload("bars", batch=1, seq_len=T, n_q=1, n_kv_heads=1, group_size=G, k_total=k_total,
                        n_local=n_local, seed=seed)
    f = inputs.normal_bf16((1, 1, 1, 128), seed, 1)
    k = inputs.keys_with_plants(w, f[:, :, 0, :], T, seed=seed)
    q = inputs.normal_bf16((1, G, 1, 128), seed, 0)
    return inputs.to_u16(q), inputs.to_u16(f), inputs.to_u16(k)


@pytest.mark.parametrize("T,G,k_total,n_local,positions", CASES)
def test_one_block_change_exceeds_ten_tight_bars(T, G, k_total, n_local, positions):
    q16, f16, k16 = _row_inputs(T, G, k_total, n_local, 8800 + T // 1024 + G + k_total)
    v16 = inputs.to_u16(inputs.block_coded_values(1, 1, T))
    nb = T // 64
    o = oracle.Shape(batch=1, n_kv_heads=1, group_size=G, k_total=k_total, t_cap=T, nc_cap=nb, n_local=n_local)
    kc = oracle.compress_keys(o, k16, T, 0, nb)
    rng = np.random.default_rng(3)
    for p in positions:
        # the row's set as the Forecast selection at p chooses it (f's last row stands for row p)
        sel, cnt = oracle.forecast_select(o, f16, 1, p, kc)
        n = int(cnt[0, 0, 0])
        S = sel[0, 0, 0, :n].astype(np.int64)
        attend = lambda blocks: oracle.sparse_attn(
            o, q16, 1, p, k16, v16, 0, np.pad(np.asarray(blocks, np.int16), (0, k_total - len(blocks)),
                                              constant_values=-1)[None, None, None],
            np.array([[[len(blocks)]]], np.int16), SCALE)
        ref = attend(S)
        wab = oracle.sparse_attn(o, q16, 1, p, k16, abs_bits(v16), 0, sel, cnt, SCALE)
        bar = tight_bar(ref, wab)
        unattended = np.setdiff1d(np.arange(p // 64 + 1), S)
        worst_margin = np.inf
        for i, j in enumerate(S):
            dropped = np.delete(S, i)
            moved = np.max(np.abs(attend(dropped) - ref) / np.maximum(bar, 1e-30))
            worst_margin = min(worst_margin, moved)
            assert moved > 10, f"p={p}: leaving out block {j} moves the output by only {moved:.2f} tight bars"
            if len(unattended):
                jj = int(rng.choice(unattended))
                swapped = np.sort(np.append(dropped, jj))
                moved = np.max(np.abs(attend(swapped) - ref) / np.maximum(bar, 1e-30))
                worst_margin = min(worst_margin, moved)
                assert moved > 10, f"p={p}: block {jj} for {j} moves the output by only {moved:.2f} tight bars"
        assert n == min(k_total, p // 64 + 1)
        print(f"T={T} G={G} k={k_total} local={n_local} p={p}: every one-block change moves the output by "
              f">= {worst_margin:.1f} tight bars")


def test_tight_bar_on_gaussian_values_is_near_observed_errors():
    """On N(0, 1) values the tight bar is a few 1e-3 (observed GPU errors are about 5e-4), well
    inside the 2e-2 acceptance bar."""
    T, G, k_total = 32768, 4, 64
    q16, f16, k16 = _row_inputs(T, G, k_total, 2, 77)
    v16 = inputs.to_u16(inputs.normal_bf16((1, 1, T, 128), 77, 3))
    nb = T // 64
    o = oracle.Shape(batch=1, n_kv_heads=1, group_size=G, k_total=k_total, t_cap=T, nc_cap=nb)
    kc = oracle.compress_keys(o, k16, T, 0, nb)
    sel, cnt = oracle.forecast_select(o, f16, 1, T - 1, kc)
    ref = oracle.sparse_attn(o, q16, 1, T - 1, k16, v16, 0, sel, cnt, SCALE)
    wab = oracle.sparse_attn(o, q16, 1, T - 1, k16, abs_bits(v16), 0, sel, cnt, SCALE)
    bar = tight_bar(ref, wab)
    assert 1e-3 < float(bar.max()) < 6e-3
    assert np.all(wab >= np.abs(ref) - 1e-12)  # w bounds |o| (a weighted mean of |v| vs of v)
