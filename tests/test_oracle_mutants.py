"""Plant plausible mistakes in copies of the oracle (on the CPU) and check that the pins catch
each one: a flipped sort direction, a dropped softmax scale, an off-by-one local window, a
causal mask that lets the next token in, an init block left out of the candidates' exclusion,
a swapped operand index in the score, a rounding mode change in the compressed keys, and a block
listed twice in a set being attended twice; on the paper's (32, 16) grid, a max-pool that uses
windows not yet complete at the query and one that skips the windows straddling a block edge; in
the InfLLM-V2 multi-head selector, raw scores summed without the softmax, an unnormalised
softmax, a single head standing for the group, a softmax normalised over fewer keys and a
dropped temperature; in the staging plan of step-to-step reuse, a staged block kept whatever
its token count, freed slots left holding their old blocks, and fetches placed from the top; in
the indexer-training loss, a sum instead of the max-pool of the target, a dropped rest bucket, a
flipped gradient sign and local positions left among the candidates; in the row maximum of the
scores, a local or an initial block counted as a candidate."""
import math
import os

import numpy as np
import pytest

import brute
import oracle
from paper_2606_04511_amd import inputs

MUTANTS = {
    "sort_ascending": ("if (a->score > b->score) return -1;", "if (a->score < b->score) return -1;"),
    "index_tiebreak_reversed": ("return (a->block > b->block) - (a->block < b->block);",
                                "return (a->block < b->block) - (a->block > b->block);"),
    "scale_dropped": ("z[t] = sm_scale * dot;", "z[t] = dot;"),
    "local_window_short": ("int64_t local_lo = blk - s->n_local + 1;", "int64_t local_lo = blk - s->n_local + 2;"),
    "causal_leak": ("if (t > p) break;", "if (t > p + 1) break;"),
    "candidates_include_init": ("const int64_t cand_lo = s->n_init,", "const int64_t cand_lo = 0,"),
    "score_wrong_operand": ("sparda_ref_bf16_to_f64(kc[i * D + d])", "sparda_ref_bf16_to_f64(kc[d * D + i % D])"),
    "compress_truncates": ("double q = nearbyint(ldexp(m, 8));", "double q = floor(ldexp(m, 8));"),
    "compress_wrong_divisor": ("sum / (double)lw", "sum / (double)(lw - 1)"),
    "duplicate_attended_twice": ("if (seen) continue;", "(void)seen;"),
    "pool_ignores_visibility": ("if (hi > w_vis) hi = w_vis;", "(void)w_vis;"),
    "pool_inner_windows_only": ("int64_t lo = (j * L - lw) / sw + 1;", "int64_t lo = (j * L) / sw;"),
    "multihead_raw_sum": ("shared[i] += exp(z[i] - zmax) / denom;", "shared[i] += z[i];"),
    "multihead_unnormalised": ("shared[i] += exp(z[i] - zmax) / denom;", "shared[i] += exp(z[i] - zmax);"),
    "multihead_first_head_only": ("for (int64_t h = m * G; h < (m + 1) * G; ++h)",
                                  "for (int64_t h = m * G; h < m * G + 1; ++h)"),
    "multihead_softmax_over_fewer_keys": ("for (int64_t i = 0; i < n_vis; ++i) denom += exp(z[i] - zmax);",
                                          "for (int64_t i = 1; i < n_vis - 2; ++i) denom += exp(z[i] - zmax);"),
    "multihead_temperature_dropped": ("z[i] = sm_scale * acc;", "z[i] = acc;"),
    "plan_ignores_token_count": ("if (srow[i] == j && !held[i] && len[t] >= need) {",
                                 "if (srow[i] == j && !held[i]) {"),
    "plan_keeps_unattended_slots": ("      if (att[t] < 0) {\n        blk[t] = -1;", "      if (0) {\n        blk[t] = -1;"),
    "kl_sum_pool": ("&& shared[i] > best) best = shared[i];", ") best += shared[i];"),
    "kl_no_rest_bucket": ("if (t_rest > 0.0) kl += t_rest * log(t_rest / R);", "(void)R;"),
    "kl_gradient_sign": ("? P[w] - T[w] / t_total :", "? T[w] / t_total - P[w] :"),
    "kl_local_positions_are_candidates": ("cand_tok_hi = (blk - s->n_local + 1) * L;", "cand_tok_hi = (blk + 1) * L;"),
    "score_max_counts_a_local_block": ("for (int64_t j = s->n_init; j <= p / L - s->n_local; ++j) {",
                                       "for (int64_t j = s->n_init; j <= p / L - s->n_local + 1; ++j) {"),
    "score_max_counts_the_init_block": ("for (int64_t j = s->n_init; j <= p / L - s->n_local; ++j) {",
                                        "for (int64_t j = 0; j <= p / L - s->n_local; ++j) {"),
    "plan_fills_from_the_top": ("while (next_free < K && kept[next_free]) ++next_free;",
                                "while (next_free < K && kept[K - 1 - next_free]) ++next_free;"),
}


def _pins_pass(o) -> bool:
    """A compact subset of the pins: brute-force select, dense-masked attention, compress."""
    rng_seed = 41
    T, n_q, H, G = 640, 130, 2, 4
    s = o.Shape(batch=1, n_kv_heads=H, group_size=G, head_dim=128, n_init=1, n_local=2, k_total=5, t_cap=640,
                nc_cap=9)
    u = lambda shp, tid: inputs.to_u16(inputs.normal_bf16(shp, rng_seed, tid))
    k = u((1, H, 640, 128), 2)
    v = u((1, H, 640, 128), 3)
    q = u((1, H * G, n_q, 128), 0)
    f = u((1, H, n_q, 128), 1)
    try:
        kc = o.compress_keys(s, k, 640, 0, 9)
        if not np.array_equal(kc, brute.compress(k, 9)):
            return False
        sel, cnt = o.forecast_select(s, f, n_q, T - n_q, kc)
        bsel, bcnt, _ = brute.select_rows(f, kc, T - n_q, 5, 1, 2)
        if not (np.array_equal(sel, bsel) and np.array_equal(cnt, bcnt)):
            return False
        scale = 1.0 / math.sqrt(128)
        got = o.sparse_attn(s, q, n_q, T - n_q, k, v, 0, bsel, bcnt, scale)
        want = brute.attend_dense_masked(q, k, v, bsel, bcnt, T - n_q, G, scale)
        if not np.allclose(got, want, rtol=0, atol=1e-12):
            return False
        # a block listed twice is attended once (the attended tokens are a union of blocks)
        sd = np.ascontiguousarray(np.concatenate([bsel[..., 2:], bsel], axis=-1))
        s3 = o.Shape(**{**s.__dict__, "k_total": sd.shape[-1]})
        got = o.sparse_attn(s3, q, n_q, T - n_q, k, v, 0, sd, np.full(bcnt.shape, sd.shape[-1], np.int16), scale)
        if not np.allclose(got, want, rtol=0, atol=1e-12):
            return False
        # the hand-worked tie (test_select_worked_example_with_tie): block 1 beats block 3
        to = lambda a: np.array(a, np.float32).view(np.uint32).__rshift__(16).astype(np.uint16)
        s2 = o.Shape(batch=1, n_kv_heads=1, group_size=1, head_dim=2, n_init=1, n_local=2, k_total=5,
                     t_cap=448, nc_cap=7)
        kc2 = to([[[[9, 9], [1, 0], [0, 4], [2, -2], [-1, 0], [9, 9], [9, 9]]]])
        sel2, cnt2, _ = o.select_row(s2, to([[[[1.0, 0.5]]]]), 1, 447, kc2, 0, 0, 0)
        if not (cnt2 == 5 and list(sel2) == [0, 1, 2, 5, 6]):
            return False
        # the paper's (32, 16) grid: compress and max-pooled selection against the brute force,
        # with one local block so that the visibility of the edge windows matters
        sg = o.Shape(batch=1, n_kv_heads=H, group_size=G, head_dim=128, n_init=1, n_local=1, k_total=4, t_cap=640,
                     nc_cap=39, cmp_kernel=32, cmp_stride=16)
        kcg = o.compress_keys(sg, k, 640, 0, 39)
        if not np.array_equal(kcg, brute.compress_windows(k, 39, 32, 16)):
            return False
        selg, cntg = o.forecast_select(sg, f, n_q, T - n_q, kcg)
        bselg, bcntg, _ = brute.select_rows_pooled(f, kcg, T - n_q, 4, 1, 1, 32, 16)
        if not (np.array_equal(selg, bselg) and np.array_equal(cntg, bcntg)):
            return False
        # the InfLLM-V2 multi-head selector: the hand-worked example, then brute force on both grids
        s5 = o.Shape(batch=1, n_kv_heads=1, group_size=2, head_dim=2, n_init=1, n_local=2, k_total=5, t_cap=448,
                     nc_cap=7)
        kc5 = to([[[[1, 0], [0, 1], [1, 1], [2, 0], [0, 2], [1, -1], [0, 0]]]])
        sel5, cnt5, _, _ = o.multihead_select_row(s5, to([[[[1, 0]], [[0, 1]]]]), 1, 447, kc5, math.log(2.0), 0, 0, 0)
        if not (cnt5 == 5 and list(sel5) == [0, 3, 4, 5, 6]):
            return False
        s10 = o.Shape(**{**s.__dict__, "nc_cap": 10})  # the softmax reads every complete block
        kc10 = o.compress_keys(s10, k, 640, 0, 10)
        for shp, kcx, lw, sw, n_local in ((s10, kc10, 64, 64, 2), (sg, kcg, 32, 16, 1)):
            msel, mcnt = o.multihead_select(shp, q, n_q, T - n_q, kcx, scale)
            bsel, bcnt, _ = brute.multihead_select_rows(q, kcx, T - n_q, shp.k_total, 1, n_local, G, scale, lw, sw)
            if not (np.array_equal(msel, bsel) and np.array_equal(mcnt, bcnt)):
                return False
        # the staging plan of step-to-step reuse
        import test_oracle_pins as pins
        pins.test_plan_first_step_is_the_plain_gather_layout(o)
        pins.test_plan_emulated_cache_serves_exact_tokens_with_minimal_fetches(o)
        # the indexer-training loss
        pins.test_kl_matches_bruteforce_and_gradient_matches_finite_differences(o, 640, 2, 4, 6, 2)
        pins.test_kl_matches_bruteforce_and_gradient_matches_finite_differences(o, 1000, 1, 2, 10, 1)
        pins.test_kl_uniform_closed_forms(o)
        # the scoring contraction alone: each row's largest candidate score
        pins.test_score_max_closed_form_skips_forced_blocks(o)
        pins.test_score_max_matches_bruteforce(o, 1024, 200, 1, 2, 32, 16)
        return True
    except (oracle.OracleError, AssertionError, IndexError, TypeError):
        return False


def test_unmutated_oracle_passes(oracle_lib):
    assert _pins_pass(oracle_lib)


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_planted_mistake_is_caught(oracle_lib, tmp_path, name):
    old, new = MUTANTS[name]
    src = oracle.source_text()
    assert src.count(old) == 1, f"mutation anchor for {name} not unique"
    path = oracle.build_variant(src.replace(old, new), os.path.join(str(tmp_path), f"mut_{name}.so"))
    with oracle.use_library(path):
        assert not _pins_pass(oracle), f"mutant {name} slipped past the pins"
