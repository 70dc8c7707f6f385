"""The oracle pins must catch plausible mistakes.

Each case plants one mistake into the oracle (on the CPU, by swapping one of
its functions for a wrong variant written here) and checks that at least one
pin of test_oracle_pins fails.
"""

import math

import numpy as np
import pytest

import oracle as O
import oracle.spla_oracle as OS
import test_oracle_pins as P
import test_oracle_windows as W


def _patch(monkeypatch, name, fn):
    monkeypatch.setattr(OS, name, fn)
    monkeypatch.setattr(O, name, fn)


def _expect_failure(*pins):
    failed = 0
    for pin, args in pins:
        try:
            pin(*args)
        except (AssertionError, ValueError, IndexError):
            failed += 1
    assert failed > 0, "planted mistake went unnoticed"


def _lbm(half=0.5, s_pow=2, with_count=True, with_scale=True):
    def f(q, mean, var, counts, s, first_order=False):
        ss = s if with_scale else 1.0
        ell = ss * (q @ mean.T)
        if with_count:
            ell = ell + np.log(counts.astype(float))[None, :]
        if not first_order:
            ell = ell + np.log1p(half * ss ** s_pow * ((q * q) @ var.T))
        return ell
    return f


def test_dropped_half_in_taylor_term(monkeypatch):
    _patch(monkeypatch, "log_block_mass", _lbm(half=1.0))
    _expect_failure((P.test_x5_pm_eps_blocks_closed_form, (0.3,)),
                    (P.test_x6_taylor_error_is_third_order_with_known_coefficient, ()))


def test_scale_not_squared_in_taylor_term(monkeypatch):
    _patch(monkeypatch, "log_block_mass", _lbm(s_pow=1))
    _expect_failure((P.test_x5_pm_eps_blocks_closed_form, (0.3,)))


def test_missing_block_count(monkeypatch):
    _patch(monkeypatch, "log_block_mass", _lbm(with_count=False))
    _expect_failure((P.test_x4_identical_keys_taylor_mass_is_exact, ()))


def test_missing_scale_in_block_score(monkeypatch):
    _patch(monkeypatch, "log_block_mass", _lbm(with_scale=False))
    _expect_failure((P.test_x4_identical_keys_taylor_mass_is_exact, ()))


def test_sample_instead_of_population_variance(monkeypatch):
    orig = OS.block_stats

    def bad(K, L, B):
        mean, var, counts = orig(K, L, B)
        return mean, var * counts[:, None] / np.maximum(counts[:, None] - 1, 1), counts
    _patch(monkeypatch, "block_stats", bad)
    _expect_failure((P.test_x6_taylor_error_is_third_order_with_known_coefficient, ()))


def test_global_instead_of_per_head_normalisation(monkeypatch):
    def bad(ell):
        e = np.exp(ell - ell.max())
        return (e / e.sum()).sum(axis=0)
    _patch(monkeypatch, "group_block_scores", bad)
    _expect_failure((P.test_x7_group_scores_sum_to_G, (4, 37)))


def test_ties_to_higher_index(monkeypatch):
    def bad(score, k, n_sink, n_local):
        nb = len(score)
        if nb <= k:
            return np.arange(nb)
        forced = OS.forced_blocks(nb, k, n_sink, n_local)
        rest = [i for i in range(nb) if i not in set(forced)]
        rest.sort(key=lambda i: (-float(score[i]), -i))
        return np.array(sorted(forced + rest[:k - len(forced)]))
    _patch(monkeypatch, "select_blocks", bad)
    _expect_failure(*[(P.test_x9_selection_brute_force_with_ties, (s,)) for s in range(12)])


def test_transposed_global_state(monkeypatch):
    def bad(K, V, L):
        phik = OS.feature_map(np.asarray(K, float)[:L])
        return (phik.T @ np.asarray(V, float)[:L]).T, phik.sum(0)
    _patch(monkeypatch, "global_state", bad)
    _expect_failure((P.test_x1_subtraction_residual_equals_bruteforce_recurrence, (0,)))


def test_feature_map_on_scaled_vectors(monkeypatch):
    orig = OS.residual_linear_attention

    def bad(q, s_bar, z_bar, K, V, tok, L, normalize=False):
        return orig(q / math.sqrt(q.shape[-1]), s_bar, z_bar, K, V, tok, L, normalize)
    _patch(monkeypatch, "residual_linear_attention", bad)
    _expect_failure((P.test_x1_subtraction_residual_equals_bruteforce_recurrence, (0,)))


def test_exact_branch_without_scale(monkeypatch):
    orig = OS.exact_sparse_attention
    _patch(monkeypatch, "exact_sparse_attention", lambda q, K, V, tok, s: orig(q, K, V, tok, 1.0))
    _expect_failure((P.test_x2_selecting_every_block_is_dense_attention, (100,)),
                    (P.test_x3_exact_branch_is_masked_dense_attention, (0,)))


def test_rmsnorm_sum_instead_of_mean(monkeypatch):
    def bad(o_sparse, r, gamma, eps):
        return o_sparse + gamma * r / np.sqrt((r * r).sum(-1, keepdims=True) + eps)
    _patch(monkeypatch, "combine", bad)
    _expect_failure((P.test_x12_constant_values_closed_form, ()))


def test_residual_not_zeroed_when_all_selected(monkeypatch):
    # the count test never fires: the residual is the cancellation noise of
    # o_bar - o_tilde, and RMSNorm blows it up to unit scale
    _patch(monkeypatch, "nothing_unselected", lambda n, L: False)
    _expect_failure((P.test_x2_selecting_every_block_is_dense_attention, (100,)),
                    (P.test_x23_every_block_selected_with_zero_eps_is_dense_attention, (37,)))


def test_cutoff_is_the_highest_admitted_score(monkeypatch):
    def bad(score, sel, k, n_sink, n_local):
        nb = len(score)
        if nb <= k:
            return None
        fset = set(OS.forced_blocks(nb, k, n_sink, n_local))
        ranked = [float(score[i]) for i in sel if int(i) not in fset]
        return max(ranked) if ranked else None
    _patch(monkeypatch, "cutoff_score", bad)
    _expect_failure(*[(P.test_x21_cutoff_score_hand_worked, (n,)) for n in P.CUTOFF_CASES])


def test_cutoff_counts_forced_blocks(monkeypatch):
    def bad(score, sel, k, n_sink, n_local):
        if len(score) <= k:
            return None
        return min(float(score[i]) for i in sel)
    _patch(monkeypatch, "cutoff_score", bad)
    _expect_failure(*[(P.test_x21_cutoff_score_hand_worked, (n,)) for n in P.CUTOFF_CASES])


def test_normaliser_over_every_token(monkeypatch):
    # <phi(q), z_bar> in place of <phi(q), z_bar - z_tilde>
    def bad(q, s_bar, z_bar, K, V, tok, L, normalize=False):
        phiq = OS.feature_map(q)
        o_bar = phiq @ s_bar
        phik = OS.feature_map(np.asarray(K, float)[tok])
        o_tilde = (phiq @ phik.T) @ np.asarray(V, float)[tok]
        if OS.nothing_unselected(len(tok), L):
            return np.zeros_like(o_bar), o_bar, o_tilde
        r = o_bar - o_tilde
        if normalize:
            r = r / (phiq @ z_bar)[:, None]
        return r, o_bar, o_tilde
    _patch(monkeypatch, "residual_linear_attention", bad)
    _expect_failure(*[(P.test_x22_rla_normaliser_is_the_unselected_linear_mass, (s,))
                      for s in range(3)])


def test_strided_instead_of_contiguous_groups(monkeypatch):
    def bad(q, states, K, V, gamma, p, force_selection=None):
        Hkv = len(states)
        G = q.shape[0] // Hkv
        return [OS.decode_kv_head(q[h::Hkv], states[h], K[h], V[h], gamma[h::Hkv], p)
                for h in range(Hkv)]
    _patch(monkeypatch, "decode_from_state", bad)
    _expect_failure((P.test_x2_selecting_every_block_is_dense_attention, (100,)))


def test_welford_wrong_update(monkeypatch):
    orig = OS.append_state

    def bad(state, k_new, v_new, B, d=None):
        st = orig(state, k_new, v_new, B, d)
        st.var = st.var * (1 + 1e-6)
        return st
    _patch(monkeypatch, "append_state", bad)
    _expect_failure((P.test_x13_streaming_stats_and_state_match_textbook, ()))


@pytest.mark.parametrize("flip", ["sink", "local"])
def test_forced_blocks_dropped(monkeypatch, flip):
    orig = OS.forced_blocks

    def bad(nb, k, n_sink, n_local):
        if flip == "sink":
            return orig(nb, k, 0, n_local)
        return orig(nb, k, n_sink, 0)
    _patch(monkeypatch, "forced_blocks", bad)
    _expect_failure((P.test_forced_blocks_always_selected_even_with_lowest_scores, ()))


def _pool(rule):
    def f(wscore, L, B, C, s):
        wscore = np.asarray(wscore, dtype=float)
        out = np.zeros(-(-L // B))
        for i, (a, b) in enumerate(OS.block_ranges(L, B)):
            ws = [w for w in range(len(wscore))
                  if (rule == "start" and a <= w * s < b)
                  or (rule == "inside" and a <= w * s and min(w * s + C, L) <= b)]
            out[i] = max(wscore[w] for w in ws) if ws else 0.0
        return out
    return f


@pytest.mark.parametrize("rule", ["start", "inside"])
def test_pooling_over_the_wrong_windows(monkeypatch, rule):
    """Blocks pooling only the windows that start in them, or only those
    inside them, in place of every window that touches them."""
    _patch(monkeypatch, "pool_windows_to_blocks", _pool(rule))
    _expect_failure((W.test_x17_pooling_matches_token_set_overlap, (117, 32, 32, 16)),
                    (W.test_x18_planted_tokens_at_a_block_end_select_both_blocks, ()))


@pytest.mark.parametrize("mistake", ["no_partial", "short"])
def test_wrong_window_ranges(monkeypatch, mistake):
    """Partial windows at the end dropped, or every window a token short."""
    def bad(L, C, s):
        if mistake == "no_partial":
            return [(w * s, w * s + C) for w in range(L // s) if w * s + C <= L]
        return [(w * s, min(w * s + C - 1, L)) for w in range(-(-L // s))]
    _patch(monkeypatch, "window_ranges", bad)
    _expect_failure((W.test_x15_constant_keys_window_and_block_scores_closed_form, ()),
                    (W.test_x16_window_mass_matches_token_sum, (32, 16)))


def test_prefill_that_sees_the_whole_chunk(monkeypatch):
    """Every query of a chunk decoded against the whole chunk (no causal
    mask) in place of its own prefix."""
    import test_oracle_prefill as PF

    def bad(Q, K, V, L0, gamma, p):
        n = L0 + Q.shape[0]
        state = OS.build_state(K, V, n, p.block_size)
        return [OS.decode_kv_head(Q[i], state, K[:n], V[:n], gamma, p) for i in range(Q.shape[0])]
    _patch(monkeypatch, "prefill_kv_head", bad)
    _expect_failure((PF.test_p1_all_blocks_selected_is_causal_dense_attention, (5, 12)),
                    (PF.test_p3_later_tokens_do_not_change_earlier_outputs, ()))
