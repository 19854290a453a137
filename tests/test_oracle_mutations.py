"""Plant plausible mistakes in the oracle (on the CPU, in this process only) and
check that the pins catch each of them."""
import math

import numpy as np
import pytest

import oracle
import oracle.growpage_oracle as G
import test_oracle_pins as pins


def _patch(monkeypatch, name, fn):
    monkeypatch.setattr(G, name, fn)
    monkeypatch.setattr(oracle, name, fn, raising=False)


def _fails(test, *args):
    with pytest.raises(AssertionError):
        test(*args)


def test_rope_sign_flip_is_caught(monkeypatch):
    orig = G.rope

    def bad(x, pos, theta):
        return orig(x, -pos, theta)
    _patch(monkeypatch, "rope", bad)
    _fails(pins.test_p7_rope_properties)


def test_ema_weights_swapped_are_caught(monkeypatch):
    _patch(monkeypatch, "ema_update", lambda qbar, q, beta: (1.0 - beta) * qbar + beta * q)
    _fails(pins.test_p6_ema_closed_form_and_special_cases)


def test_top_p_off_by_one_is_caught(monkeypatch):
    orig = G.top_p_count
    _patch(monkeypatch, "top_p_count", lambda a, p: max(1, orig(a, p) - 1))
    _fails(pins.test_p5_top_p_count_equals_brute_force)


def test_selection_tie_break_reversed_is_caught(monkeypatch):
    def bad_order(s32, idx):
        return idx[np.lexsort((-idx, -s32[idx].astype(np.float64)))]
    monkeypatch.setattr(G, "_order", bad_order)
    _fails(pins.test_golden_selection)


def test_compaction_order_is_caught(monkeypatch):
    def bad(tokens, kept, P, b):
        out = tokens.copy()
        K_t = (P - 2) * b
        out[:b] = tokens[(P - 1) * b: P * b]
        out[b:K_t + b] = tokens[kept]
        return out
    _patch(monkeypatch, "compact_tokens", bad)
    _fails(pins.test_golden_selection)


def test_calibration_inverted_is_caught(monkeypatch):
    def bad(q_t, qbar):
        return (G.rms(qbar) / G.rms(q_t)) * np.asarray(qbar, dtype=np.float64)
    _patch(monkeypatch, "calibrate", bad)
    _fails(pins.test_p7_calibration_matches_rms)


def test_threshold_not_strict_is_caught(monkeypatch):
    orig = G.demand_trend
    # Delta = 0 must compress; a "greater or equal" rule would grow
    _patch(monkeypatch, "demand_trend", lambda k_s, k_l, C: orig(k_s, k_l, C) + G.Fraction(1, 10**9))
    _fails(pins.test_p8_equal_summaries_give_zero_trend_and_compress)


def test_dropped_grouped_head_is_caught(monkeypatch):
    def bad(K_cand, q_t, qbar_s, qbar_l, pos, theta, scale):
        C, Hkv, d = K_cand.shape
        Hq = q_t.shape[0]
        Gq = Hq // Hkv
        a = np.zeros((2, Hkv, C))
        for x, qbar in enumerate((qbar_s, qbar_l)):
            for g in range(0, Hq, Gq):          # only the first head of each group
                qt = G.rope(G.calibrate(q_t[g], qbar[g]), pos, theta)
                a[x, g // Gq] = G.softmax(scale * (K_cand[:, g // Gq] @ qt))
        return a
    _patch(monkeypatch, "view_distributions", bad)
    _fails(pins.test_view_distributions_special_case_is_softmax)


def test_token_score_mean_instead_of_max_is_caught(monkeypatch):
    _patch(monkeypatch, "token_scores",
           lambda a_s, a_l: ((np.asarray(a_s, np.float64) + np.asarray(a_l, np.float64)) / 2).astype(np.float32))
    _fails(pins.test_golden_token_scores)


def test_token_score_short_view_alone_is_caught(monkeypatch):
    _patch(monkeypatch, "token_scores", lambda a_s, a_l: np.asarray(a_s, np.float32).copy())
    _fails(pins.test_golden_token_scores)


def test_token_score_long_view_alone_is_caught(monkeypatch):
    _patch(monkeypatch, "token_scores", lambda a_s, a_l: np.asarray(a_l, np.float32).copy())
    _fails(pins.test_golden_token_scores)


def _fragile_with(shift: int, eps_factor: float = 1.0):
    """top_p_fragile that checks the running sums `shift` terms later than it
    should, or with a band eps_factor times too wide."""
    def bad(a32, p, eps=1e-6):
        v = np.sort(np.asarray(a32, dtype=np.float32).astype(np.float64))[::-1]
        csum = np.cumsum(v)
        k = G.top_p_count(a32, p) + shift
        e = eps * eps_factor
        near = 0 <= k - 1 < csum.size and abs(csum[k - 1] - p) <= e
        if 0 <= k - 2 < csum.size:
            near = near or abs(csum[k - 2] - p) <= e
        return bool(near)
    return bad


@pytest.mark.parametrize("shift", [1, -1])
def test_top_p_fragile_index_off_by_one_is_caught(monkeypatch, shift):
    _patch(monkeypatch, "top_p_fragile", _fragile_with(shift))
    _fails(pins.test_golden_top_p_fragile)


def test_top_p_fragile_band_ten_times_too_wide_is_caught(monkeypatch):
    _patch(monkeypatch, "top_p_fragile", _fragile_with(0, 10.0))
    _fails(pins.test_golden_top_p_fragile)


def test_entropy_fragile_band_ten_times_too_wide_is_caught(monkeypatch):
    orig = G.entropy_fragile
    _patch(monkeypatch, "entropy_fragile", lambda a32, eps=1e-6: orig(a32, 10 * eps))
    _fails(pins.test_golden_entropy_fragile)


def test_entropy_fragile_at_integers_instead_of_midpoints_is_caught(monkeypatch):
    def bad(a32, eps=1e-6):
        v = np.asarray(a32, dtype=np.float32).astype(np.float64)
        v = v[v > 0]
        e = float(np.exp(-np.sum(v * np.log(v))))
        return bool(abs(e - round(e)) <= eps * max(1.0, e))
    _patch(monkeypatch, "entropy_fragile", bad)
    _fails(pins.test_golden_entropy_fragile)
