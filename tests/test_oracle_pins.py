"""The oracle against what the paper and mathematics fix (CPU only).

Second half: planted mistakes.  Each mutant is a copy of one oracle routine with one
plausible error (a dropped term, a wrong sign or index, a swapped operand or update
order); the corresponding pin must reject it.  This shows that the pins can see the
kind of mistake they are meant to catch.
"""
import math
import os

import numpy as np
import pytest

import oracle as O
from tests import oracle_pins as pins

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


# ----------------------------------------------------------------------------- pins hold

def test_meta_minmax_bounds_attained():
    assert pins.check_meta_bounds_attained(O.page_metadata_minmax)


def test_meta_identical_page():
    assert pins.check_meta_identical_page(O.page_metadata_minmax)


def test_meta_mean():
    assert pins.check_meta_mean(O.page_metadata_mean)


@pytest.mark.parametrize("g", [1, 4, 16])
def test_quest_upper_bound(g):
    assert pins.check_quest_upper_bound(O.page_metadata_minmax, O.representative_query, O.criticality_minmax, g=g)


def test_quest_tight_at_corner():
    assert pins.check_quest_tight_at_corner(O.page_metadata_minmax, O.representative_query, O.criticality_minmax)


def test_score_special_cases():
    assert pins.check_score_special_cases(O.page_metadata_minmax, O.representative_query, O.criticality_minmax)


def test_mean_score_is_dot_with_block_mean():
    r = np.random.default_rng(0)
    k = r.standard_normal((1, 3, 64, 8))
    q = r.standard_normal((4, 8))
    s = O.criticality_mean(O.representative_query(q, 1), O.page_metadata_mean(k, 64, 192))
    # linearity: qbar . mean(k) == mean over tokens of qbar . k
    want = (k[0] @ q.mean(axis=0)).mean(axis=1)
    assert np.allclose(s[0], want, atol=1e-12)


def test_gqa_grouping():
    assert pins.check_gqa_grouping(O.representative_query)


def test_topk_brute_force():
    assert pins.check_topk(O.select_topk)


def test_topk_all_pages_and_ties():
    s = np.zeros(9)
    assert list(O.select_topk(s, 4)) == [0, 1, 2, 3]  # ties: lower index first
    assert list(O.select_topk(s, 20)) == list(range(9))
    assert list(O.select_topk(np.arange(9.0), 2, forced=[0, 8], forced_in_budget=True)) == [0, 8]
    assert list(O.select_topk(np.arange(9.0), 2, forced=[0, 8], forced_in_budget=False)) == [0, 6, 7, 8]


def test_topk_decides_in_float32():
    # two scores that differ in float64 but round to the same float32: tie -> lower index
    s = np.array([1.0, 1.0 + 1e-12])
    assert list(O.select_topk(s, 1)) == [0]


def test_ema_hand_example():
    assert pins.check_ema_hand_example(O.ema_init, O.ema_predict, O.ema_update)


def test_ema_constant():
    assert pins.check_ema_constant(O.ema_init, O.ema_predict, O.ema_update)


def test_ema_ramp_closed_form():
    assert pins.check_ema_ramp(O.ema_init, O.ema_predict, O.ema_update)


def test_ema_s1_reduction():
    assert pins.check_ema_s1(O.ema_init, O.ema_predict, O.ema_update)


@pytest.mark.parametrize("g", [1, 4])
def test_attend_equals_dense_sdpa(g):
    assert pins.check_attend_dense(O.attend, g=g)


def test_attend_subset_equals_sdpa_on_gathered_pages():
    assert pins.check_attend_subset(O.attend)


def test_merge_algebra():
    assert pins.check_merge_algebra(O.merge_two)


def test_merge_union():
    assert pins.check_merge_union(O.attend, O.merge_two)


def test_speculate_then_repair_every_subset():
    assert pins.check_speculate_repair(O.speculate_then_repair, O.attend)


def test_missed_wasted_sets():
    m, n = O.missed_and_wasted([1, 2, 3, 5], [2, 3, 4])
    assert list(m) == [1, 5] and list(n) == [4]
    assert O.hit_rate([1, 2, 3, 5], [2, 3, 4]) == 0.5


def test_theta_grid_matches_paper():
    vals = {}
    with open(os.path.join(GOLDEN, "theta_grid.txt")) as f:
        for line in f:
            if line.startswith("#") or not line.strip():
                continue
            key, *rest = line.split()
            vals[key] = [float(x) for x in rest]
    assert len(O.THETA_GRID) == int(vals["count"][0])
    assert sorted({t[0] for t in O.THETA_GRID}) == vals["alpha"]
    assert sorted({t[1] for t in O.THETA_GRID}) == vals["beta"]
    assert sorted({t[2] for t in O.THETA_GRID}) == vals["gamma"]


def test_calibration_objective_limits():
    r = np.random.default_rng(3)
    row = np.abs(r.standard_normal(12)) + 0.1
    const = np.tile(row, (6, 1))
    for theta in O.THETA_GRID[:10]:
        assert O.calibration_objective(const, 4, theta) == pytest.approx(1.0)
    traj = np.abs(r.standard_normal((8, 12))) + 0.1
    # predicting every block covers every selection
    assert O.calibration_objective(traj, 4, (0.5, 0.5, 0.0), p_select=12) == pytest.approx(1.0)
    # brute force of Eq. (4) for the reuse-previous predictor (alpha = 1, gamma = 0)
    want = np.mean([
        traj[t][np.intersect1d(np.argsort(-traj[t])[:4], np.argsort(-traj[t - 1])[:4])].sum()
        / traj[t][np.argsort(-traj[t])[:4]].sum()
        for t in range(1, 8)])
    assert O.calibration_objective(traj, 4, (1.0, 0.3, 0.0)) == pytest.approx(want, abs=1e-12)


def test_calibration_picks_trend_on_ramps():
    # blocks whose scores ramp at different rates: extrapolating the trend (gamma > 0)
    # predicts the crossing order better than the lagging level alone
    t = np.arange(30)[:, None]
    traj = 5.0 + np.array([[0.5, -0.5, 0.3, -0.3, 0.1, -0.1, 0.0, 0.2]]) * t + np.array([[0, 9, 2, 7, 4, 5, 4.5, 3]])
    best, val = O.calibrate(traj, 3)
    assert best[2] > 0.0 and val >= O.calibration_objective(traj, 3, (best[0], best[1], 0.0))


def test_calibrate_closed_form_argmax():
    assert pins.check_calibrate_closed_form(O.calibration_objective, O.calibrate, O.THETA_GRID)


def test_calibrate_ties_take_first_grid_point():
    assert pins.check_calibrate_all_tied(O.calibrate, O.THETA_GRID)


def test_calibration_blocks_form_during_prefill():
    assert pins.check_calibration_formation(O.calibration_objective, O.THETA_GRID)


def test_criticality_mean_bounds():
    assert pins.check_criticality_mean_bounds(O.page_metadata_mean, O.representative_query, O.criticality_mean)


def test_dropped_page_changes_output():
    """On the tiny workload, removing any one selected page moves the output by more
    than the internal tolerance (1e-4), so a missed page is visible to the parity tests."""
    import workloads as W
    cfg = W.CONFIGS["tiny"]
    li = W.layer_inputs(cfg)
    _, qb = W.query_trajectory(cfg, steps=1)
    q = W.bits_to_f64(qb[1], cfg.dtype)
    k, v = li.k64(), li.v64()
    _, sel, (o, m, l) = O.serial_step(q, k, v, cfg.page_size, cfg.context, cfg.k_select)
    for p in sel[0]:
        rest = [x for x in sel[0] if x != p]
        o2, _, _ = O.attend(q, k, v, [rest], cfg.page_size, cfg.context)
        assert np.abs(o2 - o).max() > 1e-4


# ----------------------------------------------------------------------------- planted mistakes

def _meta_ignores_num_tokens(k, ps, nt):
    return k.min(axis=2), k.max(axis=2)


def _meta_swapped(k, ps, nt):
    mn, mx = O.page_metadata_minmax(k, ps, nt)
    return mx, mn


def _score_min_instead_of_max(qbar, mins, maxs):
    return np.minimum(qbar[:, None, :] * mins, qbar[:, None, :] * maxs).sum(-1)


def _score_ignores_sign(qbar, mins, maxs):
    return (qbar[:, None, :] * maxs).sum(-1)


def _score_drops_min_term(qbar, mins, maxs):
    return np.maximum(0.0, qbar[:, None, :] * maxs).sum(-1)


def _qbar_strided_groups(q, hkv):
    # head j -> KV head j % Hkv instead of j // G
    return np.stack([q[h::hkv].mean(axis=0) for h in range(hkv)])


def _qbar_sum_not_mean(q, hkv):
    return O.representative_query(q, hkv) * (q.shape[0] // hkv)


def _topk_ties_to_higher_index(s, k, forced=(), fib=True):
    n = len(s)
    forced = sorted(set(forced))
    extra = max(0, k - len(forced)) if fib else k
    cand = [p for p in range(n) if p not in forced]
    cand.sort(key=lambda p: (-float(np.float32(s[p])), -p))
    return np.array(sorted(forced + cand[:extra]))


def _topk_forced_outside_budget(s, k, forced=(), fib=True):
    return O.select_topk(s, k, forced, False)


def _ema_update_level_first(l, v, s, a, b):
    nl = a * s + (1 - a) * l
    return nl, b * (s - nl) + (1 - b) * v


def _ema_update_beta_swapped(l, v, s, a, b):
    return a * s + (1 - a) * l, (1 - b) * (s - l) + b * v


def _ema_predict_minus(l, v, g):
    return l - g * v


def _attend_no_scale(q, k, v, pages, ps, nt):
    return O.attend(q * math.sqrt(q.shape[1]), k, v, pages, ps, nt)


def _attend_strided_gqa(q, k, v, pages, ps, nt):
    hq, hkv = q.shape[0], k.shape[0]
    g = hq // hkv
    perm = np.array([(j % hkv) * g + j // hkv for j in range(hq)])
    o, m, l = O.attend(q[np.argsort(perm)], k, v, pages, ps, nt)
    return o[perm], m[perm], l[perm]


def _attend_ignores_num_tokens(q, k, v, pages, ps, nt):
    return O.attend(q, k, v, pages, ps, k.shape[1] * ps)


def _merge_wrong_sign(a, b):
    oa, ma, la = a
    ob, mb, lb = b
    mo = np.maximum(ma, mb)
    wa, wb = np.exp(mo - ma) * la, np.exp(mo - mb) * lb
    lo = wa + wb
    return (wa[:, None] * oa + wb[:, None] * ob) / lo[:, None], mo, lo


def _merge_forgets_l(a, b):
    oa, ma, la = a
    ob, mb, lb = b
    mo = np.maximum(ma, mb)
    wa, wb = np.exp(ma - mo), np.exp(mb - mo)
    lo = wa * la + wb * lb
    return (wa[:, None] * oa + wb[:, None] * ob) / (wa + wb)[:, None], mo, lo


def _calibrate_argmin(traj, k, grid=O.THETA_GRID, p_select=None, form_row=None):
    vals = [O.calibration_objective(traj, k, th, p_select, form_row) for th in grid]
    i = int(np.argmin(vals))
    return grid[i], vals[i]


def _calibrate_last_on_ties(traj, k, grid=O.THETA_GRID, p_select=None, form_row=None):
    vals = [O.calibration_objective(traj, k, th, p_select, form_row) for th in grid]
    i = len(vals) - 1 - int(np.argmax(vals[::-1]))
    return grid[i], vals[i]


def _objective_state_from_row0(traj, k, theta, p_select=None, form_row=None):
    return O.calibration_objective(traj, k, theta, p_select)


def _objective_placeholder_zero(traj, k, theta, p_select=None, form_row=None):
    t = np.array(traj, dtype=np.float64, copy=True)
    if form_row is not None:
        for b, r in enumerate(form_row):
            t[:r, b] = 0.0
    return O.calibration_objective(t, k, theta, p_select)


def _objective_level_first(traj, k, theta, p_select=None, form_row=None):
    import unittest.mock as um
    from oracle import prr_oracle
    with um.patch.object(prr_oracle, "ema_update", _ema_update_level_first):
        return O.calibration_objective(traj, k, theta, p_select, form_row)


def _criticality_mean_sum(qbar, means):
    return O.criticality_mean(qbar, means) * 16


def _spec_repair_skips_missed(q, k, v, sel, pred, ps, nt, keep_wasted=False):
    hq, hkv = q.shape[0], k.shape[0]
    spec = [(set(p) if keep_wasted else set(p) & set(a)) for a, p in zip(sel, pred)]
    return O.attend(q, k, v, spec, ps, nt)


def _spec_repair_keeps_wasted_always(q, k, v, sel, pred, ps, nt, keep_wasted=False):
    return O.speculate_then_repair(q, k, v, sel, pred, ps, nt, keep_wasted=True)


MUTANTS = [
    ("meta ignores num_tokens", lambda: pins.check_meta_bounds_attained(_meta_ignores_num_tokens)),
    ("meta min/max swapped", lambda: pins.check_meta_bounds_attained(_meta_swapped)),
    ("score min instead of max", lambda: pins.check_quest_upper_bound(
        O.page_metadata_minmax, O.representative_query, _score_min_instead_of_max)),
    ("score ignores qbar sign", lambda: pins.check_quest_upper_bound(
        O.page_metadata_minmax, O.representative_query, _score_ignores_sign)),
    ("score drops the min term", lambda: pins.check_quest_tight_at_corner(
        O.page_metadata_minmax, O.representative_query, _score_drops_min_term)),
    ("qbar strided groups", lambda: pins.check_gqa_grouping(_qbar_strided_groups)),
    ("qbar sum not mean", lambda: pins.check_score_special_cases(
        O.page_metadata_minmax, _qbar_sum_not_mean, O.criticality_minmax)),
    ("top-k ties to higher index", lambda: pins.check_topk(_topk_ties_to_higher_index)),
    ("top-k forced outside budget", lambda: pins.check_topk(_topk_forced_outside_budget)),
    ("ema level updated first", lambda: pins.check_ema_ramp(O.ema_init, O.ema_predict, _ema_update_level_first)),
    ("ema level first (hand example)", lambda: pins.check_ema_hand_example(
        O.ema_init, O.ema_predict, _ema_update_level_first)),
    ("ema beta swapped", lambda: pins.check_ema_hand_example(O.ema_init, O.ema_predict, _ema_update_beta_swapped)),
    ("ema predict minus trend", lambda: pins.check_ema_hand_example(O.ema_init, _ema_predict_minus, O.ema_update)),
    ("attend without 1/sqrt(d)", lambda: pins.check_attend_dense(_attend_no_scale)),
    ("attend strided GQA", lambda: pins.check_attend_dense(_attend_strided_gqa)),
    ("attend ignores num_tokens", lambda: pins.check_attend_dense(_attend_ignores_num_tokens)),
    ("merge exponent sign", lambda: pins.check_merge_algebra(_merge_wrong_sign)),
    ("merge forgets l", lambda: pins.check_merge_union(O.attend, _merge_forgets_l)),
    ("repair skips missed pages", lambda: pins.check_speculate_repair(_spec_repair_skips_missed, O.attend)),
    ("repair keeps wasted in exact mode", lambda: pins.check_speculate_repair(
        _spec_repair_keeps_wasted_always, O.attend)),
    ("calibrate takes the argmin", lambda: pins.check_calibrate_closed_form(
        O.calibration_objective, _calibrate_argmin, O.THETA_GRID)),
    ("calibrate takes the last maximiser", lambda: pins.check_calibrate_closed_form(
        O.calibration_objective, _calibrate_last_on_ties, O.THETA_GRID)),
    ("calibrate last on all-tied grid", lambda: pins.check_calibrate_all_tied(_calibrate_last_on_ties, O.THETA_GRID)),
    ("calibration objective with the level updated first", lambda: pins.check_calibrate_closed_form(
        _objective_level_first, O.calibrate, O.THETA_GRID)),
    ("calibration state from row 0 (junk)", lambda: pins.check_calibration_formation(
        _objective_state_from_row0, O.THETA_GRID)),
    ("calibration state from a placeholder 0", lambda: pins.check_calibration_formation(
        _objective_placeholder_zero, O.THETA_GRID)),
    ("block-mean score as a sum", lambda: pins.check_criticality_mean_bounds(
        O.page_metadata_mean, O.representative_query, _criticality_mean_sum)),
]


@pytest.mark.parametrize("name,check", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_planted_mistake_is_caught(name, check):
    with np.errstate(all="ignore"):
        assert not check(), f"pin did not catch: {name}"
