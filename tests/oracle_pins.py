"""Checks that pin the oracle to facts fixed by the paper or by mathematics.

Each check takes the routine(s) under test as arguments and returns True when the
pin holds, so the same check can be run on the oracle (must pass) and on a copy of
the oracle with a planted mistake (must fail).  Nothing here re-types an oracle
formula: the checks are bounds, closed forms, brute force, special cases and
library routines (torch's scaled_dot_product_attention, scipy's logsumexp, numpy's
lexsort).
"""
from __future__ import annotations

import itertools
import math

import numpy as np
import scipy.special
import torch


def _rng(seed):
    return np.random.default_rng(seed)


# ----------------------------------------------------------------------------- metadata

def check_meta_bounds_attained(meta_fn, seed=0):
    """Every key lies in [m, M] channel-wise, and both bounds are attained by some token
    of the page; tokens at or beyond num_tokens never matter."""
    r = _rng(seed)
    k = r.standard_normal((2, 5, 16, 8))
    num_tokens = 4 * 16 + 7  # last page has 7 valid tokens
    kk = k.copy()
    kk[:, 4, 7:] = 1e9 * np.sign(r.standard_normal((2, 9, 8)))  # junk beyond the end
    mins, maxs = meta_fn(kk, 16, num_tokens)
    for p in range(5):
        valid = 16 if p < 4 else 7
        kv = k[:, p, :valid]
        if not (np.all(kv >= mins[:, p, None] ) and np.all(kv <= maxs[:, p, None])):
            return False
        if not (np.all(np.any(kv == mins[:, p, None], axis=1)) and np.all(np.any(kv == maxs[:, p, None], axis=1))):
            return False
    return True


def check_meta_identical_page(meta_fn):
    tok = np.linspace(-3, 3, 8)
    k = np.broadcast_to(tok, (1, 1, 16, 8)).copy()
    mins, maxs = meta_fn(k, 16, 16)
    return np.array_equal(mins[0, 0], tok) and np.array_equal(maxs[0, 0], tok)


def check_meta_mean(mean_fn, seed=1):
    """Mean of identical tokens is the token; adding a constant shifts the mean by it;
    a partial page averages its valid tokens only."""
    r = _rng(seed)
    tok = r.standard_normal(8)
    k = np.broadcast_to(tok, (1, 2, 16, 8)).copy()
    if not np.allclose(mean_fn(k, 16, 32)[0], tok, rtol=0, atol=1e-15):
        return False
    k2 = r.standard_normal((1, 2, 16, 8))
    c = r.standard_normal(8)
    if not np.allclose(mean_fn(k2 + c, 16, 32), mean_fn(k2, 16, 32) + c, atol=1e-12):
        return False
    k3 = k2.copy()
    k3[0, 1, 5:] = 1e9
    got = mean_fn(k3, 16, 16 + 5)[0, 1]
    return np.allclose(got, k2[0, 1, :5].sum(axis=0) / 5, atol=1e-12)


# ----------------------------------------------------------------------------- score

def check_quest_upper_bound(meta_fn, qbar_fn, score_fn, g=1, seed=2):
    """The criticality of a page upper-bounds qbar . k for every token of the page
    (the defining property of Quest's estimate; under MHA, G = 1, qbar = q)."""
    r = _rng(seed)
    hkv, n, d = 2, 6, 16
    k = r.standard_normal((hkv, n, 16, d))
    q = r.standard_normal((hkv * g, d))
    mins, maxs = meta_fn(k, 16, n * 16)
    qbar = qbar_fn(q, hkv)
    s = score_fn(qbar, mins, maxs)
    for h in range(hkv):
        qb = q[h * g:(h + 1) * g].mean(axis=0)  # mean of the group, by numpy
        for p in range(n):
            dots = k[h, p] @ qb
            if not np.all(s[h, p] >= dots - 1e-12 * (1 + abs(dots))):
                return False
    return True


def check_quest_tight_at_corner(meta_fn, qbar_fn, score_fn, seed=3):
    """If the page contains the 'corner' token (the max channel where qbar >= 0, the
    min channel where qbar < 0) the bound is attained: score = qbar . corner."""
    r = _rng(seed)
    d = 16
    q = r.standard_normal((1, d))
    k = r.standard_normal((1, 1, 16, d))
    lo, hi = k[0, 0].min(axis=0), k[0, 0].max(axis=0)
    corner = np.where(q[0] >= 0, hi, lo)
    k[0, 0, 3] = corner
    mins, maxs = meta_fn(k, 16, 16)
    s = score_fn(qbar_fn(q, 1), mins, maxs)
    return abs(s[0, 0] - corner @ q[0]) <= 1e-12 * (1 + abs(s[0, 0]))


def check_score_special_cases(meta_fn, qbar_fn, score_fn, seed=4):
    """Identical-token page: score = qbar . k.  Non-negative qbar: score = qbar . M."""
    r = _rng(seed)
    d = 16
    q = np.abs(r.standard_normal((2, d)))  # both heads of a G = 2 group non-negative
    k = r.standard_normal((1, 2, 16, d))
    k[0, 0] = k[0, 0, 0]
    mins, maxs = meta_fn(k, 16, 32)
    qb = qbar_fn(q, 1)
    s = score_fn(qb, mins, maxs)
    qm = q.mean(axis=0)
    ok = abs(s[0, 0] - k[0, 0, 0] @ qm) <= 1e-12 * (1 + abs(s[0, 0]))
    ok &= abs(s[0, 1] - k[0, 1].max(axis=0) @ qm) <= 1e-12 * (1 + abs(s[0, 1]))
    return bool(ok)


def check_gqa_grouping(qbar_fn, seed=5):
    """Query head j belongs to KV head j // G: changing heads of other groups leaves a
    group's representative query unchanged; G copies of one head give that head."""
    r = _rng(seed)
    hkv, g, d = 3, 4, 8
    q = r.standard_normal((hkv * g, d))
    base = qbar_fn(q, hkv)
    for h in range(hkv):
        q2 = q.copy()
        others = [j for j in range(hkv * g) if j // g != h]
        q2[others] += 100.0
        if not np.array_equal(qbar_fn(q2, hkv)[h], base[h]):
            return False
    same = np.repeat(r.standard_normal((hkv, d)), g, axis=0)
    return np.allclose(qbar_fn(same, hkv), same[::g], atol=1e-15)


# ----------------------------------------------------------------------------- top-K

def _lexsort_topk(scores32, k, forced, forced_in_budget):
    """Library route: numpy.lexsort on (index, -score)."""
    n = len(scores32)
    forced = sorted(set(forced))
    mask = np.ones(n, bool)
    mask[forced] = False
    cand = np.nonzero(mask)[0]
    order = cand[np.lexsort((cand, -scores32[cand].astype(np.float64)))]
    extra = max(0, k - len(forced)) if forced_in_budget else k
    return np.sort(np.concatenate([np.array(forced, dtype=np.int64), order[:extra]]))


def check_topk(select_fn, seed=6, trials=60):
    """Brute force on small inputs with many ties: every selected non-forced page beats
    every unselected one by (float32 score desc, index asc); forced pages are always
    selected; the size matches the budget; agrees with numpy.lexsort."""
    r = _rng(seed)
    for t in range(trials):
        n = int(r.integers(1, 24))
        s = r.integers(-3, 4, size=n).astype(np.float64) * 0.5 + (r.standard_normal(n) * 1e-9 if t % 3 == 0 else 0)
        k = int(r.integers(0, n + 3))
        forced = sorted(set(r.integers(0, n, size=int(r.integers(0, 3))).tolist()))
        fib = bool(r.integers(0, 2))
        got = np.asarray(select_fn(s, k, forced, fib))
        want_n = min(n, max(len(forced), k) if fib else k + len(forced))
        if len(got) != want_n or len(set(got.tolist())) != len(got):
            return False
        if not set(forced) <= set(got.tolist()):
            return False
        s32 = s.astype(np.float32)
        sel = set(got.tolist()) - set(forced)
        uns = set(range(n)) - set(got.tolist())
        for a, b in itertools.product(sel, uns):
            if not (s32[a] > s32[b] or (s32[a] == s32[b] and a < b)):
                return False
        if not np.array_equal(got, _lexsort_topk(s32, k, forced, fib)):
            return False
    return True


# ----------------------------------------------------------------------------- EMA

def check_ema_hand_example(init_fn, predict_fn, update_fn):
    """Steps worked by hand from Eqs. (2)-(3) (all values dyadic, so exact in floating
    point).

    Example 1, alpha = beta = gamma = 1/2, scores 4, 8, 2:
      init:   l = 4, v = 0
      t = 1:  predict 4;   v = (8-4)/2 + 0 = 2;        l = (8+4)/2 = 6
      t = 2:  predict 7;   v = (2-6)/2 + 2/2 = -1;     l = (2+6)/2 = 4
      t = 3:  predict 3.5
    Example 2, alpha = 1/2, beta = 1/4, gamma = 1, scores 4, 8, 0:
      init:   l = 4, v = 0
      t = 1:  predict 4;   v = (8-4)/4 + 0 = 1;        l = 6
      t = 2:  predict 7;   v = (0-6)/4 + 3/4 = -0.75;  l = 3
      t = 3:  predict 2.25"""
    cases = [((0.5, 0.5, 0.5), (4.0, 8.0, 2.0), [4.0, 7.0, 3.5], (4.0, -1.0)),
             ((0.5, 0.25, 1.0), (4.0, 8.0, 0.0), [4.0, 7.0, 2.25], (3.0, -0.75))]
    for (a, b, g), seq, want_pred, (want_l, want_v) in cases:
        l, v = init_fn(np.array([seq[0]]))
        preds = []
        for s in seq[1:]:
            preds.append(predict_fn(l, v, g)[0])
            l, v = update_fn(l, v, np.array([s]), a, b)
        preds.append(predict_fn(l, v, g)[0])
        if not (preds == want_pred and l[0] == want_l and v[0] == want_v):
            return False
    return True


def check_ema_constant(init_fn, predict_fn, update_fn):
    l, v = init_fn(np.array([3.25, -1.5]))
    for _ in range(20):
        if not np.array_equal(predict_fn(l, v, 0.75), np.array([3.25, -1.5])):
            return False
        l, v = update_fn(l, v, np.array([3.25, -1.5]), 0.4, 0.3)
    return True


def check_ema_ramp(init_fn, predict_fn, update_fn):
    """On a linear ramp y_t = a + b t the steady state has trend b / alpha and the
    prediction of step t+1 misses y_{t+1} by b (gamma - 1) / alpha (derived from the
    recurrences); it is exact when gamma = 1."""
    a, b = 2.0, 0.3
    for alpha, beta, gamma in [(0.5, 0.3, 0.0), (0.2, 0.5, 0.75), (0.8, 0.1, 1.0)]:
        l, v = init_fn(np.array([a]))
        for t in range(1, 400):
            l, v = update_fn(l, v, np.array([a + b * t]), alpha, beta)
        pred = predict_fn(l, v, gamma)[0]
        want = a + b * 400 + b * (gamma - 1.0) / alpha
        if abs(pred - want) > 1e-9 or abs(v[0] - b / alpha) > 1e-9:
            return False
    return True


def check_ema_s1(init_fn, predict_fn, update_fn, seed=7):
    """alpha = 1, gamma = 0 reduces the predictor to 'reuse the previous step's scores'
    (the paper's stage S1 baseline)."""
    r = _rng(seed)
    seq = r.standard_normal((10, 5))
    l, v = init_fn(seq[0])
    for t in range(1, 10):
        if not np.array_equal(predict_fn(l, v, 0.0), seq[t - 1]):
            return False
        l, v = update_fn(l, v, seq[t], 1.0, 0.3)
    return True


# ----------------------------------------------------------------------------- attention

def _sdpa_reference(q, k, v, num_tokens):
    """Dense attention by torch's library routine (CPU, float64) over the first
    num_tokens tokens; GQA by repeating each KV head G times."""
    hq, d = q.shape
    hkv = k.shape[0]
    g = hq // hkv
    kf = torch.from_numpy(k.reshape(hkv, -1, d)[:, :num_tokens]).repeat_interleave(g, dim=0)
    vf = torch.from_numpy(v.reshape(hkv, -1, d)[:, :num_tokens]).repeat_interleave(g, dim=0)
    qt = torch.from_numpy(q)[:, None, :]
    o = torch.nn.functional.scaled_dot_product_attention(qt[None], kf[None], vf[None])[0, :, 0]
    s = np.einsum("hd,htd->ht", q, kf.numpy()) / math.sqrt(d)
    return o.numpy(), scipy.special.logsumexp(s, axis=1)


def check_attend_dense(attend_fn, seed=8, g=4):
    """With every page selected the sparse output is dense attention (library SDPA),
    for a partial last page too; m + log l is the log-sum-exp of the logits."""
    r = _rng(seed)
    hkv, n, ps, d = 2, 5, 16, 32
    q = r.standard_normal((hkv * g, d))
    k = r.standard_normal((hkv, n, ps, d))
    v = r.standard_normal((hkv, n, ps, d))
    for num_tokens in (n * ps, n * ps - 9):
        o, m, l = attend_fn(q, k, v, [range(n)] * hkv, ps, num_tokens)
        o_ref, lse_ref = _sdpa_reference(q, k, v, num_tokens)
        if not (np.allclose(o, o_ref, atol=1e-12, rtol=0) and np.allclose(m + np.log(l), lse_ref, atol=1e-12)):
            return False
        s = np.einsum("hd,htd->ht", q, np.repeat(k.reshape(hkv, -1, d)[:, :num_tokens], g, axis=0)) / math.sqrt(d)
        if not np.allclose(m, s.max(axis=1), atol=1e-12, rtol=0):
            return False
    return True


def check_attend_subset(attend_fn, seed=9):
    """Attention over a page subset is dense attention over the concatenation of those
    pages only (library SDPA on the gathered tokens)."""
    r = _rng(seed)
    hkv, g, n, ps, d = 1, 2, 7, 16, 16
    q = r.standard_normal((g, d))
    k = r.standard_normal((hkv, n, ps, d))
    v = r.standard_normal((hkv, n, ps, d))
    pages = [1, 4, 6]
    o, m, l = attend_fn(q, k, v, [pages], ps, n * ps)
    o_ref, lse_ref = _sdpa_reference(q, k[:, pages], v[:, pages], len(pages) * ps)
    return np.allclose(o, o_ref, atol=1e-12) and np.allclose(m + np.log(l), lse_ref, atol=1e-12)


# ----------------------------------------------------------------------------- merge / repair

def check_merge_algebra(merge_fn, seed=10):
    """Associativity, commutativity and the identity of the partial-state merge, and
    merged states reproduce the log-sum-exp and the weighted mean they stand for."""
    r = _rng(seed)

    def rand_state():
        return r.standard_normal((3, 4)), r.standard_normal(3) * 3, np.exp(r.standard_normal(3))

    a, b, c = rand_state(), rand_state(), rand_state()
    e = (np.zeros((3, 4)), np.full(3, -np.inf), np.zeros(3))
    ab_c = merge_fn(merge_fn(a, b), c)
    a_bc = merge_fn(a, merge_fn(b, c))
    ba = merge_fn(b, a)
    ab = merge_fn(a, b)
    ok = all(np.allclose(x, y, atol=1e-12) for x, y in zip(ab_c, a_bc))
    ok &= all(np.allclose(x, y, atol=1e-12) for x, y in zip(ab, ba))
    ae = merge_fn(a, e)
    ok &= all(np.allclose(x, y, atol=0) for x, y in zip(ae, a))
    lse = scipy.special.logsumexp(np.stack([a[1] + np.log(a[2]), b[1] + np.log(b[2])]), axis=0)
    ok &= np.allclose(ab[1] + np.log(ab[2]), lse, atol=1e-12)
    wa = np.exp(a[1] + np.log(a[2]) - lse)
    ok &= np.allclose(ab[0], wa[:, None] * a[0] + (1 - wa)[:, None] * b[0], atol=1e-12)
    return bool(ok)


def check_merge_union(attend_fn, merge_fn, seed=11):
    """Merging attention over disjoint page sets gives attention over their union."""
    r = _rng(seed)
    hkv, g, n, ps, d = 2, 2, 6, 16, 16
    q = r.standard_normal((hkv * g, d))
    k = r.standard_normal((hkv, n, ps, d))
    v = r.standard_normal((hkv, n, ps, d)) * 2
    x, y = [[0, 2], [1]], [[3, 5], [2, 4]]
    sx = attend_fn(q, k, v, x, ps, n * ps)
    sy = attend_fn(q, k, v, y, ps, n * ps)
    su = attend_fn(q, k, v, [a + b for a, b in zip(x, y)], ps, n * ps)
    mg = merge_fn(sx, sy)
    return all(np.allclose(p, w, atol=1e-12) for p, w in zip(mg, su))


def check_speculate_repair(spec_repair_fn, attend_fn, seed=12):
    """For EVERY predicted subset P of a tiny cache, speculation over P followed by the
    repair recurrence over A \\ P gives attention over exactly A (or over P u A when
    wasted pages are kept)."""
    r = _rng(seed)
    hkv, g, n, ps, d = 1, 2, 5, 16, 8
    q = r.standard_normal((g, d)) * 2
    k = r.standard_normal((hkv, n, ps, d))
    v = r.standard_normal((hkv, n, ps, d))
    num_tokens = n * ps - 5
    a = [0, 2, 4]
    ref = attend_fn(q, k, v, [a], ps, num_tokens)
    for p in itertools.chain.from_iterable(itertools.combinations(range(n), c) for c in range(n + 1)):
        got = spec_repair_fn(q, k, v, [a], [list(p)], ps, num_tokens, keep_wasted=False)
        if not all(np.allclose(x, y, atol=1e-12) for x, y in zip(got, ref)):
            return False
        kw = spec_repair_fn(q, k, v, [a], [list(p)], ps, num_tokens, keep_wasted=True)
        ref_u = attend_fn(q, k, v, [sorted(set(a) | set(p))], ps, num_tokens)
        if not all(np.allclose(x, y, atol=1e-12) for x, y in zip(kw, ref_u)):
            return False
    return True


# ----------------------------------------------------------------------------- calibration

def check_calibrate_closed_form(objective_fn, calibrate_fn, grid):
    """Three rows of two blocks, k = |P| = 1, scores s0 = (1, 3), s1 = (2, 1), s2 = (5, 1).
    Worked by hand from Eqs. (2)-(3): the state after row 1 is v = beta (s1 - s0),
    l = s0 + alpha (s1 - s0), so the prediction of row 2 is s0 + c (s1 - s0) with
    c = alpha + gamma beta: block 0 is predicted iff 1 + c > 3 - 2c, i.e. c > 2/3.  Row 1's
    prediction is s0 (block 1) while A_1 = {0}: no hit.  Row 2's A_2 = {0}.  So Eq. (4) is
    1/2 where alpha + gamma beta > 2/3 and 0 elsewhere (no grid point has c = 2/3), and
    Eq. (5)'s first maximiser in grid order (alpha outer, then beta, then gamma) is
    (0.4, 0.4, 0.75), the first point with c > 2/3."""
    traj = np.array([[1.0, 3.0], [2.0, 1.0], [5.0, 1.0]])
    for a, b, g in grid:
        want = 0.5 if a + g * b > 2.0 / 3.0 else 0.0
        if abs(objective_fn(traj, 1, (a, b, g)) - want) > 1e-12:
            return False
    best, val = calibrate_fn(traj, 1, grid)
    return tuple(best) == (0.4, 0.4, 0.75) and abs(val - 0.5) <= 1e-12


def check_calibrate_all_tied(calibrate_fn, grid, seed=13):
    """A constant trajectory is predicted exactly by every theta (Eq. (4) = 1 for all), so
    Eq. (5) returns the first grid point."""
    row = np.abs(_rng(seed).standard_normal(10)) + 0.1
    best, val = calibrate_fn(np.tile(row, (5, 1)), 3, grid)
    return tuple(best) == tuple(grid[0]) and abs(val - 1.0) <= 1e-12


def check_calibration_formation(objective_fn, grid):
    """Block 1 forms at row 1 (its row-0 entry is junk that must never be read).  By hand,
    k = |P| = 1, rows (2, junk), (2, 3), (2, 3): at row 1 only block 0 has a state, so
    P_1 = {0} while A_1 = {1} (no hit); block 1's state starts at row 1 as (3, 0) and block
    0 stays at (2, 0), so P_2 = {1} = A_2.  Eq. (4) is 1/2 for every theta.  A state begun at
    row 0 -- from the junk, or from a placeholder 0 -- predicts row 1 or row 2 differently
    for some theta."""
    for junk in (100.0, 0.0):
        traj = np.array([[2.0, junk], [2.0, 3.0], [2.0, 3.0]])
        for theta in grid:
            if abs(objective_fn(traj, 1, theta, None, [0, 1]) - 0.5) > 1e-12:
                return False
    return True


def check_criticality_mean_bounds(meta_mean_fn, qbar_fn, score_fn, seed=14):
    """The block-mean score lies between the smallest and the largest token score of the
    block (a mean of the tokens' q-bar . k), equals it for a block of identical tokens, and
    ignores tokens at or past num_tokens."""
    r = _rng(seed)
    k = r.standard_normal((2, 4, 16, 8))
    q = r.standard_normal((6, 8))
    nt = 3 * 16 + 5
    kk = k.copy()
    kk[:, 3, 5:] = 1e6
    s = score_fn(qbar_fn(q, 2), meta_mean_fn(kk, 16, nt))
    qb = qbar_fn(q, 2)
    for h in range(2):
        for p in range(4):
            valid = 16 if p < 3 else 5
            tok = k[h, p, :valid] @ qb[h]
            if not (tok.min() - 1e-12 <= s[h, p] <= tok.max() + 1e-12):
                return False
    same = np.broadcast_to(k[0, 0, :1], (1, 1, 16, 8)).copy()
    s1 = score_fn(qbar_fn(q[:3], 1), meta_mean_fn(same, 16, 16))
    return abs(s1[0, 0] - float(same[0, 0, 0] @ qbar_fn(q[:3], 1)[0])) <= 1e-12
