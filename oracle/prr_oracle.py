"""Plain, slow, float64 CPU oracle of the speculate-reuse-repair decode path.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path imports, calls or links this
module; only the test suite, the smoke check and the bench's CPU-baseline leg do.
It shares no code with the HIP library.

What it computes, in the paper's notation (citations are to the paper's sections,
equations and appendix):

* page metadata: channel-wise min m_p and max M_p of each page's keys, per KV head
  (Appendix A.1, "Extend Quest to GQA"); the block-mean variant stands in for
  InfLLM-v2's mean-compressed blocks (Section 2.1);
* representative query  Qbar = (1/G) sum_g Q_g  of each KV head's group (A.1);
* criticality  s_p = sum_i max(Qbar_i m_{p,i}, Qbar_i M_{p,i})  (A.1); block-mean
  variant  s_b = Qbar . kbar_b;
* top-K page selection per KV head, shared by the group (A.1, Section 1); ties go to
  the lower page index; forced pages are always selected;
* the EMA predictor: initialisation, prediction Eq. (2), update Eq. (3) (Section 4.1),
  and the predicted set P = top-|P| pages by predicted score with |P| <= delta |A|
  (Eq. (1));
* missed and wasted sets M = A \\ P, N = P \\ A (Section 3);
* the attention output over exactly the tokens of the selected pages, computed
  directly from its definition (softmax of q.k / sqrt(d), then a weighted sum of v);
* the two-state merge of partial online-softmax states and the block-by-block repair
  recurrence, Eqs. (6)-(8) (Section 4.3), used only to check the merge algebra and the
  speculate-then-repair identity;
* the calibration objective H(theta; IS), Eq. (4), and its grid arg-max, Eq. (5)
  (Section 4.2).

Where the paper is silent the readings are: contiguous query-head groups (head j
belongs to KV head j // G); softmax scale 1/sqrt(d) on attention logits only (the
criticality score is unscaled); (m, l) in natural-log units of the scaled logits with
o normalised; the top-K decision is taken on the float32-rounded score (the kernel's
precision), ties to the lower page index; a partial last page uses its valid tokens
only; the EMA trend update reads the previous level, so v is updated before l.

Parity: every function here is pinned by a CPU test against a property the paper or
mathematics fixes (bounds, closed forms, brute force, a library routine); none is
"parity unpinned".
"""
from __future__ import annotations

import itertools
import math
from typing import Iterable, List, Optional, Sequence, Tuple

import numpy as np

NEG_INF = -np.inf


# ----------------------------------------------------------------------------- metadata (A.1)

def _valid_tokens(page: int, page_size: int, num_tokens: int) -> int:
    return max(0, min(page_size, num_tokens - page * page_size))


def page_metadata_minmax(k: np.ndarray, page_size: int, num_tokens: int) -> Tuple[np.ndarray, np.ndarray]:
    """Channel-wise min and max of the keys of each page (Appendix A.1).

    k: [Hkv][N][page_size][d] float64 in logical page order.  Tokens at or beyond
    ``num_tokens`` are not part of the cache and do not contribute.
    Returns (mins, maxs), each [Hkv][N][d]; a page with no valid token gets +inf / -inf.
    """
    hkv, n, ps, d = k.shape
    assert ps == page_size
    mins = np.full((hkv, n, d), np.inf)
    maxs = np.full((hkv, n, d), -np.inf)
    for p in range(n):
        valid = _valid_tokens(p, page_size, num_tokens)
        if valid:
            mins[:, p] = k[:, p, :valid].min(axis=1)
            maxs[:, p] = k[:, p, :valid].max(axis=1)
    return mins, maxs


def page_metadata_mean(k: np.ndarray, page_size: int, num_tokens: int) -> np.ndarray:
    """Mean key of each block over its valid tokens: the block compression of
    mean-pooled block selection (Section 2.1).  Returns [Hkv][N][d]."""
    hkv, n, ps, d = k.shape
    out = np.zeros((hkv, n, d))
    for p in range(n):
        valid = _valid_tokens(p, page_size, num_tokens)
        if valid:
            out[:, p] = k[:, p, :valid].mean(axis=1)
    return out


# ----------------------------------------------------------------------------- scoring (A.1)

def representative_query(q: np.ndarray, num_kv_heads: int) -> np.ndarray:
    """Qbar for each KV head: the mean of the G query heads sharing it (Appendix A.1).

    q: [Hq][d].  Query head j belongs to KV head j // G.  Returns [Hkv][d].
    """
    hq, d = q.shape
    g = hq // num_kv_heads
    qbar = np.zeros((num_kv_heads, d))
    for h in range(num_kv_heads):
        for j in range(h * g, (h + 1) * g):
            qbar[h] += q[j]
        qbar[h] /= g
    return qbar


def criticality_minmax(qbar: np.ndarray, mins: np.ndarray, maxs: np.ndarray) -> np.ndarray:
    """Quest criticality per (KV head, page): sum over channels of the larger of
    Qbar_i * m_{p,i} and Qbar_i * M_{p,i} (Appendix A.1).  Unscaled.  Returns [Hkv][N]."""
    lo = qbar[:, None, :] * mins
    hi = qbar[:, None, :] * maxs
    return np.maximum(lo, hi).sum(axis=-1)


def criticality_mean(qbar: np.ndarray, means: np.ndarray) -> np.ndarray:
    """Block score of mean-pooled selection: Qbar . kbar_b.  Returns [Hkv][N]."""
    return np.einsum("hd,hnd->hn", qbar, means)


# ----------------------------------------------------------------------------- selection

def decision_keys(scores: np.ndarray) -> np.ndarray:
    """The value a top-K decision compares: the score rounded to float32."""
    return np.asarray(scores, dtype=np.float64).astype(np.float32)


def select_topk(scores_row: np.ndarray, k: int, forced: Sequence[int] = (),
                forced_in_budget: bool = True) -> np.ndarray:
    """Top-K pages of one KV head, by (float32 score descending, page index ascending).

    Forced pages are always selected.  With ``forced_in_budget`` the result has k
    pages in total, otherwise k pages beyond the forced ones.  Returns the selected
    page indices in ascending order.
    """
    n = scores_row.shape[0]
    forced = sorted(set(int(f) for f in forced))
    extra = k - len(forced) if forced_in_budget else k
    extra = max(0, extra)
    keys = decision_keys(scores_row)
    cand = [p for p in range(n) if p not in set(forced)]
    # rank candidates: higher key first, then lower index first
    cand.sort(key=lambda p: (-float(keys[p]), p))
    chosen = cand[:extra]
    return np.array(sorted(forced + chosen), dtype=np.int64)


# ----------------------------------------------------------------------------- EMA predictor (4.1)

def ema_init(scores: np.ndarray) -> Tuple[np.ndarray, np.ndarray]:
    """A page's state when it first enters the cache: level = its score, trend = 0."""
    level = np.array(scores, dtype=np.float64, copy=True)
    return level, np.zeros_like(level)


def ema_predict(level: np.ndarray, trend: np.ndarray, gamma: float) -> np.ndarray:
    """Eq. (2): predicted score of step t from the state after step t-1."""
    return level + gamma * trend


def ema_update(level: np.ndarray, trend: np.ndarray, scores: np.ndarray,
               alpha: float, beta: float) -> Tuple[np.ndarray, np.ndarray]:
    """Eq. (3): the trend first (it reads the previous level), then the level."""
    new_trend = beta * (scores - level) + (1.0 - beta) * trend
    new_level = alpha * scores + (1.0 - alpha) * level
    return new_level, new_trend


def predicted_set(pred_row: np.ndarray, p_select: int, forced: Sequence[int] = (),
                  forced_in_budget: bool = True) -> np.ndarray:
    """P: the |P| pages with the highest predicted score (Eq. (1) with a fixed budget)."""
    return select_topk(pred_row, p_select, forced, forced_in_budget)


def missed_and_wasted(selected: Iterable[int], predicted: Iterable[int]) -> Tuple[np.ndarray, np.ndarray]:
    """Section 3: missed M = A \\ P (on the critical path), wasted N = P \\ A."""
    a, p = set(int(x) for x in selected), set(int(x) for x in predicted)
    return np.array(sorted(a - p), dtype=np.int64), np.array(sorted(p - a), dtype=np.int64)


def hit_rate(selected: Iterable[int], predicted: Iterable[int]) -> float:
    a, p = set(int(x) for x in selected), set(int(x) for x in predicted)
    return len(a & p) / len(a) if a else 1.0


# ----------------------------------------------------------------------------- attention

def page_tokens(pages: Iterable[int], page_size: int, num_tokens: int) -> np.ndarray:
    """Token positions covered by the given logical pages (valid tokens only)."""
    toks = []
    for p in sorted(set(int(x) for x in pages)):
        for r in range(page_size):
            t = p * page_size + r
            if t < num_tokens:
                toks.append(t)
    return np.array(toks, dtype=np.int64)


def attend(q: np.ndarray, k: np.ndarray, v: np.ndarray, pages_per_kv_head: Sequence[Iterable[int]],
           page_size: int, num_tokens: int) -> Tuple[np.ndarray, np.ndarray, np.ndarray]:
    """Attention of each query head over exactly the tokens of its KV head's pages.

    q: [Hq][d]; k, v: [Hkv][N][page_size][d] (logical order).  For query head j of KV
    head h = j // G over tokens T of h's pages:
        S_t = q_j . k_t / sqrt(d),  m = max_t S_t,  l = sum_t exp(S_t - m),
        o = sum_t exp(S_t - m) v_t / l.
    An empty token set gives (o = 0, m = -inf, l = 0).
    Returns o [Hq][d], m [Hq], l [Hq] in float64.
    """
    hq, d = q.shape
    hkv = k.shape[0]
    g = hq // hkv
    kf = k.reshape(hkv, -1, d)
    vf = v.reshape(hkv, -1, d)
    o = np.zeros((hq, d))
    m = np.full(hq, NEG_INF)
    l = np.zeros(hq)
    scale = 1.0 / math.sqrt(d)
    for h in range(hkv):
        toks = page_tokens(pages_per_kv_head[h], page_size, num_tokens)
        if toks.size == 0:
            continue
        kt, vt = kf[h, toks], vf[h, toks]
        for j in range(h * g, (h + 1) * g):
            s = (kt @ q[j]) * scale
            m[j] = s.max()
            w = np.exp(s - m[j])
            l[j] = w.sum()
            o[j] = (w @ vt) / l[j]
    return o, m, l


def merge_two(a: Tuple[np.ndarray, np.ndarray, np.ndarray],
              b: Tuple[np.ndarray, np.ndarray, np.ndarray]) -> Tuple[np.ndarray, np.ndarray, np.ndarray]:
    """Merge two normalised partial states (Eqs. (6)-(8) for two arbitrary states).

    m' = max(m_a, m_b); l' = e^{m_a-m'} l_a + e^{m_b-m'} l_b;
    o' = (e^{m_a-m'} l_a o_a + e^{m_b-m'} l_b o_b) / l'.  The empty state
    (o = 0, m = -inf, l = 0) is the identity.
    """
    oa, ma, la = a
    ob, mb, lb = b
    oa, ob = np.atleast_2d(oa), np.atleast_2d(ob)
    ma, mb, la, lb = (np.atleast_1d(x).astype(np.float64) for x in (ma, mb, la, lb))
    mo = np.maximum(ma, mb)
    with np.errstate(invalid="ignore"):
        wa = np.where(la > 0, np.exp(ma - mo) * la, 0.0)
        wb = np.where(lb > 0, np.exp(mb - mo) * lb, 0.0)
    lo = wa + wb
    oo = np.zeros_like(oa)
    nz = lo > 0
    oo[nz] = (wa[nz, None] * oa[nz] + wb[nz, None] * ob[nz]) / lo[nz, None]
    return oo, np.where(nz, mo, NEG_INF), lo


def merge_states(states: Sequence[Tuple[np.ndarray, np.ndarray, np.ndarray]]):
    """Left fold of merge_two over a list of partial states."""
    out = None
    for s in states:
        out = s if out is None else merge_two(out, s)
    return out


def repair_block(state, q_row: np.ndarray, k_block: np.ndarray, v_block: np.ndarray):
    """One step of the repair recurrence of Section 4.3 for one query head.

    state = (O, l, m) over the blocks attended so far (O normalised); the block's
    logits S_j = q . k_j / sqrt(d); with its local max m~ and l~ = sum_j e^{S_j - m~}:
      Eq. (6)  m' = max(m, m~)
      Eq. (7)  l' = e^{m - m'} l + e^{m~ - m'} l~
      Eq. (8)  O' = e^{m - m'} l / l' * O + e^{m~ - m'} / l' * sum_j e^{S_j - m~} V_j
    Returns the new (O, l, m).
    """
    o, l, m = state
    d = q_row.shape[0]
    s = (k_block @ q_row) / math.sqrt(d)
    if s.size == 0:
        return o, l, m
    mt = s.max()
    e = np.exp(s - mt)
    lt = e.sum()
    m_new = max(m, mt)
    a = math.exp(m - m_new) * l if l > 0 else 0.0
    b = math.exp(mt - m_new)
    l_new = a + b * lt
    o_new = (a / l_new) * o + (b / l_new) * (e @ v_block)
    return o_new, l_new, m_new


def speculate_then_repair(q: np.ndarray, k: np.ndarray, v: np.ndarray, selected, predicted,
                          page_size: int, num_tokens: int, keep_wasted: bool = False):
    """The method's route to the output, for checking it against the definition:
    attention over the speculated pages (P, or P restricted to A when the output
    must cover exactly A), then the repair recurrence over each missed page."""
    hq, d = q.shape
    hkv = k.shape[0]
    g = hq // hkv
    o = np.zeros((hq, d))
    m = np.full(hq, NEG_INF)
    l = np.zeros(hq)
    for h in range(hkv):
        a, p = set(int(x) for x in selected[h]), set(int(x) for x in predicted[h])
        spec = p if keep_wasted else (p & a)
        missed = sorted(a - p)
        os_, ms_, ls_ = attend(q[h * g:(h + 1) * g], k[h:h + 1], v[h:h + 1], [spec], page_size, num_tokens)
        for jj in range(g):
            st = (os_[jj], ls_[jj], ms_[jj])
            for pg in missed:
                toks = page_tokens([pg], page_size, num_tokens) - pg * page_size
                st = repair_block(st, q[h * g + jj], k[h, pg, toks], v[h, pg, toks])
            o[h * g + jj], l[h * g + jj], m[h * g + jj] = st
    return o, m, l


# ----------------------------------------------------------------------------- calibration (4.2)

THETA_GRID = [(a, b, c)
              for a in (0.2, 0.4, 0.6, 0.8)
              for b in (0.1, 0.2, 0.3, 0.4, 0.5)
              for c in (0.0, 0.25, 0.5, 0.75)]


def calibration_objective(is_matrix: np.ndarray, k: int, theta, p_select: Optional[int] = None,
                          form_row: Optional[Sequence[int]] = None) -> float:
    """Eq. (4): the score-weighted hit rate of the predictor simulated over a prefill
    trajectory of score vectors (rows = prefill tokens phi, columns = blocks b).

    Blocks form as the prefill grows: block b exists from row form_row[b] on (default:
    every block from row 0).  As Section 4.1 initialises a block when it enters the
    cache, block b's state is (level = IS_{phi,b}, trend = 0) at phi = form_row[b], and
    the EMA of Eqs. (2)-(3) runs from there.  At row phi, A_phi is the top-k of the
    blocks that exist, P_phi the top-|P| predictions of the blocks that already had a
    state before phi (a block cannot be predicted at the row it forms); entries of
    blocks that do not exist yet are never read.  The mean runs over the rows that have
    a prediction (phi >= 1); a row whose selected scores sum to 0 contributes 0.
    """
    alpha, beta, gamma = theta
    p_select = k if p_select is None else p_select
    n_rows, n_blocks = is_matrix.shape
    born = np.zeros(n_blocks, dtype=np.int64) if form_row is None else np.asarray(form_row, dtype=np.int64)
    level = np.zeros(n_blocks)
    trend = np.zeros(n_blocks)
    has_state = np.zeros(n_blocks, dtype=bool)
    total, count = 0.0, 0
    for phi in range(n_rows):
        row = is_matrix[phi]
        exists = born <= phi
        if phi >= 1:
            pred = ema_predict(level, trend, gamma)
            live = np.flatnonzero(exists)
            a = live[select_topk(row[live], k)]
            old = np.flatnonzero(has_state)
            p = old[predicted_set(pred[old], p_select)]
            denom = row[a].sum()
            total += row[np.intersect1d(a, p)].sum() / denom if denom != 0.0 else 0.0
            count += 1
            level[has_state], trend[has_state] = ema_update(level[has_state], trend[has_state], row[has_state],
                                                            alpha, beta)
        new = exists & ~has_state
        level[new], trend[new] = ema_init(row[new])
        has_state |= new
    return total / max(count, 1)


def calibrate(is_matrix: np.ndarray, k: int, grid=THETA_GRID, p_select: Optional[int] = None,
              form_row: Optional[Sequence[int]] = None):
    """Eq. (5): the grid point with the largest objective (first one on ties)."""
    best, best_val = None, -np.inf
    for theta in grid:
        val = calibration_objective(is_matrix, k, theta, p_select, form_row)
        if val > best_val:
            best, best_val = theta, val
    return best, best_val


# ----------------------------------------------------------------------------- one decode step

def serial_step(q: np.ndarray, k: np.ndarray, v: np.ndarray, page_size: int, num_tokens: int,
                k_select: int, forced: Sequence[int] = (), forced_in_budget: bool = True,
                meta_kind: str = "minmax", meta=None):
    """One layer's select-then-attend step: metadata -> Qbar -> scores -> top-K ->
    attention over exactly the selected pages.  Returns (scores, selected, (o, m, l))."""
    hkv = k.shape[0]
    if meta is None:
        meta = (page_metadata_minmax(k, page_size, num_tokens) if meta_kind == "minmax"
                else page_metadata_mean(k, page_size, num_tokens))
    qbar = representative_query(q, hkv)
    scores = criticality_minmax(qbar, *meta) if meta_kind == "minmax" else criticality_mean(qbar, meta)
    selected = [select_topk(scores[h], k_select, forced, forced_in_budget) for h in range(hkv)]
    return scores, selected, attend(q, k, v, selected, page_size, num_tokens)


def all_subsets(items: Sequence[int]):
    for r in range(len(items) + 1):
        for c in itertools.combinations(items, r):
            yield list(c)
