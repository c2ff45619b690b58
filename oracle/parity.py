"""Acceptance checks: GPU outputs against the CPU oracle.

TEST INFRASTRUCTURE ONLY (tests, smoke check, benchmark baseline). Takes numpy
arrays; never imports the GPU package.

Tolerances (floating point fixed at 1e-5 relative for decisions and 1e-4 for
values):
  rel(a, b) = |a - b| / max(|a|, |b|, f), f = 1 for squared distances of
  unit-scale embeddings (fp32 cancellation in |q|^2 + |x|^2 - 2<q,x> is
  absolute, about 1e-6 at d = 768); f = 1e-2 for Eq. 1 scores, which are
  unit-scale sums of terms in [0, 1] (1 - C/Cmax near the maximum loses all
  relative precision in fp32, leaving ~1e-7 absolute error); f = 1e-6 for
  predictions and state.
  * neighbours: an index in one list but not the other must sit within 1e-5 of
    the oracle's k-th distance (a boundary near-tie); order may differ only
    among near-equal distances; GPU distances of listed rows within 1e-5.
  * predictions: teacher-forced, recomputed by the oracle from the GPU's own
    neighbour list (and, for the inverse-distance weights, the GPU's own
    distances), within 1e-4.
  * scores: from the GPU's predictions, within 1e-4.
  * assignment: teacher-forced replay; each GPU pick must be the oracle's pick
    or score within 1e-5 of the oracle's best (a near tie, counted); the
    replay continues with the GPU's pick; the state after the batch within
    1e-4. Free-running (the oracle on its own): bit-identical picks when the
    replay saw no near tie.
  * LPT order: the oracle's order from the GPU's predictions, bit-identical
    to the GPU's (max and comparisons are exact in both precisions).
  * candidate sets: both sides take the admission test in fp32, so the set
    must be identical: -1 exactly when it is empty, else a pick inside it.
"""
from __future__ import annotations

import numpy as np

from . import assign as _assign, knn as _knn, lpt_order as _lpt_order, predict as _predict, \
    score as _score, score_row as _score_row

DIST_RTOL = 1e-5
DIST_FLOOR = 1.0
VAL_RTOL = 1e-4
VAL_FLOOR = 1e-6
SCORE_FLOOR = 1e-2
PICK_RTOL = 1e-5


def rel(a, b, floor):
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    return np.abs(a - b) / np.maximum(np.maximum(np.abs(a), np.abs(b)), floor)


def check_neighbours(g_idx, g_dist, o_idx, o_dist, rows=None, label=""):
    """Compare per-request neighbour lists. ``rows`` maps row i of the oracle
    arrays to row rows[i] of the GPU arrays (sampled checks). Returns the number
    of boundary near-tie substitutions."""
    g_idx = np.asarray(g_idx)
    g_dist = None if g_dist is None else np.asarray(g_dist, np.float64)
    o_idx = np.asarray(o_idx)
    o_dist = np.asarray(o_dist, np.float64)
    B, k = o_idx.shape
    rows = np.arange(B) if rows is None else np.asarray(rows)
    ties = 0
    for i in range(B):
        gi = g_idx[rows[i]]
        oi = o_idx[i]
        od = dict(zip(oi.tolist(), o_dist[i].tolist()))
        kth = o_dist[i, -1]
        assert len(set(gi.tolist())) == k, f"{label} row {rows[i]}: duplicate indices {gi}"
        only_g = set(gi.tolist()) - set(oi.tolist())
        only_o = set(oi.tolist()) - set(gi.tolist())
        for j in only_o:
            assert rel(od[j], kth, DIST_FLOOR) <= DIST_RTOL, \
                f"{label} row {rows[i]}: oracle neighbour {j} (d={od[j]}) missing, k-th {kth}"
        if g_dist is not None:
            gd = g_dist[rows[i]]
            for pos, j in enumerate(gi.tolist()):
                if j in od:
                    assert rel(gd[pos], od[j], DIST_FLOOR) <= DIST_RTOL, \
                        f"{label} row {rows[i]}: idx {j} gpu d={gd[pos]} oracle d={od[j]}"
                else:
                    # a substituted row: its distance must tie the oracle's k-th
                    assert rel(gd[pos], kth, DIST_FLOOR) <= DIST_RTOL, \
                        f"{label} row {rows[i]}: extra idx {j} d={gd[pos]} vs k-th {kth}"
            assert np.all(np.diff(gd) >= -1e-12), f"{label} row {rows[i]}: not sorted {gd}"
        # order: the GPU list sorted by oracle distance where known must agree up to near ties
        for pos, j in enumerate(gi.tolist()):
            if j in od and oi[pos] != j:
                assert rel(od[j], o_dist[i, pos], DIST_FLOOR) <= DIST_RTOL, \
                    f"{label} row {rows[i]} pos {pos}: gpu {j} oracle {oi[pos]}"
        ties += len(only_g)
    return ties


def check_predictions(g_idx, g_qhat, g_lhat, qual, length, label="", g_dist=None,
                      weighting="uniform"):
    """Teacher-forced: the oracle averages the GPU's own neighbour lists (with
    the GPU's own distances for the weighted average)."""
    qh, lh = _predict(np.asarray(g_idx), qual, length,
                      dist=None if g_dist is None else np.asarray(g_dist, np.float64),
                      weighting=weighting)
    eq = rel(g_qhat, qh, VAL_FLOOR)
    el = rel(g_lhat, lh, VAL_FLOOR)
    assert eq.max() <= VAL_RTOL, f"{label} q_hat rel err {eq.max()}"
    assert el.max() <= VAL_RTOL, f"{label} l_hat rel err {el.max()}"
    return float(max(eq.max(), el.max()))


def check_scores(g_S0, g_qhat, g_lhat, plen, inst, weights, label=""):
    S0 = _score(np.asarray(g_qhat, np.float64), np.asarray(g_lhat, np.float64), plen, inst, weights)
    e = rel(g_S0, S0, SCORE_FLOOR)
    assert e.max() <= VAL_RTOL, f"{label} S0 rel err {e.max()} at {np.unravel_index(e.argmax(), e.shape)}"
    return float(e.max())


def check_assign(g_assign, g_chosen, g_qhat, g_lhat, plen, inst, weights, g_final_p=None,
                 g_final_a=None, p0=None, a0=None, label="", order="arrival", g_order=None,
                 budget=None, mask=None):
    """Teacher-forced replay of the greedy loop. Returns the near-tie count.

    ``order`` "lpt" replays in the oracle's LPT order of the GPU's predictions,
    which must equal ``g_order`` when given; ``budget`` [B] and ``mask`` [I]
    restrict the candidate sets as in the GPU call."""
    qh = np.asarray(g_qhat, np.float64)
    lh = np.asarray(g_lhat, np.float64)
    g_assign = np.asarray(g_assign)
    B = qh.shape[0]
    p = np.asarray(inst.prefill_q if p0 is None else p0, np.float64).copy()
    a = np.asarray(inst.decode_q if a0 is None else a0, np.float64).copy()
    model = np.asarray(inst.model)
    seq = _lpt_order(lh) if order == "lpt" else np.arange(B)
    if g_order is not None:
        assert np.array_equal(np.asarray(g_order), seq), \
            f"{label} processing order differs at step {int(np.argmax(np.asarray(g_order) != seq))}"
    budget = None if budget is None else np.asarray(budget, np.float32)
    ties = 0
    for r in seq:
        S, _, _, cand = _score_row(qh[r], lh[r], plen[r], inst, p, a, weights,
                                   budget_r=None if budget is None else budget[r], mask=mask,
                                   with_candidates=True)
        ig = int(g_assign[r])
        if not cand.any():
            assert ig == -1, f"{label} request {r}: no candidate, gpu picked {ig}"
            if g_chosen is not None:
                assert np.isnan(g_chosen[r]), f"{label} request {r}: chosen {g_chosen[r]}"
            continue
        assert 0 <= ig < S.shape[0], f"{label} request {r}: pick {ig} out of range"
        assert cand[ig], f"{label} request {r}: gpu picked {ig}, not a candidate"
        io = int(np.nanargmax(S))
        if ig != io:
            gap = S[io] - S[ig]
            assert gap <= PICK_RTOL * max(abs(S[io]), SCORE_FLOOR), \
                f"{label} request {r}: gpu picked {ig} (S={S[ig]}) oracle {io} (S={S[io]})"
            ties += 1
        if g_chosen is not None:
            assert rel(g_chosen[r], S[ig], SCORE_FLOOR) <= VAL_RTOL, \
                f"{label} request {r}: chosen score {g_chosen[r]} vs {S[ig]}"
        p[ig] += plen[r]
        a[ig] += lh[r, model[ig]]
    if g_final_p is not None:
        e = rel(g_final_p, p, VAL_FLOOR)
        assert e.max() <= VAL_RTOL, f"{label} final prefill state rel err {e.max()}"
    if g_final_a is not None:
        e = rel(g_final_a, a, VAL_FLOOR)
        assert e.max() <= VAL_RTOL, f"{label} final decode state rel err {e.max()}"
    return ties


def free_running(queries, bank, k, qual, length, plen, inst, weights, nthreads=1,
                 order="arrival", weighting="uniform", budget=None, mask=None):
    """The oracle alone: its own KNN, predictions and greedy loop."""
    idx, dist = _knn(queries, bank, k, nthreads=nthreads)
    qh, lh = _predict(idx, qual, length, dist=dist, weighting=weighting)
    res = _assign(qh, lh, plen, inst, weights, order=order, budget=budget, mask=mask)
    res.update(idx=idx, dist=dist, q_hat=qh, l_hat=lh)
    return res
