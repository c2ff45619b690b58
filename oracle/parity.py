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
  * candidate sets (Alg. 1 budget filter on the Eq. 2 cost): the oracle
    admits an instance when its exact (fp64) cost is at most the budget; the
    GPU decides the same test in fp32. An instance whose exact cost lies
    within 1e-5 relative of the budget (floor 1e-6) is a boundary near-tie
    and may be decided either way: the replay accepts the GPU's pick if some
    admission of the boundary instances explains it (each such request is
    counted); every other instance must be admitted exactly as the oracle
    admits it: -1 exactly when the set is empty, else a pick inside it.
  * exact ties: where the oracle's fp64 distances of two rows are exactly
    equal (a duplicated row, for instance), the lower bank index must come
    first, also across the k-th position.
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
ADMIT_RTOL = 1e-5
ADMIT_MAX_BOUNDARY = 8     # boundary instances per request the replay enumerates


def rel(a, b, floor):
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    return np.abs(a - b) / np.maximum(np.maximum(np.abs(a), np.abs(b)), floor)


def check_neighbours(g_idx, g_dist, o_idx, o_dist, rows=None, label=""):
    """Compare per-request neighbour lists. ``rows`` maps row i of the oracle
    arrays to row rows[i] of the GPU arrays (sampled checks). The oracle lists
    may be longer than the GPU's k (the oracle run with a larger k): the extra
    entries give the exact distance of a row the GPU took in place of one of
    the oracle's k, and decide exact ties across the k-th position. Returns the
    number of boundary near-tie substitutions."""
    g_idx = np.asarray(g_idx)
    g_dist = None if g_dist is None else np.asarray(g_dist, np.float64)
    o_idx = np.asarray(o_idx)
    o_dist = np.asarray(o_dist, np.float64)
    B, k_ext = o_idx.shape
    k = g_idx.shape[1]
    assert k_ext >= k, f"{label}: oracle lists shorter than the GPU's"
    rows = np.arange(B) if rows is None else np.asarray(rows)
    ties = 0
    for i in range(B):
        r = rows[i]
        gi = g_idx[r].tolist()
        oi = o_idx[i, :k].tolist()
        od = dict(zip(o_idx[i].tolist(), o_dist[i].tolist()))   # every known oracle distance
        kth = o_dist[i, k - 1]
        last = o_dist[i, -1]
        assert len(set(gi)) == k, f"{label} row {r}: duplicate indices {gi}"
        only_g = set(gi) - set(oi)
        only_o = set(oi) - set(gi)
        for j in only_o:
            assert rel(od[j], kth, DIST_FLOOR) <= DIST_RTOL, \
                f"{label} row {r}: oracle neighbour {j} (d={od[j]}) missing, k-th {kth}"
        for j in only_g:
            if j in od:
                # a substitution: a boundary near-tie, and never a higher index
                # for a lower one at exactly the same distance
                assert rel(od[j], kth, DIST_FLOOR) <= DIST_RTOL, \
                    f"{label} row {r}: extra idx {j} (oracle d={od[j]}) vs k-th {kth}"
                for a in only_o:
                    assert od[a] != od[j], \
                        f"{label} row {r}: exact tie d={od[j]}: took {j} and dropped lower {a}"
            else:
                # beyond the oracle's extended list: its distance is at least
                # the list's last, which must still tie the k-th
                assert k_ext == k or rel(last, kth, DIST_FLOOR) <= DIST_RTOL, \
                    f"{label} row {r}: extra idx {j} not among the oracle's {k_ext} nearest"
        if g_dist is not None:
            gd = g_dist[r]
            for pos, j in enumerate(gi):
                if j in od and j in oi:
                    assert rel(gd[pos], od[j], DIST_FLOOR) <= DIST_RTOL, \
                        f"{label} row {r}: idx {j} gpu d={gd[pos]} oracle d={od[j]}"
                else:
                    # a substituted row: its distance must tie the oracle's k-th
                    assert rel(gd[pos], kth, DIST_FLOOR) <= DIST_RTOL, \
                        f"{label} row {r}: extra idx {j} d={gd[pos]} vs k-th {kth}"
            assert np.all(np.diff(gd) >= -1e-12), f"{label} row {r}: not sorted {gd}"
        # order: the GPU list against the oracle's, up to near-ties; rows at
        # exactly the same oracle distance in ascending index order
        for pos, j in enumerate(gi):
            if j in od and oi[pos] != j:
                assert rel(od[j], o_dist[i, pos], DIST_FLOOR) <= DIST_RTOL, \
                    f"{label} row {r} pos {pos}: gpu {j} oracle {oi[pos]}"
        for pos in range(k - 1):
            j1, j2 = gi[pos], gi[pos + 1]
            if j1 in od and j2 in od and od[j1] == od[j2]:
                assert j1 < j2, f"{label} row {r} pos {pos}: exact tie d={od[j1]} as {j1}, {j2}"
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


def admission_boundary(C, budget_r):
    """Instances whose exact Eq. 2 cost C lies within ADMIT_RTOL (relative,
    floor VAL_FLOOR) of the budget: rounding decides their admission, so the
    fp32 path may admit them the other way."""
    C = np.asarray(C, np.float64)
    b = float(budget_r)
    if not np.isfinite(b):
        return np.zeros(C.shape, bool)
    return np.abs(C - b) <= ADMIT_RTOL * np.maximum(np.maximum(np.abs(C), abs(b)), VAL_FLOOR)


def _judge_pick(ig, chosen_r, S, cand):
    """(message or None, near): is the GPU's pick ig, with its chosen score,
    what the greedy step does with scores S over the candidate set cand?"""
    if not cand.any():
        if ig != -1:
            return f"no candidate, gpu picked {ig}", False
        if chosen_r is not None and not np.isnan(chosen_r):
            return f"no candidate, chosen {chosen_r}", False
        return None, False
    if not 0 <= ig < S.shape[0]:
        return f"pick {ig} out of range", False
    if not cand[ig]:
        return f"gpu picked {ig}, not a candidate", False
    io = int(np.nanargmax(S))
    near = False
    if ig != io:
        gap = S[io] - S[ig]
        if gap > PICK_RTOL * max(abs(S[io]), SCORE_FLOOR):
            return f"gpu picked {ig} (S={S[ig]}) oracle {io} (S={S[io]})", False
        near = True
    if chosen_r is not None and rel(chosen_r, S[ig], SCORE_FLOOR) > VAL_RTOL:
        return f"chosen score {chosen_r} vs {S[ig]}", near
    return None, near


def check_assign(g_assign, g_chosen, g_qhat, g_lhat, plen, inst, weights, g_final_p=None,
                 g_final_a=None, p0=None, a0=None, label="", order="arrival", g_order=None,
                 budget=None, mask=None, stats=None, g_decided=None):
    """Teacher-forced replay of the greedy loop. Returns the near-tie count
    (pick near-ties plus requests with an instance at the budget boundary).

    ``order`` "lpt" replays in the oracle's LPT order of the GPU's predictions,
    which must equal ``g_order`` when given; ``budget`` [B] and ``mask`` [I]
    restrict the candidate sets as in the GPU call. ``stats`` (a dict), when
    given, receives the counts by kind ("pick", "admission"). ``g_decided``
    [B][I], when given, is the GPU's row of Eq. 1 scores for each request at
    the state it was decided in (NaN outside the candidate set); each row
    must match the oracle's row at the replayed state within 1e-4."""
    qh = np.asarray(g_qhat, np.float64)
    lh = np.asarray(g_lhat, np.float64)
    g_assign = np.asarray(g_assign)
    B = qh.shape[0]
    p = np.asarray(inst.prefill_q if p0 is None else p0, np.float64).copy()
    a = np.asarray(inst.decode_q if a0 is None else a0, np.float64).copy()
    model = np.asarray(inst.model)
    I = model.shape[0]
    seq = _lpt_order(lh) if order == "lpt" else np.arange(B)
    if g_order is not None:
        assert np.array_equal(np.asarray(g_order), seq), \
            f"{label} processing order differs at step {int(np.argmax(np.asarray(g_order) != seq))}"
    budget = None if budget is None else np.asarray(budget, np.float32)
    avail = np.ones(I, bool) if mask is None else np.asarray(mask) != 0
    counts = {"pick": 0, "admission": 0}
    for r in seq:
        S, _, C, cand = _score_row(qh[r], lh[r], plen[r], inst, p, a, weights,
                                   budget_r=None if budget is None else budget[r], mask=mask,
                                   with_candidates=True)
        ig = int(g_assign[r])
        chosen_r = None if g_chosen is None else g_chosen[r]
        amb = admission_boundary(C, budget[r]) & avail if budget is not None else \
            np.zeros(I, bool)
        if not amb.any():
            msg, near = _judge_pick(ig, chosen_r, S, cand)
            assert msg is None, f"{label} request {r}: {msg}"
            S_used = S
        else:
            # the candidate sets that admitting the boundary instances either
            # way gives; some one of them must explain the GPU's pick
            idx = np.flatnonzero(amb)
            assert len(idx) <= ADMIT_MAX_BOUNDARY, \
                f"{label} request {r}: {len(idx)} instances at the budget boundary"
            fixed = cand & ~amb
            found = None
            for bits in range(1 << len(idx)):
                cs = fixed.copy()
                cs[idx[[(bits >> j) & 1 == 1 for j in range(len(idx))]]] = True
                if cs.any():
                    Sx, _, _ = _score_row(qh[r], lh[r], plen[r], inst, p, a, weights,
                                          mask=cs.astype(np.uint8))
                else:
                    Sx = np.full(I, np.nan)
                msg, near = _judge_pick(ig, chosen_r, Sx, cs)
                if msg is None:
                    found = Sx
                    break
            assert found is not None, \
                f"{label} request {r}: no admission of the boundary instances {idx.tolist()} " \
                f"explains the gpu's pick {ig}"
            counts["admission"] += 1
            S_used = found
        if near:
            counts["pick"] += 1
        if g_decided is not None:
            gd = np.asarray(g_decided[r], np.float64)
            fin = np.isfinite(S_used)
            assert np.array_equal(np.isfinite(gd), fin), \
                f"{label} request {r}: decided row candidates differ"
            if fin.any():
                e = rel(gd[fin], S_used[fin], SCORE_FLOOR)
                assert e.max() <= VAL_RTOL, f"{label} request {r}: decided row rel err {e.max()}"
        if ig >= 0:
            p[ig] += plen[r]
            a[ig] += lh[r, model[ig]]
    if g_final_p is not None:
        e = rel(g_final_p, p, VAL_FLOOR)
        assert e.max() <= VAL_RTOL, f"{label} final prefill state rel err {e.max()}"
    if g_final_a is not None:
        e = rel(g_final_a, a, VAL_FLOOR)
        assert e.max() <= VAL_RTOL, f"{label} final decode state rel err {e.max()}"
    if stats is not None:
        stats.update(counts)
    return counts["pick"] + counts["admission"]


def replay_state(g_assign, g_lhat, plen, inst, p0, a0):
    """The state after a batch's picks (the dead-reckoning update of Sec. 4.2,
    p += l_r and a += L[r][m(i)] for each assigned request), in fp64 from
    (p0, a0). Unassigned requests (-1) change nothing."""
    p = np.asarray(p0, np.float64).copy()
    a = np.asarray(a0, np.float64).copy()
    lh = np.asarray(g_lhat, np.float64)
    model = np.asarray(inst.model)
    for r, i in enumerate(np.asarray(g_assign).tolist()):
        if i >= 0:
            p[i] += plen[r]
            a[i] += lh[r, model[i]]
    return p, a


def free_running(queries, bank, k, qual, length, plen, inst, weights, nthreads=1,
                 order="arrival", weighting="uniform", budget=None, mask=None):
    """The oracle alone: its own KNN, predictions and greedy loop."""
    idx, dist = _knn(queries, bank, k, nthreads=nthreads)
    qh, lh = _predict(idx, qual, length, dist=dist, weighting=weighting)
    res = _assign(qh, lh, plen, inst, weights, order=order, budget=budget, mask=mask)
    res.update(idx=idx, dist=dist, q_hat=qh, l_hat=lh)
    return res
