"""The acceptance rules themselves (oracle.parity), on hand-made results.

These run on the CPU: each feeds a made-up "GPU" result to a parity check and
requires it to be accepted or rejected as the rules say. A rule that accepted
a wrong result would let a wrong kernel pass its parity test.
"""
import numpy as np
import pytest

import oracle
import oracle.parity as par
import synth


def _two_instances(cin0, cout0):
    """Instance 0 with the given prices, instance 1 dear and slow."""
    return synth.Instances(np.array([0, 0], np.int32), np.zeros(2, np.float32),
                           np.zeros(2, np.float32), np.array([1e4, 5e3], np.float32),
                           np.array([1e3, 5e2], np.float32),
                           np.array([cin0, 1e-2], np.float32), np.array([cout0, 1e-2], np.float32))


def test_admission_boundary_flip_is_a_counted_near_tie():
    # instance 0's exact cost sits 1e-7 relative above the budget: the oracle
    # rejects it; a GPU whose fp32 cost rounds to the budget admits it and,
    # instance 1 being over budget too, picks instance 0. Accepted, counted.
    inst = _two_instances(np.float32(1e-3), np.float32(1e-3))
    qh = np.array([[0.5]])
    lh = np.array([[300.0]])
    pl = np.array([1000], np.int32)
    C0 = 1000 * np.float64(np.float32(1e-3)) + 300 * np.float64(np.float32(1e-3))
    budget = np.array([np.float32(C0 * (1 - 1e-7))], np.float32)
    assert budget[0] < C0
    o = oracle.assign(qh, lh, pl, inst, (0.4, 0.3, 0.3), budget=budget)
    assert o["assign"].tolist() == [-1]
    st = {}
    n = par.check_assign([0], [0.4 * 0.5], qh, lh, pl, inst, (0.4, 0.3, 0.3), budget=budget,
                         stats=st, g_final_p=[1000.0, 0.0], g_final_a=[300.0, 0.0])
    assert n == 1 and st == {"pick": 0, "admission": 1}
    # the oracle's own decision (-1) is accepted as well
    assert par.check_assign([-1], [np.nan], qh, lh, pl, inst, (0.4, 0.3, 0.3), budget=budget) == 1


def test_admission_far_from_the_boundary_must_match():
    inst = _two_instances(np.float32(1e-3), np.float32(1e-3))
    qh = np.array([[0.5]])
    lh = np.array([[300.0]])
    pl = np.array([1000], np.int32)
    C0 = 1000 * np.float64(np.float32(1e-3)) + 300 * np.float64(np.float32(1e-3))
    budget = np.array([np.float32(C0 * (1 - 1e-3))], np.float32)   # 1e-3 below: no near-tie
    with pytest.raises(AssertionError):
        par.check_assign([0], [0.2], qh, lh, pl, inst, (0.4, 0.3, 0.3), budget=budget)
    assert par.check_assign([-1], [np.nan], qh, lh, pl, inst, (0.4, 0.3, 0.3),
                            budget=budget) == 0


def test_pick_outside_candidates_or_not_best_is_rejected():
    rng = np.random.default_rng(3)
    cfg = synth.tiny_config(B=6, M=2, inst_per_model=(3, 2))
    inst = synth.make_instances(cfg)
    qh = rng.uniform(0, 1, (6, 2))
    lh = rng.uniform(1, 800, (6, 2))
    pl = rng.integers(1, 3000, 6).astype(np.int32)
    w = (0.4, 0.3, 0.3)
    o = oracle.assign(qh, lh, pl, inst, w)
    assert par.check_assign(o["assign"], o["chosen"], qh, lh, pl, inst, w) == 0
    bad = o["assign"].copy()
    S = oracle.score(qh[:1], lh[:1], pl[:1], inst, w)[0]
    bad[0] = int(np.argmin(S))
    with pytest.raises(AssertionError):
        par.check_assign(bad, None, qh, lh, pl, inst, w)
    mask = np.ones(inst.I, np.uint8)
    mask[o["assign"][0]] = 0
    with pytest.raises(AssertionError):   # the pick is masked out
        par.check_assign(o["assign"], None, qh, lh, pl, inst, w, mask=mask)


def test_decided_rows_are_checked():
    rng = np.random.default_rng(4)
    cfg = synth.tiny_config(B=5, M=2, inst_per_model=(3, 2))
    inst = synth.make_instances(cfg)
    qh = rng.uniform(0, 1, (5, 2))
    lh = rng.uniform(1, 800, (5, 2))
    pl = rng.integers(1, 3000, 5).astype(np.int32)
    w = (0.4, 0.3, 0.3)
    o = oracle.assign(qh, lh, pl, inst, w, trace=True)
    rows = np.stack([oracle.score_row(qh[r], lh[r], pl[r], inst, o["trace_p"][r],
                                      o["trace_a"][r], w)[0] for r in range(5)])
    assert par.check_assign(o["assign"], o["chosen"], qh, lh, pl, inst, w, g_decided=rows) == 0
    wrong = rows.copy()
    wrong[3, 1] += 1e-3
    with pytest.raises(AssertionError):
        par.check_assign(o["assign"], o["chosen"], qh, lh, pl, inst, w, g_decided=wrong)
    # the batch-start scores are not the scores each step saw
    S0 = oracle.score(qh, lh, pl, inst, w)
    with pytest.raises(AssertionError):
        par.check_assign(o["assign"], o["chosen"], qh, lh, pl, inst, w, g_decided=S0)


def test_neighbour_exact_tie_takes_the_lower_index():
    # oracle (k = 3, extended to 5): rows 7 and 2 at exactly the same distance
    # straddle the k-th position; the lower index (2) belongs in the list
    o_idx = np.array([[5, 1, 2, 7, 9]])
    o_dist = np.array([[0.1, 0.2, 0.3, 0.3, 0.9]])
    ok = np.array([[5, 1, 2]])
    assert par.check_neighbours(ok, np.array([[0.1, 0.2, 0.3]]), o_idx, o_dist) == 0
    with pytest.raises(AssertionError):        # the higher index in place of the lower
        par.check_neighbours(np.array([[5, 1, 7]]), np.array([[0.1, 0.2, 0.3]]), o_idx, o_dist)
    # inside the list, equal distances go in ascending index order
    o_idx = np.array([[5, 2, 7, 9]])
    o_dist = np.array([[0.1, 0.3, 0.3, 0.9]])
    assert par.check_neighbours(np.array([[5, 2, 7]]), None, o_idx, o_dist) == 0
    with pytest.raises(AssertionError):
        par.check_neighbours(np.array([[5, 7, 2]]), None, o_idx, o_dist)


def test_neighbour_near_tie_substitution_is_counted():
    o_idx = np.array([[5, 1, 2, 7]])
    o_dist = np.array([[0.1, 0.2, 0.3, 0.3 + 1e-7]])
    assert par.check_neighbours(np.array([[5, 1, 7]]), np.array([[0.1, 0.2, 0.3]]), o_idx,
                                o_dist) == 1
    # a row far beyond the k-th is not a near-tie
    o_dist = np.array([[0.1, 0.2, 0.3, 0.5]])
    with pytest.raises(AssertionError):
        par.check_neighbours(np.array([[5, 1, 7]]), None, o_idx, o_dist)
    # a row not even in the extended list, whose last entry is far: rejected
    with pytest.raises(AssertionError):
        par.check_neighbours(np.array([[5, 1, 42]]), None, o_idx, o_dist)
