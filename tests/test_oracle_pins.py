"""Pins for the CPU oracle: each test ties it to something other than itself.

Kinds of pin used (RouteBalance, arXiv 2606.17949):
  * hand-worked examples with their arithmetic written out (tests/golden/);
  * an independent brute force (numpy full distance matrix + lexsort) on tiny banks;
  * closed forms (constant labels, k = N, k = 1, the inter-batch drain);
  * invariants of Eq. 1 and of the greedy loop of Alg. 1 (simplex corners,
    scale invariance, score range, conservation of the dead-reckoned state,
    w_lat = 0 reducing the greedy to a row-wise argmax).
The paper prints no worked example of its own, so no pin is a printed paper value.
"""
import json
import os

import numpy as np
import pytest
import torch

import oracle
import synth

GOLD = os.path.join(os.path.dirname(__file__), "golden")


def _gold(name):
    with open(os.path.join(GOLD, name)) as f:
        return json.load(f)


def _inst_from(g):
    return synth.Instances(np.array(g["model"], np.int32), np.array(g["prefill_q"], np.float32),
                           np.array(g["decode_q"], np.float32),
                           np.array(g["prefill_rate"], np.float32),
                           np.array(g["decode_rate"], np.float32),
                           np.array(g["price_in"], np.float32), np.array(g["price_out"], np.float32))


# ----------------------------------------------------------------------------- KNN


def test_knn_hand_example_with_ties():
    g = _gold("knn_ties_d2.json")
    q = np.array(g["query"], np.float32)
    x = np.array(g["bank"], np.float32)
    idx, dist = oracle.knn(q, x, g["k"])
    assert idx.tolist() == g["expect_idx"]
    np.testing.assert_allclose(dist, g["expect_dist"], rtol=0, atol=1e-6)
    idx, dist = oracle.knn(q, x, x.shape[0])
    assert idx.tolist() == g["full_order_idx"]
    np.testing.assert_allclose(dist, g["full_order_dist"], rtol=0, atol=1e-6)


def _brute(q64, x64, k):
    """Independent brute force: full fp64 distance matrix, lexsort by (dist, idx)."""
    out_i, out_d = [], []
    for b in range(q64.shape[0]):
        dd = ((x64 - q64[b][None, :]) ** 2).sum(axis=1)
        order = np.lexsort((np.arange(x64.shape[0]), dd))[:k]
        out_i.append(order)
        out_d.append(dd[order])
    return np.array(out_i, np.int32), np.array(out_d)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("N,d,k", [(10, 3, 10), (257, 8, 1), (1000, 16, 10), (4096, 64, 17),
                                   (333, 40, 64)])
def test_knn_matches_bruteforce(dtype, N, d, k):
    rng = np.random.default_rng(N * 7 + d)
    B = 5
    q = torch.from_numpy(rng.standard_normal((B, d)).astype(np.float32))
    x = torch.from_numpy(rng.standard_normal((N, d)).astype(np.float32))
    if dtype == "bf16":
        q, x = q.bfloat16(), x.bfloat16()
    # plant exact duplicates and exact distance ties
    x[N // 2] = x[N // 3]
    x[N - 1] = q[0]
    idx, dist = oracle.knn(q, x, k)
    ei, ed = _brute(q.double().numpy(), x.double().numpy(), k)
    assert np.array_equal(idx, ei)
    np.testing.assert_allclose(dist, ed, rtol=1e-12, atol=1e-12)


def test_knn_special_cases():
    rng = np.random.default_rng(3)
    x = rng.standard_normal((50, 6)).astype(np.float32)
    q = x[[7, 20]].copy()
    # k = 1 returns the row itself at distance 0
    idx, dist = oracle.knn(q, x, 1)
    assert idx[:, 0].tolist() == [7, 20] and np.all(dist == 0)
    # a duplicated row: both copies at distance 0, lower index first
    x2 = np.concatenate([x, x[[7]]])
    idx, dist = oracle.knn(q[:1], x2, 2)
    assert idx[0].tolist() == [7, 50] and np.all(dist[0] == 0)
    # k = N gives every row, ascending
    idx, dist = oracle.knn(q, x, 50)
    assert sorted(idx[0].tolist()) == list(range(50))
    assert np.all(np.diff(dist, axis=1) >= 0)
    # all rows equal: the order is plain index order
    x3 = np.ones((9, 4), np.float32)
    idx, _ = oracle.knn(np.zeros((1, 4), np.float32), x3, 9)
    assert idx[0].tolist() == list(range(9))


def test_knn_rejects_bad_args():
    x = np.zeros((4, 2), np.float32)
    with pytest.raises(ValueError):
        oracle.knn(x[:1], x, 5)            # k > N
    with pytest.raises(ValueError):
        oracle.knn(x[:1], x, 0)


# ----------------------------------------------------------------------------- predict


def test_predict_hand_example():
    g = _gold("knn_ties_d2.json")
    idx, _ = oracle.knn(np.array(g["query"], np.float32), np.array(g["bank"], np.float32), g["k"])
    qh, lh = oracle.predict(idx, np.array(g["qual"], np.float32), np.array(g["len"], np.float32))
    np.testing.assert_allclose(qh, g["expect_q_hat"], rtol=1e-7)
    np.testing.assert_allclose(lh, g["expect_l_hat"], rtol=1e-12)


def test_predict_closed_forms():
    rng = np.random.default_rng(5)
    N, M, d = 40, 3, 5
    x = rng.standard_normal((N, d)).astype(np.float32)
    q = rng.standard_normal((4, d)).astype(np.float32)
    qual = rng.uniform(0, 1, (N, M)).astype(np.float32)
    ln = rng.integers(1, 500, (N, M)).astype(np.float32)
    # constant labels give that constant
    idx, _ = oracle.knn(q, x, 7)
    qh, lh = oracle.predict(idx, np.full((N, M), 0.25, np.float32), np.full((N, M), 42, np.float32))
    assert np.all(qh == 0.25) and np.all(lh == 42)
    # k = N gives the global mean per model
    idx, _ = oracle.knn(q, x, N)
    qh, lh = oracle.predict(idx, qual, ln)
    np.testing.assert_allclose(qh, np.broadcast_to(qual.astype(np.float64).mean(0), qh.shape),
                               rtol=1e-12)
    np.testing.assert_allclose(lh, np.broadcast_to(ln.astype(np.float64).mean(0), lh.shape),
                               rtol=1e-12)
    # k = 1 gives the nearest row's labels exactly, per model column
    idx, _ = oracle.knn(q, x, 1)
    qh, lh = oracle.predict(idx, qual, ln)
    assert np.array_equal(qh, qual[idx[:, 0]].astype(np.float64))
    assert np.array_equal(lh, ln[idx[:, 0]].astype(np.float64))


# ----------------------------------------------------------------------------- score


def test_score_hand_example():
    g = _gold("score_2x3.json")
    inst = _inst_from(g)
    S0 = oracle.score(g["q_hat"], g["l_hat"], g["prompt_len"], inst, g["weights"])
    np.testing.assert_allclose(S0, g["expect_S0"], rtol=1e-12)
    for r in range(2):
        S, T, C = oracle.score_row(g["q_hat"][r], g["l_hat"][r], g["prompt_len"][r], inst,
                                   inst.prefill_q, inst.decode_q, g["weights"])
        np.testing.assert_allclose(T, g["expect_T0"][r], rtol=1e-12)
        np.testing.assert_allclose(C, g["expect_C"][r], rtol=1e-6)   # fp32 prices
        np.testing.assert_allclose(S, g["expect_S0"][r], rtol=1e-12)


def test_assign_hand_example_and_corners():
    g = _gold("score_2x3.json")
    inst = _inst_from(g)
    res = oracle.assign(g["q_hat"], g["l_hat"], g["prompt_len"], inst, g["weights"], trace=True)
    assert res["assign"].tolist() == g["expect_assign"]
    np.testing.assert_allclose(res["chosen"], g["expect_chosen"], rtol=1e-12)
    np.testing.assert_array_equal(res["p"], g["expect_final_p"])
    np.testing.assert_array_equal(res["a"], g["expect_final_a"])
    # step 1 is scored after step 0's update
    S, _, _ = oracle.score_row(g["q_hat"][1], g["l_hat"][1], g["prompt_len"][1], inst,
                               res["trace_p"][1], res["trace_a"][1], g["weights"])
    np.testing.assert_allclose(S, g["expect_step1_S"], rtol=1e-12)
    for c in g["corners"]:
        r = oracle.assign(g["q_hat"], g["l_hat"], g["prompt_len"], inst, c["weights"])
        assert r["assign"].tolist() == c["assign"], c
        np.testing.assert_array_equal(r["p"], c["final_p"])
        np.testing.assert_array_equal(r["a"], c["final_a"])


def test_cost_uses_input_price_for_prompt_and_output_price_for_output():
    # i0 charges only input tokens, i1 only output tokens. A short prompt with a
    # long predicted output is cheap on i0; a long prompt with a short output is
    # cheap on i1. Swapping the two prices in Eq. 2 flips both picks.
    inst = synth.Instances(np.array([0, 0], np.int32), np.zeros(2, np.float32),
                           np.zeros(2, np.float32), np.full(2, 1000, np.float32),
                           np.full(2, 100, np.float32), np.array([1e-3, 0], np.float32),
                           np.array([0, 1e-3], np.float32))
    qh = [[0.5], [0.5]]
    lh = [[1000.0], [10.0]]
    res = oracle.assign(qh, lh, [10, 1000], inst, (0, 0, 1))
    assert res["assign"].tolist() == [0, 1]


def test_latency_uses_prefill_rate_for_prompt_and_decode_rate_for_output():
    # i0 prefills fast but decodes slowly; i1 the reverse. Both idle. A long
    # prompt with a 1-token output is faster on i0; a short prompt with a long
    # output is faster on i1.
    inst = synth.Instances(np.array([0, 0], np.int32), np.zeros(2, np.float32),
                           np.zeros(2, np.float32), np.array([100000, 1000], np.float32),
                           np.array([10, 1000], np.float32), np.zeros(2, np.float32),
                           np.zeros(2, np.float32))
    r = oracle.assign([[0.5]], [[1.0]], [50000], inst, (0, 1, 0))
    assert r["assign"].tolist() == [0]
    r = oracle.assign([[0.5]], [[500.0]], [10], inst, (0, 1, 0))
    assert r["assign"].tolist() == [1]
    # queued work counts: the same request avoids an instance with a long queue
    inst2 = inst.copy()
    inst2.prefill_rate[:] = 1000
    inst2.decode_rate[:] = 1000
    inst2.prefill_q[:] = [5000, 0]
    r = oracle.assign([[0.5]], [[10.0]], [10], inst2, (0, 1, 0))
    assert r["assign"].tolist() == [1]
    inst2.prefill_q[:] = [0, 0]
    inst2.decode_q[:] = [0, 5000]
    r = oracle.assign([[0.5]], [[10.0]], [10], inst2, (0, 1, 0))
    assert r["assign"].tolist() == [0]


def _random_case(seed, B=24, M=3, I=11):
    rng = np.random.default_rng(seed)
    cfg = synth.tiny_config(B=B, M=M, inst_per_model=tuple([I // M + (1 if m < I % M else 0)
                                                            for m in range(M)]), seed=seed)
    inst = synth.make_instances(cfg)
    qh = rng.uniform(0, 1, (B, M))
    lh = rng.uniform(1, 800, (B, M))
    pl = rng.integers(1, 3000, B).astype(np.int32)
    return qh, lh, pl, inst


@pytest.mark.parametrize("seed", range(5))
def test_simplex_corners(seed):
    qh, lh, pl, inst = _random_case(seed)
    B, I = qh.shape[0], inst.I
    # (1,0,0): highest predicted quality of the instance's model, lowest index on ties
    r = oracle.assign(qh, lh, pl, inst, (1, 0, 0))
    for b in range(B):
        vals = qh[b][inst.model]
        assert r["assign"][b] == int(np.flatnonzero(vals == vals.max())[0])
    # (0,0,1): cheapest; (0,1,0): fastest at the state seen by that step
    for w, key in (((0, 0, 1), 2), ((0, 1, 0), 1)):
        r = oracle.assign(qh, lh, pl, inst, w, trace=True)
        for b in range(B):
            S, T, C = oracle.score_row(qh[b], lh[b], pl[b], inst, r["trace_p"][b], r["trace_a"][b],
                                       w)
            v = C if key == 2 else T
            assert r["assign"][b] == int(np.flatnonzero(v == v.min())[0])


@pytest.mark.parametrize("seed", range(5))
def test_score_range_and_scale_invariance(seed):
    qh, lh, pl, inst = _random_case(seed)
    w = (0.2, 0.5, 0.3)
    S0 = oracle.score(qh, lh, pl, inst, w)
    assert np.all(S0 >= -1e-12) and np.all(S0 <= 1 + 1e-12)
    scaled = inst.copy()
    scaled.price_in = (inst.price_in.astype(np.float64) * 3.0)
    scaled.price_out = (inst.price_out.astype(np.float64) * 3.0)
    np.testing.assert_allclose(oracle.score(qh, lh, pl, scaled, w), S0, rtol=1e-12, atol=1e-14)
    scaled = inst.copy()
    scaled.prefill_rate = inst.prefill_rate.astype(np.float64) * 0.25
    scaled.decode_rate = inst.decode_rate.astype(np.float64) * 0.25
    np.testing.assert_allclose(oracle.score(qh, lh, pl, scaled, w), S0, rtol=1e-12, atol=1e-14)


@pytest.mark.parametrize("seed", range(5))
def test_greedy_invariants(seed):
    qh, lh, pl, inst = _random_case(seed)
    B, I = qh.shape[0], inst.I
    w = (0.3, 0.4, 0.3)
    r = oracle.assign(qh, lh, pl, inst, w, trace=True)
    tp, ta = r["trace_p"], r["trace_a"]
    # conservation, step by step: only the chosen instance grows, by the prompt
    # and by the predicted output on its model
    for b in range(B):
        i = r["assign"][b]
        dp = tp[b + 1] - tp[b]
        da = ta[b + 1] - ta[b]
        expect_p = np.zeros(I)
        expect_p[i] = pl[b]
        expect_a = np.zeros(I)
        expect_a[i] = lh[b][inst.model[i]]
        np.testing.assert_allclose(dp, expect_p, rtol=0, atol=1e-9)
        np.testing.assert_allclose(da, expect_a, rtol=0, atol=1e-9)
        S, _, _ = oracle.score_row(qh[b], lh[b], pl[b], inst, tp[b], ta[b], w)
        assert i == int(np.argmax(S)) and r["chosen"][b] == S[i]
    np.testing.assert_array_equal(tp[B], r["p"])
    # with w_lat = 0 the state never matters: greedy == row-wise argmax of S0
    w0 = (0.6, 0.0, 0.4)
    r0 = oracle.assign(qh, lh, pl, inst, w0)
    S0 = oracle.score(qh, lh, pl, inst, w0)
    assert r0["assign"].tolist() == np.argmax(S0, axis=1).tolist()
    # B = 1 is the argmax of S0's first row
    r1 = oracle.assign(qh[:1], lh[:1], pl[:1], inst, w)
    S1 = oracle.score(qh[:1], lh[:1], pl[:1], inst, w)
    assert r1["assign"][0] == int(np.argmax(S1[0]))


def test_zero_cost_maximum():
    # all prices zero: the cost term contributes w_cost to every instance
    qh, lh, pl, inst = _random_case(11, B=3)
    inst.price_in[:] = 0
    inst.price_out[:] = 0
    w = (0.0, 0.0, 1.0)
    S0 = oracle.score(qh, lh, pl, inst, w)
    assert np.all(S0 == 1.0)
    r = oracle.assign(qh, lh, pl, inst, w)
    assert r["assign"].tolist() == [0, 0, 0]


# ----------------------------------------------------------------------------- carry


def test_advance_closed_form():
    p = np.array([100.0, 0.0, 5000.0])
    a = np.array([1000.0, 10.0, 0.0])
    P = np.array([1000.0, 500.0, 2000.0])
    D = np.array([50.0, 100.0, 10.0])
    p1, a1 = oracle.advance(p, a, P, D, 0.0)
    assert np.array_equal(p1, p) and np.array_equal(a1, a)
    p1, a1 = oracle.advance(p, a, P, D, 0.5)
    # 100 - 500 clamps to 0; 5000 - 1000 = 4000; 1000 - 25 = 975; 10 - 50 clamps; 0 stays
    assert p1.tolist() == [0.0, 0.0, 4000.0]
    assert a1.tolist() == [975.0, 0.0, 0.0]
    with pytest.raises(ValueError):
        oracle.advance(p, a, P, D, -1.0)


# ----------------------------------------------------------------------------- LPT order


def test_lpt_hand_example():
    g = _gold("lpt_2x3.json")
    inst = _inst_from(g)
    for mode in ("lpt", "arrival"):
        e = g[mode]
        r = oracle.assign(g["q_hat"], g["l_hat"], g["prompt_len"], inst, g["weights"], order=mode)
        assert r["order"].tolist() == e["order"], mode
        assert r["assign"].tolist() == e["assign"], mode
        np.testing.assert_allclose(r["chosen"], e["chosen"], rtol=1e-12)
        np.testing.assert_array_equal(r["p"], e["final_p"])
        np.testing.assert_array_equal(r["a"], e["final_a"])
    assert oracle.lpt_order(g["l_hat"]).tolist() == g["lpt"]["order"]


@pytest.mark.parametrize("seed", range(4))
def test_lpt_order_matches_library_sort(seed):
    # independent: numpy's stable lexsort on (descending key, index)
    rng = np.random.default_rng(100 + seed)
    B, M = 200, 1 + seed
    lh = rng.integers(1, 40, (B, M)).astype(np.float64) / 4   # many exactly equal keys
    key = lh.max(axis=1)
    expect = np.lexsort((np.arange(B), -key))
    assert oracle.lpt_order(lh).tolist() == expect.tolist()
    # a single model: the key is that column
    assert oracle.lpt_order(lh[:, :1]).tolist() == np.lexsort((np.arange(B), -lh[:, 0])).tolist()


@pytest.mark.parametrize("seed", range(4))
def test_lpt_is_arrival_order_over_the_sorted_batch(seed):
    # LPT decides exactly what the arrival-order loop decides on the batch
    # permuted into LPT order (Alg. 1 only changes the iteration order)
    qh, lh, pl, inst = _random_case(200 + seed, B=30)
    w = (0.3, 0.4, 0.3)
    r = oracle.assign(qh, lh, pl, inst, w, order="lpt")
    perm = np.lexsort((np.arange(qh.shape[0]), -lh.max(axis=1)))
    assert r["order"].tolist() == perm.tolist()
    ra = oracle.assign(qh[perm], lh[perm], pl[perm], inst, w)
    assert np.array_equal(r["assign"][perm], ra["assign"])
    np.testing.assert_array_equal(r["chosen"][perm], ra["chosen"])
    np.testing.assert_array_equal(r["p"], ra["p"])
    np.testing.assert_array_equal(r["a"], ra["a"])
    # equal keys everywhere: LPT is arrival order
    lh_eq = np.full_like(lh, 123.0)
    r1 = oracle.assign(qh, lh_eq, pl, inst, w, order="lpt")
    r2 = oracle.assign(qh, lh_eq, pl, inst, w)
    assert r1["order"].tolist() == list(range(qh.shape[0]))
    assert np.array_equal(r1["assign"], r2["assign"])


# ----------------------------------------------------------------------------- weighted average


def test_inv_dist_weights_closed_forms():
    qual = np.array([[0.0, 1.0], [1.0, 0.0], [0.25, 0.5]], np.float32)
    ln = np.array([[10.0, 1.0], [40.0, 2.0], [7.0, 3.0]], np.float32)
    # squared distances 1 and 4: Euclidean 1 and 2, weights 1/(1+e) and
    # 1/(2+e) with e = 1e-6, normalised: (2+e)/(3+2e) and (1+e)/(3+2e)
    e = 1e-6
    w0, w1 = (2 + e) / (3 + 2 * e), (1 + e) / (3 + 2 * e)
    qh, lh = oracle.predict([[0, 1]], qual, ln, dist=[[1.0, 4.0]], weighting="inv_dist")
    np.testing.assert_allclose(qh[0], [w1, w0], rtol=1e-14)
    np.testing.assert_allclose(lh[0], [10 * w0 + 40 * w1, w0 + 2 * w1], rtol=1e-14)
    # equal distances: the plain mean, whatever the common distance
    for dd in (0.0, 0.3, 2.0):
        qw, lw = oracle.predict([[0, 1, 2]], qual, ln, dist=[[dd] * 3], weighting="inv_dist")
        qu, lu = oracle.predict([[0, 1, 2]], qual, ln)
        np.testing.assert_allclose(qw, qu, rtol=1e-14)
        np.testing.assert_allclose(lw, lu, rtol=1e-14)
    # k = 1: that row's labels (w*x/w, exact up to one rounding)
    qh, lh = oracle.predict([[2]], qual, ln, dist=[[0.7]], weighting="inv_dist")
    np.testing.assert_allclose(qh[0], qual[2].astype(np.float64), rtol=1e-15)
    np.testing.assert_allclose(lh[0], ln[2].astype(np.float64), rtol=1e-15)
    # a negative squared distance (cancellation) counts as 0
    qa, _ = oracle.predict([[0, 1]], qual, ln, dist=[[-0.5, 1.0]], weighting="inv_dist")
    qb, _ = oracle.predict([[0, 1]], qual, ln, dist=[[0.0, 1.0]], weighting="inv_dist")
    assert np.array_equal(qa, qb)
    # the neighbour order does not matter
    qa, la = oracle.predict([[0, 1, 2]], qual, ln, dist=[[0.1, 0.5, 0.9]], weighting="inv_dist")
    qb, lb = oracle.predict([[2, 0, 1]], qual, ln, dist=[[0.9, 0.1, 0.5]], weighting="inv_dist")
    np.testing.assert_allclose(qa, qb, rtol=1e-14)
    np.testing.assert_allclose(la, lb, rtol=1e-14)


def test_inv_dist_hand_example_duplicates_dominate():
    # the KNN hand example: rows 0 and 4 sit at distance 0 and take weight
    # 1e6 each against ~1.1 and ~0.7 for the rows at 0.8 and 2, so the
    # prediction is the mean of rows 0 and 4 to within ~1e-6 relative
    g = _gold("knn_ties_d2.json")
    idx, dist = oracle.knn(np.array(g["query"], np.float32), np.array(g["bank"], np.float32),
                           g["k"])
    qual = np.array(g["qual"], np.float32)
    ln = np.array(g["len"], np.float32)
    qh, lh = oracle.predict(idx, qual, ln, dist=dist, weighting="inv_dist")
    np.testing.assert_allclose(qh[0], (qual[0] + qual[4]) / 2, rtol=1e-6)
    np.testing.assert_allclose(lh[0], (ln[0] + ln[4]) / 2, rtol=1e-6)
    assert not np.allclose(qh[0], g["expect_q_hat"][0], rtol=1e-3)   # differs from the plain mean


# ----------------------------------------------------------------------------- candidate sets


def _inf(v):
    return np.float32(np.inf) if v == "inf" else np.float32(v)


def test_budget_and_mask_hand_examples():
    g = _gold("budget_mask_2x3.json")
    inst = _inst_from(g)
    for c in g["cases"]:
        budget = None if c["budget"] is None else np.array([_inf(v) for v in c["budget"]])
        mask = None if c["mask"] is None else np.array(c["mask"], np.uint8)
        r = oracle.assign(g["q_hat"], g["l_hat"], g["prompt_len"], inst, g["weights"],
                          budget=budget, mask=mask)
        assert r["assign"].tolist() == c["assign"], c["name"]
        expect = np.array([np.nan if v == "nan" else v for v in c["chosen"]])
        np.testing.assert_allclose(r["chosen"], expect, rtol=1e-12, equal_nan=True)
        np.testing.assert_array_equal(r["p"], c["final_p"])
        np.testing.assert_array_equal(r["a"], c["final_a"])
    b = g["boundary"]
    binst = synth.Instances(np.array(b["model"], np.int32), np.zeros(2, np.float32),
                            np.zeros(2, np.float32), np.array(b["prefill_rate"], np.float32),
                            np.array(b["decode_rate"], np.float32),
                            np.array(b["price_in"], np.float32),
                            np.array(b["price_out"], np.float32))
    for budget, admitted in b["budgets"]:
        _, _, C, cand = oracle.score_row(b["q_hat"][0], b["l_hat"][0], b["prompt_len"][0], binst,
                                         np.zeros(2), np.zeros(2), (0.4, 0.3, 0.3),
                                         budget_r=budget, with_candidates=True)
        assert np.flatnonzero(cand).tolist() == admitted, budget
        np.testing.assert_array_equal(C, [125.0, 300.0])
        r = oracle.assign(b["q_hat"], b["l_hat"], b["prompt_len"], binst, (0.4, 0.3, 0.3),
                          budget=np.array([budget], np.float32))
        assert r["assign"].tolist() == [admitted[0] if admitted else -1]


def _exact_cost(l, cin, L, cout):
    """Eq. 2 cost of fp32 inputs in exact rational arithmetic."""
    from fractions import Fraction as F
    return F(int(l)) * F(float(cin)) + F(float(L)) * F(float(cout))


def _fp32_cost(l, cin, L, cout):
    """The same cost in fp32 with one fused multiply-add (C library fmaf)."""
    import ctypes
    import ctypes.util
    libm = ctypes.CDLL(ctypes.util.find_library("m"))
    libm.fmaf.restype = ctypes.c_float
    libm.fmaf.argtypes = [ctypes.c_float] * 3
    return np.float32(libm.fmaf(float(np.float32(l)), float(cin),
                                float(np.float32(np.float32(L) * np.float32(cout)))))


def test_budget_admission_is_exact_at_one_ulp():
    # Eq. 2 compares the expected cost with the budget; the oracle decides it
    # on the exact cost. Find fp32 inputs whose exact cost lies strictly
    # between two adjacent fp32 budgets b_lo < C < b_hi while the fp32 fused
    # evaluation rounds to b_lo: b_lo must reject (although fp32 arithmetic
    # would admit), b_hi must admit, and a budget equal to an exactly
    # representable cost admits (the boundary case of the hand example).
    from fractions import Fraction as F
    rng = np.random.default_rng(17)
    found = 0
    for _ in range(2000):
        l = int(rng.integers(50, 5000))
        L = np.float32(rng.integers(1, 2000))
        cin = np.float32(rng.uniform(1e-4, 2e-3))
        cout = np.float32(rng.uniform(1e-4, 2e-3))
        C = _exact_cost(l, cin, L, cout)
        lo = np.float32(float(C))
        if F(float(lo)) > C:
            lo = np.nextafter(lo, np.float32(-np.inf))
        hi = np.nextafter(lo, np.float32(np.inf))
        if not F(float(lo)) < C < F(float(hi)) or _fp32_cost(l, cin, L, cout) > lo:
            continue
        inst = synth.Instances(np.array([0], np.int32), np.zeros(1, np.float32),
                               np.zeros(1, np.float32), np.full(1, 1e4, np.float32),
                               np.full(1, 1e3, np.float32), np.array([cin]), np.array([cout]))
        for budget, admit in ((lo, False), (hi, True)):
            _, _, Cc, cand = oracle.score_row([0.5], [float(L)], l, inst, np.zeros(1),
                                              np.zeros(1), (0.4, 0.3, 0.3), budget_r=budget,
                                              with_candidates=True)
            assert bool(cand[0]) == admit, (l, float(L), float(cin), float(cout), float(budget))
            r = oracle.assign(np.array([[0.5]]), np.array([[float(L)]]), np.array([l], np.int32),
                              inst, (0.4, 0.3, 0.3), budget=np.array([budget], np.float32))
            assert r["assign"].tolist() == [0 if admit else -1]
        found += 1
        if found == 20:
            break
    assert found == 20


@pytest.mark.parametrize("seed", range(4))
def test_mask_is_removing_instances(seed):
    # an unavailable instance is as if it were not in the table: the masked
    # run equals the plain run over the sub-table of available instances
    qh, lh, pl, inst = _random_case(300 + seed, B=30, I=13)
    rng = np.random.default_rng(seed)
    mask = (rng.uniform(size=inst.I) < 0.6).astype(np.uint8)
    mask[rng.integers(inst.I)] = 1
    keep = np.flatnonzero(mask)
    sub = synth.Instances(*(np.asarray(getattr(inst, f))[keep] for f in
                            ("model", "prefill_q", "decode_q", "prefill_rate", "decode_rate",
                             "price_in", "price_out")))
    for order in ("arrival", "lpt"):
        w = (0.3, 0.4, 0.3)
        r = oracle.assign(qh, lh, pl, inst, w, mask=mask, order=order)
        rs = oracle.assign(qh, lh, pl, sub, w, order=order)
        assert r["assign"].tolist() == keep[rs["assign"]].tolist()
        np.testing.assert_array_equal(r["chosen"], rs["chosen"])
        np.testing.assert_array_equal(r["p"][keep], rs["p"])
        np.testing.assert_array_equal(r["a"][keep], rs["a"])
        off = np.flatnonzero(mask == 0)
        np.testing.assert_array_equal(r["p"][off], inst.prefill_q[off])
        np.testing.assert_array_equal(r["a"][off], inst.decode_q[off])
    # nothing available: every request unassigned, state unchanged
    r = oracle.assign(qh, lh, pl, inst, (0.3, 0.4, 0.3), mask=np.zeros(inst.I, np.uint8))
    assert np.all(r["assign"] == -1) and np.all(np.isnan(r["chosen"]))
    np.testing.assert_array_equal(r["p"], inst.prefill_q)


@pytest.mark.parametrize("seed", range(4))
def test_budget_filter_invariants(seed):
    qh, lh, pl, inst = _random_case(400 + seed, B=30, I=13)
    w = (0.3, 0.4, 0.3)
    base = oracle.assign(qh, lh, pl, inst, w, trace=True)
    # an infinite budget and an all-ones mask change nothing
    r = oracle.assign(qh, lh, pl, inst, w, budget=np.full(qh.shape[0], np.inf, np.float32),
                      mask=np.ones(inst.I, np.uint8))
    assert np.array_equal(r["assign"], base["assign"])
    np.testing.assert_array_equal(r["chosen"], base["chosen"])
    # per-request budgets between the cheapest and the dearest instance,
    # away from every cost (relative gap 1e-3 or more, so precision does not
    # decide): each pick is an admitted instance and the best among them
    rng = np.random.default_rng(seed)
    C = pl[:, None] * inst.price_in[None, :].astype(np.float64) + \
        lh[:, inst.model] * inst.price_out[None, :].astype(np.float64)
    budget = np.exp(rng.uniform(np.log(C.min(1)), np.log(C.max(1)))).astype(np.float32)
    near = np.abs(C / budget[:, None].astype(np.float64) - 1).min(axis=1) < 1e-3
    budget[near] = np.inf
    r = oracle.assign(qh, lh, pl, inst, w, budget=budget, trace=True)
    for t, b in enumerate(r["order"]):
        admitted = C[b] <= budget[b]
        i = r["assign"][b]
        if not admitted.any():
            assert i == -1
            continue
        assert admitted[i]
        S, _, _ = oracle.score_row(qh[b], lh[b], pl[b], inst, r["trace_p"][t], r["trace_a"][t], w,
                                   budget_r=budget[b])
        assert np.all(np.isnan(S[~admitted]))
        assert i == int(np.nanargmax(S)) and r["chosen"][b] == S[i]
        # a single admitted instance is its own maximum: S = w_qual * Q
        if admitted.sum() == 1:
            assert r["chosen"][b] == w[0] * qh[b][inst.model[i]]
    # conservation over the admitted picks only
    got = r["assign"] >= 0
    for i in range(inst.I):
        sel = got & (r["assign"] == i)
        np.testing.assert_allclose(r["p"][i] - inst.prefill_q[i], pl[sel].sum(), rtol=1e-12)
        np.testing.assert_allclose(r["a"][i] - inst.decode_q[i],
                                   lh[sel, inst.model[i]].sum(), rtol=1e-12, atol=1e-9)


# ----------------------------------------------------------------------------- batch matching


def _brute_matching(S0, cap):
    """All I^B assignments within the capacities; the best total and its argmax."""
    import itertools
    B, I = S0.shape
    best, arg = -np.inf, None
    for a in itertools.product(range(I), repeat=B):
        if np.any(np.bincount(a, minlength=I) > cap):
            continue
        v = S0[np.arange(B), a].sum()
        if v > best:
            best, arg = v, a
    return best, np.array(arg)


def test_batch_matching_hand_example():
    # two requests, two one-slot instances: taking 0.9 forces 0.1 (total 1.0),
    # the matching takes 0.8 + 0.85 = 1.65; without capacity both pick i0
    S0 = np.array([[0.9, 0.8], [0.85, 0.1]])
    assert oracle.batch_matching(S0, 1).tolist() == [1, 0]
    assert oracle.batch_matching(S0, 2).tolist() == [0, 0]
    # a non-candidate (NaN) is never matched while a finite choice remains
    S1 = np.array([[np.nan, 0.2], [0.3, 0.9]])
    assert oracle.batch_matching(S1, 1).tolist() == [1, 0]


@pytest.mark.parametrize("seed", range(6))
def test_batch_matching_matches_brute_force(seed):
    rng = np.random.default_rng(500 + seed)
    B, I = 6, 3
    S0 = rng.uniform(0, 1, (B, I))
    for cap in (2, 3, np.array([1, 2, 3]), np.array([4, 1, 1])):
        best, arg = _brute_matching(S0, np.broadcast_to(cap, (I,)))
        got = oracle.batch_matching(S0, cap)
        assert np.all(np.bincount(got, minlength=I) <= np.broadcast_to(cap, (I,)))
        np.testing.assert_allclose(S0[np.arange(B), got].sum(), best, rtol=1e-12)
        assert got.tolist() == arg.tolist()        # continuous scores: the optimum is unique


def test_batch_matching_without_capacity_is_row_argmax():
    rng = np.random.default_rng(7)
    S0 = rng.uniform(0, 1, (40, 5))
    S0[3, 1] = S0[3, 4] = 2.0                      # a tie: the lower instance
    got = oracle.batch_matching(S0, 40)
    assert got.tolist() == np.argmax(S0, axis=1).tolist()
    with pytest.raises(ValueError):
        oracle.batch_matching(S0, 7)               # 5 x 7 slots < 40 requests
