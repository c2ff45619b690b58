"""GPU parity of the routing options against the CPU oracle: the LPT
processing order, the inverse-distance KNN average, per-request cost budgets
and the instance availability mask (rb_assign_ex, rb_predict with
RB_KNN_INV_DIST, rb_route_batch_ex).

Acceptance rules are those of oracle.parity: the LPT order bit-identical to
the oracle's order of the GPU's own predictions; candidate sets identical
(both sides admit in fp32); picks teacher-forced with near-ties within 1e-5;
weighted predictions teacher-forced from the GPU's neighbours and distances
within 1e-4.
"""
import json
import os

import numpy as np
import pytest
import torch

import oracle
import oracle.parity as par
import synth

pytestmark = pytest.mark.gpu

DEV = "cuda"
GOLD = os.path.join(os.path.dirname(__file__), "golden")


def rb():
    import paper_2606_17949_amd as m
    return m


def say(msg):
    print(msg, flush=True)


def dev(a, dtype=None):
    t = torch.from_numpy(np.ascontiguousarray(a))
    return t.to(DEV) if dtype is None else t.to(device=DEV, dtype=dtype)


def random_case(B, M, I, seed, tie_keys=False):
    rng = np.random.default_rng(seed)
    per = [I // M + (1 if m < I % M else 0) for m in range(M)]
    cfg = synth.tiny_config(B=B, M=M, inst_per_model=tuple(per), seed=seed)
    inst = synth.make_instances(cfg)
    qh = rng.uniform(0, 1, (B, M)).astype(np.float32)
    if tie_keys:
        # few distinct values: many requests share their LPT key exactly
        lh = (rng.integers(4, 40, (B, M)) * 8).astype(np.float32)
    else:
        lh = rng.uniform(1, 800, (B, M)).astype(np.float32)
    pl = rng.integers(1, 3000, B).astype(np.int32)
    return qh, lh, pl, inst


def costs(lh, pl, inst):
    return pl[:, None] * inst.price_in[None, :].astype(np.float64) + \
        lh[:, inst.model].astype(np.float64) * inst.price_out[None, :].astype(np.float64)


def run_assign_ex(qh, lh, pl, inst, w, order=0, budget=None, mask=None):
    m = rb()
    B = qh.shape[0]
    gi = m.DeviceInstances.from_host(inst, DEV)
    order_out = torch.full((B,), -7, dtype=torch.int32, device=DEV)
    gb = None if budget is None else dev(budget.astype(np.float32))
    gm = None if mask is None else dev(mask.astype(np.uint8))
    opts = m.options(order=order, budget=gb, instance_mask=gm, order_out=order_out)
    asg, ch = m.rb_assign_ex(dev(qh), dev(lh), dev(pl), gi, w, opts)
    torch.cuda.synchronize()
    return dict(assign=asg.cpu().numpy(), chosen=ch.cpu().numpy(),
                order=order_out.cpu().numpy(), p=gi.prefill_q.cpu().numpy(),
                a=gi.decode_q.cpu().numpy())


def check(res, qh, lh, pl, inst, w, order, budget=None, mask=None, label=""):
    st = {}
    near = par.check_assign(res["assign"], res["chosen"], qh, lh, pl, inst, w,
                            g_final_p=res["p"], g_final_a=res["a"], label=label,
                            order="lpt" if order == rb().RB_ORDER_LPT else "arrival",
                            g_order=res["order"], budget=budget, mask=mask, stats=st)
    if budget is not None:
        say(f"  {label}: near-ties {st}")
    free = oracle.assign(qh.astype(np.float64), lh.astype(np.float64), pl, inst, w,
                         order="lpt" if order == rb().RB_ORDER_LPT else "arrival",
                         budget=budget, mask=mask)
    if near == 0:
        assert np.array_equal(free["assign"], res["assign"]), label
    return near


# ----------------------------------------------------------------------------- LPT order

LPT_CASES = [
    # B, M, I
    (16, 4, 13),
    (1, 1, 1),
    (255, 4, 13),
    (256, 8, 64),      # exactly one ranking workgroup
    (257, 16, 512),    # one request past it
    (1000, 4, 17),
    (3000, 2, 5),      # twelve ranking workgroups, many equal keys
]


@pytest.mark.parametrize("B,M,I", LPT_CASES)
@pytest.mark.parametrize("tie_keys", [False, True])
def test_lpt_parity(B, M, I, tie_keys):
    say(f"lpt B={B} M={M} I={I} ties={tie_keys}")
    qh, lh, pl, inst = random_case(B, M, I, seed=B + 3 * I, tie_keys=tie_keys)
    w = (0.3, 0.4, 0.3)
    res = run_assign_ex(qh, lh, pl, inst, w, order=rb().RB_ORDER_LPT)
    assert sorted(res["order"].tolist()) == list(range(B))
    near = check(res, qh, lh, pl, inst, w, rb().RB_ORDER_LPT, label=f"lpt B={B}")
    say(f"  near-ties {near}")


def test_lpt_hand_example_on_gpu():
    say("lpt hand example")
    g = json.load(open(os.path.join(GOLD, "lpt_2x3.json")))
    inst = synth.Instances(*[np.array(g[f], np.int32 if f == "model" else np.float32)
                             for f in synth.Instances.FIELDS])
    qh = np.array(g["q_hat"], np.float32)
    lh = np.array(g["l_hat"], np.float32)
    pl = np.array(g["prompt_len"], np.int32)
    for mode, code in (("lpt", rb().RB_ORDER_LPT), ("arrival", rb().RB_ORDER_ARRIVAL)):
        e = g[mode]
        res = run_assign_ex(qh, lh, pl, inst, g["weights"], order=code)
        assert res["order"].tolist() == e["order"], mode
        assert res["assign"].tolist() == e["assign"], mode
        np.testing.assert_allclose(res["chosen"], e["chosen"], rtol=1e-6)
        np.testing.assert_allclose(res["p"], e["final_p"], rtol=1e-6)
        np.testing.assert_allclose(res["a"], e["final_a"], rtol=1e-6)


# ----------------------------------------------------------------------------- budgets and mask


@pytest.mark.parametrize("B,M,I", [(16, 4, 13), (64, 8, 64), (33, 16, 512), (300, 4, 65),
                                   (40, 4, 16), (7, 3, 1024)])
@pytest.mark.parametrize("order", [0, 1])
def test_budget_mask_parity(B, M, I, order):
    say(f"budget/mask B={B} M={M} I={I} order={order}")
    qh, lh, pl, inst = random_case(B, M, I, seed=11 * B + I)
    rng = np.random.default_rng(B * I)
    C = costs(lh, pl, inst)
    # budgets spread from below the cheapest to above the dearest instance, a
    # quarter without a budget; instances down at random and one model's tier
    # lost entirely
    budget = np.exp(rng.uniform(np.log(C.min(1) * 0.8), np.log(C.max(1) * 1.1))).astype(np.float32)
    budget[rng.uniform(size=B) < 0.25] = np.inf
    mask = (rng.uniform(size=inst.I) >= 0.2).astype(np.uint8)
    mask[inst.model == M - 1] = 0 if M > 1 else mask[inst.model == M - 1]
    for w in [(0.3, 0.4, 0.3), (1, 0, 0), (0, 1, 0), (0, 0, 1)]:
        for bud, msk in ((budget, None), (None, mask), (budget, mask)):
            res = run_assign_ex(qh, lh, pl, inst, w, order=order, budget=bud, mask=msk)
            check(res, qh, lh, pl, inst, w, order, budget=bud, mask=msk,
                  label=f"w={w} budget={bud is not None} mask={msk is not None}")
            if msk is not None:
                assert not np.isin(res["assign"], np.flatnonzero(msk == 0)).any()


def test_budget_boundary_is_inclusive_on_gpu():
    # dyadic prices and integer lengths make every cost exact in fp32, so a
    # budget equal to a cost must admit that instance on both sides
    say("budget boundary")
    B, I = 64, 8
    rng = np.random.default_rng(5)
    model = np.zeros(I, np.int32)
    inst = synth.Instances(model, rng.uniform(0, 5000, I).astype(np.float32),
                           rng.uniform(0, 5000, I).astype(np.float32),
                           np.full(I, 10000, np.float32), np.full(I, 1000, np.float32),
                           (rng.integers(1, 64, I) / 1024).astype(np.float32),
                           (rng.integers(1, 64, I) / 1024).astype(np.float32))
    qh = rng.uniform(0, 1, (B, 1)).astype(np.float32)
    lh = rng.integers(1, 500, (B, 1)).astype(np.float32)
    pl = rng.integers(1, 3000, B).astype(np.int32)
    C = costs(lh, pl, inst)
    budget = C[np.arange(B), rng.integers(0, I, B)].astype(np.float32)
    assert np.array_equal(C.astype(np.float32).astype(np.float64), C)   # exact in fp32
    res = run_assign_ex(qh, lh, pl, inst, (0.3, 0.4, 0.3), budget=budget)
    check(res, qh, lh, pl, inst, (0.3, 0.4, 0.3), 0, budget=budget, label="boundary")
    assert np.all(res["assign"] >= 0)            # the budget's own instance is admitted
    assert np.all(C[np.arange(B), res["assign"]] <= budget)


def _fmaf():
    import ctypes
    import ctypes.util
    libm = ctypes.CDLL(ctypes.util.find_library("m"))
    libm.fmaf.restype = ctypes.c_float
    libm.fmaf.argtypes = [ctypes.c_float] * 3
    return libm.fmaf


@pytest.mark.parametrize("nudge", [-1, 0, 1])
def test_budget_at_the_fp32_cost_boundary(nudge):
    """Budgets placed on an instance's cost as fp32 evaluates it (one fused
    multiply-add), nudged by nudge ulps: the exact Eq. 2 cost that the oracle
    compares lies within rounding of the budget, so either admission is
    acceptable there (a counted boundary near-tie); every other instance's
    admission must match the oracle's exactly."""
    say(f"budget on the fp32 cost boundary, nudge {nudge} ulp")
    B, M, I = 200, 4, 13
    qh, lh, pl, inst = random_case(B, M, I, seed=31 + nudge)
    fmaf = _fmaf()
    rng = np.random.default_rng(8)
    pick = rng.integers(0, I, B)
    budget = np.empty(B, np.float32)
    for r in range(B):
        i = pick[r]
        prod = np.float32(np.float32(lh[r, inst.model[i]]) * np.float32(inst.price_out[i]))
        c32 = np.float32(fmaf(float(pl[r]), float(inst.price_in[i]), float(prod)))
        for _ in range(abs(nudge)):
            c32 = np.nextafter(c32, np.float32(np.inf if nudge > 0 else -np.inf))
        budget[r] = c32
    for w in [(0.3, 0.4, 0.3), (0, 0, 1)]:
        res = run_assign_ex(qh, lh, pl, inst, w, budget=budget)
        check(res, qh, lh, pl, inst, w, 0, budget=budget, label=f"w={w} nudge={nudge}")


def test_budget_mask_hand_example_on_gpu():
    say("budget/mask hand example")
    g = json.load(open(os.path.join(GOLD, "budget_mask_2x3.json")))
    inst = synth.Instances(*[np.array(g[f], np.int32 if f == "model" else np.float32)
                             for f in synth.Instances.FIELDS])
    qh = np.array(g["q_hat"], np.float32)
    lh = np.array(g["l_hat"], np.float32)
    pl = np.array(g["prompt_len"], np.int32)
    for c in g["cases"]:
        budget = None if c["budget"] is None else \
            np.array([np.inf if v == "inf" else v for v in c["budget"]], np.float32)
        mask = None if c["mask"] is None else np.array(c["mask"], np.uint8)
        res = run_assign_ex(qh, lh, pl, inst, g["weights"], budget=budget, mask=mask)
        assert res["assign"].tolist() == c["assign"], c["name"]
        expect = np.array([np.nan if v == "nan" else v for v in c["chosen"]])
        np.testing.assert_allclose(res["chosen"], expect, rtol=1e-6, equal_nan=True)
        np.testing.assert_allclose(res["p"], c["final_p"], rtol=1e-6)
        np.testing.assert_allclose(res["a"], c["final_a"], rtol=1e-6)


def test_nothing_available_leaves_everything_unassigned():
    say("empty candidate sets")
    qh, lh, pl, inst = random_case(50, 4, 13, seed=2)
    for kw in (dict(mask=np.zeros(13, np.uint8)),
               dict(budget=np.full(50, 1e-9, np.float32)),
               dict(budget=np.full(50, np.nan, np.float32))):
        res = run_assign_ex(qh, lh, pl, inst, (0.3, 0.4, 0.3), **kw)
        assert np.all(res["assign"] == -1) and np.all(np.isnan(res["chosen"]))
        assert np.array_equal(res["p"], inst.prefill_q)
        assert np.array_equal(res["a"], inst.decode_q)


def test_default_options_match_plain_assign():
    say("default options")
    qh, lh, pl, inst = random_case(300, 8, 64, seed=9)
    w = (0.4, 0.3, 0.3)
    res = run_assign_ex(qh, lh, pl, inst, w)
    gi = rb().DeviceInstances.from_host(inst, DEV)
    asg, ch = rb().rb_assign(dev(qh), dev(lh), dev(pl), gi, w)
    torch.cuda.synchronize()
    assert np.array_equal(res["assign"], asg.cpu().numpy())
    assert np.array_equal(res["chosen"].view(np.uint32), ch.cpu().numpy().view(np.uint32))
    assert res["order"].tolist() == list(range(300))     # order_out filled for arrival too


# ----------------------------------------------------------------------------- weighted average


@pytest.mark.parametrize("B,k,N,M", [(16, 10, 2048, 4), (1, 1, 5, 1), (65, 64, 3000, 16),
                                     (9, 7, 100, 70)])
def test_predict_inv_dist_parity(B, k, N, M):
    say(f"predict inv_dist B={B} k={k} N={N} M={M}")
    rng = np.random.default_rng(B * k + 1)
    nbr = np.stack([rng.choice(N, k, replace=False) for _ in range(B)]).astype(np.int32)
    dist = np.sort(rng.uniform(0, 2, (B, k)), axis=1).astype(np.float32)
    dist[0, 0] = 0.0                 # an exact duplicate
    if k > 1:
        dist[0, 1] = -3e-7           # fp32 cancellation below zero
    qual = rng.uniform(0, 1, (N, M)).astype(np.float32)
    ln = rng.integers(1, 3000, (N, M)).astype(np.float32)
    m = rb()
    qh, lh = m.rb_predict(dev(nbr), dev(qual), dev(ln), nbr_dist=dev(dist),
                          weighting=m.RB_KNN_INV_DIST)
    torch.cuda.synchronize()
    par.check_predictions(nbr, qh.cpu().numpy(), lh.cpu().numpy(), qual, ln, g_dist=dist,
                          weighting="inv_dist")


# ----------------------------------------------------------------------------- the whole path


def run_route_ex(cfg, bank, queries, qual, ln, pl, inst, order, weighting, budget, mask,
                 norms=None):
    m = rb()
    B, k, M = cfg.B, cfg.k, cfg.M
    gb = bank if bank.is_cuda else bank.to(DEV)
    norms = m.rb_bank_norms(gb) if norms is None else norms
    gi = m.DeviceInstances.from_host(inst, DEV)
    out = dict(nbr=torch.empty(B, k, dtype=torch.int32, device=DEV),
               nd=torch.empty(B, k, device=DEV), qh=torch.empty(B, M, device=DEV),
               lh=torch.empty(B, M, device=DEV), ch=torch.empty(B, device=DEV),
               order=torch.empty(B, dtype=torch.int32, device=DEV))
    opts = m.options(order=order, weighting=weighting,
                     budget=None if budget is None else dev(budget),
                     instance_mask=None if mask is None else dev(mask),
                     order_out=out["order"])
    asg = m.rb_route_batch_ex(queries.to(DEV), gb, norms, k, dev(qual), dev(ln), dev(pl), gi,
                              cfg.weights, opts, chosen=out["ch"], nbr_idx=out["nbr"],
                              nbr_dist=out["nd"], q_hat=out["qh"], l_hat=out["lh"])
    torch.cuda.synchronize()
    res = {kk: v.cpu().numpy() for kk, v in out.items()}
    res["assign"] = asg.cpu().numpy()
    res["p"] = gi.prefill_q.cpu().numpy()
    res["a"] = gi.decode_q.cpu().numpy()
    return res


def check_route_ex(cfg, res, queries, bank, qual, ln, pl, inst, order, weighting, budget, mask,
                   rows=None, label=""):
    m = rb()
    if rows is None:
        oi, od = oracle.knn(queries, bank, cfg.k, nthreads=16)
    else:
        oi, od = oracle.knn(queries[rows], bank, cfg.k, nthreads=16)
    ties = par.check_neighbours(res["nbr"], res["nd"], oi, od, rows=rows, label=label)
    wname = "inv_dist" if weighting == m.RB_KNN_INV_DIST else "uniform"
    par.check_predictions(res["nbr"], res["qh"], res["lh"], qual, ln, label=label,
                          g_dist=res["nd"], weighting=wname)
    near = par.check_assign(res["assign"], res["ch"], res["qh"], res["lh"], pl, inst, cfg.weights,
                            g_final_p=res["p"], g_final_a=res["a"], label=label,
                            order="lpt" if order == m.RB_ORDER_LPT else "arrival",
                            g_order=res["order"], budget=budget, mask=mask)
    return ties, near


@pytest.mark.parametrize("name,over", [
    ("tiny", {}),
    ("tiny-bf16", dict(dtype="bf16", d=768, N=20000, B=64, clusters=256)),
    ("tiny-wide", dict(dtype="bf16", d=384, N=5000, B=100, M=16, inst_per_model=(32,) * 16,
                       weights=(0.1, 0.2, 0.7))),
])
def test_route_batch_ex_end_to_end(name, over):
    m = rb()
    cfg = synth.tiny_config(**over)
    say(f"route_batch_ex {name}: B={cfg.B} N={cfg.N} d={cfg.d} {cfg.dtype} M={cfg.M} I={cfg.I}")
    centres = synth.make_centres(cfg)
    bank = synth.make_bank(cfg, centres=centres)
    queries = synth.make_queries(cfg, 0, centres=centres)
    qual, ln = synth.make_labels(cfg)
    pl = synth.make_prompt_lens(cfg)
    inst = synth.make_instances(cfg)
    budget = synth.make_budgets(cfg)
    mask = synth.make_availability(cfg, lost_models=(cfg.M - 1,), down_fraction=0.1)
    combos = [(m.RB_ORDER_LPT, m.RB_KNN_UNIFORM, None, None),
              (m.RB_ORDER_ARRIVAL, m.RB_KNN_INV_DIST, None, None),
              (m.RB_ORDER_ARRIVAL, m.RB_KNN_UNIFORM, budget, None),
              (m.RB_ORDER_ARRIVAL, m.RB_KNN_UNIFORM, None, mask),
              (m.RB_ORDER_LPT, m.RB_KNN_INV_DIST, budget, mask)]
    for order, weighting, bud, msk in combos:
        label = f"{name} order={order} wt={weighting} budget={bud is not None} " \
                f"mask={msk is not None}"
        say("  " + label)
        res = run_route_ex(cfg, bank, queries, qual, ln, pl, inst, order, weighting, bud, msk)
        ties, near = check_route_ex(cfg, res, queries, bank, qual, ln, pl, inst, order,
                                    weighting, bud, msk, label=label)
        free = par.free_running(queries, bank, cfg.k, qual, ln, pl, inst, cfg.weights,
                                nthreads=16, order="lpt" if order == m.RB_ORDER_LPT else "arrival",
                                weighting="inv_dist" if weighting else "uniform", budget=bud,
                                mask=msk)
        say(f"    neighbour near-ties {ties}, pick near-ties {near}")
        if ties == 0 and near == 0 and weighting == m.RB_KNN_UNIFORM:
            assert np.array_equal(free["assign"], res["assign"])
        res2 = run_route_ex(cfg, bank, queries, qual, ln, pl, inst, order, weighting, bud, msk)
        for kk in res:
            assert np.array_equal(res[kk].view(np.uint8), res2[kk].view(np.uint8)), kk


def test_route_batch_ex_defaults_match_route_batch():
    m = rb()
    cfg = synth.tiny_config(dtype="bf16", d=768, N=20000, B=64, clusters=256)
    say("route_batch_ex defaults")
    centres = synth.make_centres(cfg)
    bank = synth.make_bank(cfg, centres=centres).to(DEV)
    queries = synth.make_queries(cfg, 0, centres=centres)
    qual, ln = synth.make_labels(cfg)
    pl = synth.make_prompt_lens(cfg)
    inst = synth.make_instances(cfg)
    res = run_route_ex(cfg, bank, queries, qual, ln, pl, inst, m.RB_ORDER_ARRIVAL,
                       m.RB_KNN_UNIFORM, None, None)
    gi = m.DeviceInstances.from_host(inst, DEV)
    ch = torch.empty(cfg.B, device=DEV)
    asg = m.rb_route_batch(queries.to(DEV), bank, m.rb_bank_norms(bank), cfg.k, dev(qual),
                           dev(ln), dev(pl), gi, cfg.weights, chosen=ch)
    torch.cuda.synchronize()
    assert np.array_equal(res["assign"], asg.cpu().numpy())
    assert np.array_equal(res["ch"].view(np.uint32), ch.cpu().numpy().view(np.uint32))
    assert np.array_equal(res["p"], gi.prefill_q.cpu().numpy())


def test_full_size_options_sampled_parity():
    """The high-load workload at its real size with every option on (LPT order,
    inverse-distance average, budgets on 45 % of the requests, the last model's
    tier lost): neighbours of a spread sample of requests, every prediction and
    every pick teacher-forced."""
    m = rb()
    cfg = synth.CONFIGS["highload"]
    say(f"full-size options highload: B={cfg.B} N={cfg.N} d={cfg.d}")
    centres = synth.make_centres(cfg, DEV)
    bank = synth.make_bank(cfg, DEV, centres)
    queries = synth.make_queries(cfg, 0, DEV, centres)
    qual, ln = synth.make_labels(cfg)
    pl = synth.make_prompt_lens(cfg)
    inst = synth.make_instances(cfg)
    budget = synth.make_budgets(cfg)
    mask = synth.make_availability(cfg, lost_models=(cfg.M - 1,))
    res = run_route_ex(cfg, bank, queries, qual, ln, pl, inst, m.RB_ORDER_LPT,
                       m.RB_KNN_INV_DIST, budget, mask)
    say("  gpu done; oracle ...")
    rows = np.linspace(0, cfg.B - 1, 8).round().astype(int)
    bank_h = bank.cpu()
    q_h = queries.cpu()
    del bank
    torch.cuda.empty_cache()
    ties, near = check_route_ex(cfg, res, q_h, bank_h, qual, ln, pl, inst, m.RB_ORDER_LPT,
                                m.RB_KNN_INV_DIST, budget, mask, rows=rows, label="highload-ex")
    say(f"  neighbour near-ties {ties}, pick near-ties {near}, "
        f"unassigned {(res['assign'] < 0).sum()}")
