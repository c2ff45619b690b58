"""GPU parity: every C-ABI entry point against the CPU oracle.

Inputs are seeded synthetic workloads (synth). Acceptance rules are those of
oracle.parity: neighbours exact up to boundary near-ties within 1e-5, values
within 1e-4, assignments teacher-forced with near-ties within 1e-5 and
bit-identical free-running picks when no near tie occurred.
"""
import os

import numpy as np
import pytest
import torch

import oracle
import oracle.parity as par
import synth

pytestmark = pytest.mark.gpu

DEV = "cuda"


def rb():
    import paper_2606_17949_amd as m
    return m


def say(msg):
    print(msg, flush=True)


def gpu_knn(q, x, k, norms=None):
    m = rb()
    gq, gx = q.to(DEV), x.to(DEV)
    if norms is None:
        norms = m.rb_bank_norms(gx)
    idx, dist = m.rb_knn_topk(gq, gx, norms, k)
    torch.cuda.synchronize()
    return idx.cpu().numpy(), dist.cpu().numpy()


def clustered(B, N, d, dtype, seed, clusters=32, plant=True):
    cfg = synth.tiny_config(B=B, N=N, d=d, dtype=dtype, clusters=clusters, seed=seed)
    centres = synth.make_centres(cfg)
    x = synth.make_bank(cfg, centres=centres)
    q = synth.make_queries(cfg, 0, centres=centres)
    if plant and N >= 8:
        # exact duplicate rows (equal distances: the lower index must come first)
        x[N - 1] = x[3]
        x[N // 2] = x[N // 3]
        if B > 1:
            q[1] = x[N // 3]            # a query equal to a bank row (twice present)
    return q, x


# ----------------------------------------------------------------------------- norms


@pytest.mark.parametrize("dtype,N,d", [("f32", 1000, 384), ("bf16", 3001, 768), ("bf16", 7, 8),
                                       ("f32", 5, 2048), ("bf16", 100, 2048)])
def test_bank_norms(dtype, N, d):
    say(f"bank_norms {dtype} N={N} d={d}")
    _, x = clustered(1, N, d, dtype, seed=N + d, plant=False)
    g = rb().rb_bank_norms(x.to(DEV))
    torch.cuda.synchronize()
    ref = (x.double() ** 2).sum(1).numpy()
    e = par.rel(g.cpu().numpy(), ref, 1e-6)
    assert e.max() <= 1e-5, e.max()


# ----------------------------------------------------------------------------- KNN

KNN_CASES = [
    # dtype, B, N, d, k
    ("f32", 16, 2048, 384, 10),     # the tiny workload's shape
    ("bf16", 1, 10, 8, 10),         # k = N, one request, smallest d
    ("bf16", 3, 11, 16, 10),        # N = k + 1
    ("bf16", 63, 1000, 384, 10),
    ("bf16", 64, 4097, 768, 10),    # ragged last tile
    ("bf16", 65, 1000, 64, 1),      # two query tiles, k = 1
    ("bf16", 257, 2000, 128, 64),   # ragged query tiles, largest k
    ("f32", 5, 3000, 36, 17),       # ragged d inside a k-step
    ("bf16", 17, 5000, 1024, 10),
    ("bf16", 33, 3000, 2048, 10),   # largest d
    ("f32", 20, 500, 2048, 5),      # largest d, fp32
    ("bf16", 40, 64, 40, 33),       # fewer rows than chunks can use
    ("bf16", 256, 150, 512, 10),    # no seed (8 sample groups < k): every pair of the
                                    # first iteration is a candidate, most past the LDS staging
    # the seed bound's wave holds each lane's two smallest group minima
    ("bf16", 100, 700, 768, 20),    # 40 groups: fewer than the wave's lanes
    ("bf16", 100, 1600, 768, 64),   # 100 groups, one or two per lane, largest k
    # bf16 rows of 384, 512, 768 or 1024 elements take the query-resident
    # scan while the batch fits its registers: (query groups per wave, row
    # halves) of (1, 2) up to 64 requests, (2, 2) up to 128, then (4, 2) for
    # d = 384 and (2, 1) for d = 512 and 768 up to 256
    ("bf16", 100, 50000, 768, 10),  # (2, 2): a partly filled wave and idle waves
    ("bf16", 200, 100003, 768, 16), # (2, 1); chunks that end inside a block
    ("bf16", 129, 70000, 768, 1),   # k = 1
    ("bf16", 200, 9000, 768, 17),
    ("bf16", 70, 20, 768, 10),      # fewer bank rows than one of its 32-row blocks
    ("bf16", 65, 1, 768, 1),        # a single bank row
    ("bf16", 256, 600, 768, 10),    # a full batch with a 36-group seed
    ("bf16", 200, 4096, 768, 16),   # 128 seed groups: exactly two per lane of the bound
    ("bf16", 1, 530000, 768, 10),   # a single request: two active waves
    ("bf16", 64, 530000, 768, 64),  # (1, 2), k = 64 (batches of up to 64 take it from
                                    # 2,048 rows per compute unit)
    ("bf16", 90, 60000, 768, 20),   # (2, 2), k = 20
    ("bf16", 40, 530000, 384, 10),  # d = 384, (1, 2)
    ("bf16", 40, 530000, 384, 64),  # d = 384, (1, 2), k = 64: a two-slot ring
    ("bf16", 40, 30000, 384, 10),   # the same batch over a small bank: the tile scan
    ("bf16", 100, 30000, 384, 20),  # d = 384, (2, 2), k = 20
    ("bf16", 256, 50000, 384, 10),  # d = 384, (4, 2)
    ("bf16", 512, 60000, 384, 10),  # d = 384, (4, 1): the wide workload's batch, tiles one
                                    # after the other
    ("bf16", 300, 20000, 384, 16),  # (4, 1), k = 16: a two-slot ring; a partly filled wave
    ("bf16", 64, 530000, 512, 64),  # d = 512, (1, 2), k = 64
    ("bf16", 128, 40000, 512, 20),  # d = 512, (2, 2)
    ("bf16", 250, 40000, 512, 10),  # d = 512, (2, 1)
    ("bf16", 64, 530000, 1024, 10), # d = 1024, (1, 2)
    ("bf16", 128, 30000, 1024, 64), # d = 1024, (1, 1), k = 64: half-block stages
    ("bf16", 100, 40, 1024, 33),    # fewer rows than chunks
    ("bf16", 100, 60000, 1024, 20), # d = 1024, (1, 1), k = 20
    # batches of more than 128 over a bank of more than 32 x 32,768 rows (where
    # the seed covers less than 1/32 of it): two passes, the first eighth of
    # every chunk, then the rest under the k-th smallest entry of the first
    # pass's lists, each pass leaving its own lists
    ("bf16", 160, 1101825, 384, 10),  # (4, 2); the last chunk ends inside the first pass
    ("bf16", 300, 1100000, 384, 20),  # (4, 1), tiles one after the other
    ("bf16", 200, 1100000, 768, 10),  # (2, 1)
    ("bf16", 129, 1100000, 512, 32),  # (2, 1), k = 32: the smallest batch that splits
    # more than 256 bf16 requests whose rows are whole 64-element lines, k <= 10,
    # take the GEMM-structured scan: 256 x 256 macro tiles, 32x32x16 MFMAs
    ("bf16", 257, 3000, 128, 10),   # a second request tile of one request; two stages per tile
    ("bf16", 600, 20000, 384, 10),  # three request tiles, the last partly filled
    ("bf16", 1024, 50000, 1024, 10),# four request tiles: the largebatch shape over a small bank
    ("bf16", 513, 10007, 768, 5),   # ragged bank: the last macro tile of a chunk partly filled
    ("bf16", 400, 30, 256, 10),     # fewer rows than one macro tile, most chunks empty
    ("bf16", 300, 100000, 512, 1),  # k = 1
]


@pytest.mark.parametrize("dtype,B,N,d,k", KNN_CASES)
def test_knn_parity(dtype, B, N, d, k):
    say(f"knn {dtype} B={B} N={N} d={d} k={k}")
    q, x = clustered(B, N, d, dtype, seed=B * 1000 + N)
    gi, gd = gpu_knn(q, x, k)
    oi, od = oracle.knn(q, x, k, nthreads=8)
    ties = par.check_neighbours(gi, gd, oi, od, label=f"{dtype} B={B} N={N} d={d} k={k}")
    say(f"  boundary near-ties: {ties}")


def test_knn_exact_ties_take_lower_index():
    say("knn exact ties")
    # every bank row identical: all distances equal, order must be index order
    x = torch.ones(300, 64).bfloat16()
    q = torch.zeros(4, 64).bfloat16()
    gi, gd = gpu_knn(q, x, 64)
    assert (gi == np.arange(64)[None, :]).all()
    assert np.all(gd == 64.0)


@pytest.mark.parametrize("label,B,N,d,k", [
    ("query-resident scan", 200, 70000, 768, 10),
    ("query-resident scan, two passes", 200, 1100000, 384, 10),
    ("seeded tile scan, one tile", 64, 70000, 768, 10),
    ("seeded tile scan, two tiles", 300, 66000, 256, 16),
    ("GEMM-structured scan", 300, 66000, 256, 10),
])
def test_knn_exact_ties_across_kth(label, B, N, d, k):
    """Duplicated rows straddling the k-th position: each request's k-th
    neighbour is copied into two other rows, one lower and one higher where
    the bank allows, spread over the bank's chunks. The three rows are at
    exactly the same distance on both sides, so only the lowest index may be
    in the list; the extended oracle lists make check_neighbours enforce it."""
    say(f"knn exact ties across k: {label} B={B} N={N} d={d} k={k}")
    q, x = clustered(B, N, d, "bf16", seed=N + B, plant=False)
    oi, _ = oracle.knn(q, x, k + 2, nthreads=16)
    rng = np.random.default_rng(B)
    used = set(oi.ravel().tolist())
    free = np.array([n for n in rng.permutation(N) if n not in used])
    fi = 0
    for b in range(B):
        src = int(oi[b, k - 1])
        lo = free[fi:][free[fi:] < src][:1]
        hi = free[fi:][free[fi:] > src][:1]
        for j in np.concatenate([lo, hi]):
            x[int(j)] = x[src]
            free = free[free != j]
    oi, od = oracle.knn(q, x, k + 4, nthreads=16)
    straddle = int(np.sum(od[:, k - 1] == od[:, k]))
    say(f"  requests with an exact tie across the k-th position: {straddle}/{B}")
    assert straddle >= B // 2
    gi, gd = gpu_knn(q, x, k)
    ties = par.check_neighbours(gi, gd, oi, od, label=label)
    say(f"  boundary near-ties: {ties}")


def test_knn_deterministic():
    say("knn determinism")
    q, x = clustered(70, 20000, 256, "bf16", seed=9)
    a = gpu_knn(q, x, 10)
    b = gpu_knn(q, x, 10)
    assert np.array_equal(a[0], b[0]) and np.array_equal(a[1].view(np.uint32), b[1].view(np.uint32))


# ----------------------------------------------------------------------------- predict


@pytest.mark.parametrize("B,k,N,M", [(16, 10, 2048, 4), (1, 1, 5, 1), (65, 64, 3000, 16),
                                     (9, 7, 100, 70)])
def test_predict_parity(B, k, N, M):
    say(f"predict B={B} k={k} N={N} M={M}")
    rng = np.random.default_rng(B + k)
    nbr = np.stack([rng.choice(N, k, replace=False) for _ in range(B)]).astype(np.int32)
    qual = rng.uniform(0, 1, (N, M)).astype(np.float32)
    ln = rng.integers(1, 3000, (N, M)).astype(np.float32)
    qh, lh = rb().rb_predict(torch.from_numpy(nbr).to(DEV), torch.from_numpy(qual).to(DEV),
                             torch.from_numpy(ln).to(DEV))
    torch.cuda.synchronize()
    par.check_predictions(nbr, qh.cpu().numpy(), lh.cpu().numpy(), qual, ln)


def test_predict_out_of_range_index_gives_nan():
    say("predict bad index")
    nbr = torch.tensor([[0, 1], [2, 99]], dtype=torch.int32, device=DEV)
    qual = torch.rand(10, 3, device=DEV)
    ln = torch.rand(10, 3, device=DEV)
    qh, lh = rb().rb_predict(nbr, qual, ln)
    torch.cuda.synchronize()
    assert torch.isfinite(qh[0]).all() and torch.isnan(qh[1]).all() and torch.isnan(lh[1]).all()


# ----------------------------------------------------------------------------- score / assign

ROUTE_CASES = [
    # B, M, I
    (16, 4, 13),
    (5, 1, 1),        # one instance
    (64, 8, 64),
    (33, 16, 512),
    (7, 3, 1024),     # largest instance count
    (300, 4, 65),     # I just past one wave's lanes
    (40, 4, 16),      # the most instances one 16-lane row holds
    (40, 4, 17),      # one more: a full-wave layout
]


def random_route_case(B, M, I, seed):
    rng = np.random.default_rng(seed)
    per = [I // M + (1 if m < I % M else 0) for m in range(M)]
    cfg = synth.tiny_config(B=B, M=M, inst_per_model=tuple(per), seed=seed)
    inst = synth.make_instances(cfg)
    qh = rng.uniform(0, 1, (B, M)).astype(np.float32)
    lh = rng.uniform(1, 800, (B, M)).astype(np.float32)
    pl = rng.integers(1, 3000, B).astype(np.int32)
    return qh, lh, pl, inst


def dev(a, dtype=None):
    t = torch.from_numpy(np.ascontiguousarray(a))
    return t.to(DEV) if dtype is None else t.to(device=DEV, dtype=dtype)


@pytest.mark.parametrize("B,M,I", ROUTE_CASES)
@pytest.mark.parametrize("w", [(0.4, 0.3, 0.3), (1, 0, 0), (0, 1, 0), (0, 0, 1), (0.1, 0.2, 0.7)])
def test_score_parity(B, M, I, w):
    say(f"score B={B} M={M} I={I} w={w}")
    qh, lh, pl, inst = random_route_case(B, M, I, seed=B * 7 + I)
    gi = rb().DeviceInstances.from_host(inst, DEV)
    S0 = rb().rb_score(dev(qh), dev(lh), dev(pl), gi, w)
    torch.cuda.synchronize()
    par.check_scores(S0.cpu().numpy(), qh, lh, pl, inst, w)
    # the state is read only
    assert np.array_equal(gi.prefill_q.cpu().numpy(), inst.prefill_q)


@pytest.mark.parametrize("B,M,I", ROUTE_CASES)
@pytest.mark.parametrize("w", [(0.4, 0.3, 0.3), (1, 0, 0), (0, 1, 0), (0, 0, 1), (0.1, 0.2, 0.7)])
def test_assign_parity(B, M, I, w):
    say(f"assign B={B} M={M} I={I} w={w}")
    qh, lh, pl, inst = random_route_case(B, M, I, seed=B * 7 + I)
    gi = rb().DeviceInstances.from_host(inst, DEV)
    decided = torch.empty(B, I, device=DEV)
    asg, ch = rb().rb_assign(dev(qh), dev(lh), dev(pl), gi, w, decided=decided)
    torch.cuda.synchronize()
    a_h, c_h, d_h = asg.cpu().numpy(), ch.cpu().numpy(), decided.cpu().numpy()
    near = par.check_assign(a_h, c_h, qh, lh, pl, inst, w,
                            g_final_p=gi.prefill_q.cpu().numpy(),
                            g_final_a=gi.decode_q.cpu().numpy(), g_decided=d_h)
    # the chosen score is the decided row's entry at the pick, bit for bit
    assert np.array_equal(c_h.view(np.uint32), d_h[np.arange(B), a_h].view(np.uint32))
    # the first row was decided at the batch-start state: rb_score's row
    S0 = rb().rb_score(dev(qh), dev(lh), dev(pl), rb().DeviceInstances.from_host(inst, DEV), w)
    torch.cuda.synchronize()
    assert np.array_equal(S0.cpu().numpy()[0].view(np.uint32), d_h[0].view(np.uint32))
    free = oracle.assign(qh.astype(np.float64), lh.astype(np.float64), pl, inst, w)
    if near == 0:
        assert np.array_equal(free["assign"], a_h)
    say(f"  near-ties {near}")


def test_zero_prices_on_gpu():
    # every price zero: the cost maximum is zero, so the cost ratio is 0 and
    # the cost term adds w_cost to every instance (the zero-maximum reading);
    # with w = (0, 0, 1) every score is 1 and the lowest index wins
    say("zero prices")
    qh, lh, pl, inst = random_route_case(40, 4, 13, seed=77)
    inst.price_in[:] = 0
    inst.price_out[:] = 0
    for w in [(0, 0, 1), (0.4, 0.3, 0.3), (0.1, 0.2, 0.7)]:
        gi = rb().DeviceInstances.from_host(inst, DEV)
        S0 = rb().rb_score(dev(qh), dev(lh), dev(pl), gi, w)
        decided = torch.empty(40, 13, device=DEV)
        asg, ch = rb().rb_assign(dev(qh), dev(lh), dev(pl), gi, w, decided=decided)
        torch.cuda.synchronize()
        par.check_scores(S0.cpu().numpy(), qh, lh, pl, inst, w)
        near = par.check_assign(asg.cpu().numpy(), ch.cpu().numpy(), qh, lh, pl, inst, w,
                                g_final_p=gi.prefill_q.cpu().numpy(),
                                g_final_a=gi.decode_q.cpu().numpy(),
                                g_decided=decided.cpu().numpy())
        if w == (0, 0, 1):
            assert np.all(S0.cpu().numpy() == 1.0)
            assert np.all(asg.cpu().numpy() == 0)
        say(f"  w={w} near-ties {near}")


def test_assign_hand_example_on_gpu():
    import json
    import os
    say("assign hand example")
    g = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "score_2x3.json")))
    inst = synth.Instances(*[np.array(g[f], np.int32 if f == "model" else np.float32)
                             for f in synth.Instances.FIELDS])
    qh = np.array(g["q_hat"], np.float32)
    lh = np.array(g["l_hat"], np.float32)
    pl = np.array(g["prompt_len"], np.int32)
    for w, exp, fp, fa in [(g["weights"], g["expect_assign"], g["expect_final_p"],
                            g["expect_final_a"])] + \
            [(c["weights"], c["assign"], c["final_p"], c["final_a"]) for c in g["corners"]]:
        gi = rb().DeviceInstances.from_host(inst, DEV)
        S0 = rb().rb_score(dev(qh), dev(lh), dev(pl), gi, w)
        asg, ch = rb().rb_assign(dev(qh), dev(lh), dev(pl), gi, w)
        torch.cuda.synchronize()
        assert asg.cpu().tolist() == exp, w
        np.testing.assert_allclose(gi.prefill_q.cpu().numpy(), fp, rtol=1e-6)
        np.testing.assert_allclose(gi.decode_q.cpu().numpy(), fa, rtol=1e-6)
        if list(w) == list(g["weights"]):
            np.testing.assert_allclose(S0.cpu().numpy(), g["expect_S0"], rtol=1e-6)


def test_assign_bad_model_id_never_chosen():
    say("assign bad model id")
    qh, lh, pl, inst = random_route_case(8, 2, 4, seed=3)
    inst.model[:] = [0, 7, -1, 1]      # instances 1 and 2 name no model
    gi = rb().DeviceInstances.from_host(inst, DEV)
    asg, _ = rb().rb_assign(dev(qh), dev(lh), dev(pl), gi, (0.3, 0.4, 0.3))
    torch.cuda.synchronize()
    assert set(asg.cpu().tolist()) <= {0, 3}


def test_advance_parity():
    say("advance")
    qh, lh, pl, inst = random_route_case(4, 4, 300, seed=1)
    gi = rb().DeviceInstances.from_host(inst, DEV)
    for dt in (0.0, 0.37, 8.533333, 100.0):
        rb().rb_advance_state(gi, dt)
        torch.cuda.synchronize()
        p, a = oracle.advance(inst.prefill_q, inst.decode_q, inst.prefill_rate, inst.decode_rate,
                              np.float32(dt))
        np.testing.assert_allclose(gi.prefill_q.cpu().numpy(), p, rtol=1e-5, atol=1e-3)
        np.testing.assert_allclose(gi.decode_q.cpu().numpy(), a, rtol=1e-5, atol=1e-3)
        inst.prefill_q = gi.prefill_q.cpu().numpy()
        inst.decode_q = gi.decode_q.cpu().numpy()


# ----------------------------------------------------------------------------- the whole path


def run_route(cfg, bank, queries, qual, ln, pl, inst, norms=None):
    m = rb()
    B, k, M = cfg.B, cfg.k, cfg.M
    gb = bank if bank.is_cuda else bank.to(DEV)
    norms = m.rb_bank_norms(gb) if norms is None else norms
    gi = m.DeviceInstances.from_host(inst, DEV)
    out = dict(nbr=torch.empty(B, k, dtype=torch.int32, device=DEV),
               nd=torch.empty(B, k, device=DEV), qh=torch.empty(B, M, device=DEV),
               lh=torch.empty(B, M, device=DEV), ch=torch.empty(B, device=DEV),
               s0=torch.empty(B, gi.I, device=DEV))
    asg = m.rb_route_batch(queries.to(DEV), gb, norms, k, dev(qual), dev(ln), dev(pl), gi,
                           cfg.weights, chosen=out["ch"], nbr_idx=out["nbr"], nbr_dist=out["nd"],
                           q_hat=out["qh"], l_hat=out["lh"], score0=out["s0"])
    torch.cuda.synchronize()
    res = {kk: v.cpu().numpy() for kk, v in out.items()}
    res["assign"] = asg.cpu().numpy()
    res["p"] = gi.prefill_q.cpu().numpy()
    res["a"] = gi.decode_q.cpu().numpy()
    return res


def check_route(cfg, res, queries, bank, qual, ln, pl, inst, rows=None, label=""):
    # the oracle lists run 4 past k: they decide exact ties across the k-th
    threads = len(os.sched_getaffinity(0))
    if rows is None:
        oi, od = oracle.knn(queries, bank, cfg.k + 4, nthreads=threads)
    else:
        oi, od = oracle.knn(queries[rows], bank, cfg.k + 4, nthreads=threads)
    ties = par.check_neighbours(res["nbr"], res["nd"], oi, od, rows=rows, label=label)
    par.check_predictions(res["nbr"], res["qh"], res["lh"], qual, ln, label=label)
    par.check_scores(res["s0"], res["qh"], res["lh"], pl, inst, cfg.weights, label=label)
    near = par.check_assign(res["assign"], res["ch"], res["qh"], res["lh"], pl, inst, cfg.weights,
                            g_final_p=res["p"], g_final_a=res["a"], label=label)
    return ties, near


@pytest.mark.parametrize("name,over", [
    ("tiny", {}),
    ("tiny-bf16", dict(dtype="bf16", d=768, N=20000, B=64, clusters=256)),
    ("tiny-wide", dict(dtype="bf16", d=384, N=5000, B=100, M=16, inst_per_model=(32,) * 16,
                       weights=(0.1, 0.2, 0.7))),
])
def test_route_batch_end_to_end(name, over):
    cfg = synth.tiny_config(**over)
    say(f"route_batch {name}: B={cfg.B} N={cfg.N} d={cfg.d} {cfg.dtype} M={cfg.M} I={cfg.I}")
    centres = synth.make_centres(cfg)
    bank = synth.make_bank(cfg, centres=centres)
    queries = synth.make_queries(cfg, 0, centres=centres)
    qual, ln = synth.make_labels(cfg)
    pl = synth.make_prompt_lens(cfg)
    inst = synth.make_instances(cfg)
    res = run_route(cfg, bank, queries, qual, ln, pl, inst)
    ties, near = check_route(cfg, res, queries, bank, qual, ln, pl, inst, label=name)
    free = par.free_running(queries, bank, cfg.k, qual, ln, pl, inst, cfg.weights, nthreads=16)
    say(f"  neighbour near-ties {ties}, pick near-ties {near}")
    if ties == 0 and near == 0:
        assert np.array_equal(free["assign"], res["assign"])
    # determinism of the whole path
    res2 = run_route(cfg, bank, queries, qual, ln, pl, inst)
    for kk in res:
        assert np.array_equal(res[kk].view(np.uint8), res2[kk].view(np.uint8)), kk


# ----------------------------------------------------------------------------- full sizes


@pytest.mark.timeout(900)
@pytest.mark.parametrize("name,sample", [("online", None), ("highload", None),
                                         ("largebatch", None), ("wide", None),
                                         ("stream64", None)])
def test_full_size_parity(name, sample):
    """The workloads at their real sizes, in the configuration the benchmark
    times. The oracle recomputes every request's neighbour list (exact, on
    all host threads: up to about a minute for the largebatch workload), and
    every prediction, score and pick (teacher forced)."""
    cfg = synth.CONFIGS[name]
    say(f"full-size {name}: B={cfg.B} N={cfg.N} d={cfg.d} M={cfg.M} I={cfg.I}")
    centres = synth.make_centres(cfg, DEV)
    bank = synth.make_bank(cfg, DEV, centres)
    queries = synth.make_queries(cfg, 0, DEV, centres)
    qual, ln = synth.make_labels(cfg)
    pl = synth.make_prompt_lens(cfg)
    inst = synth.make_instances(cfg)
    res = run_route(cfg, bank, queries, qual, ln, pl, inst)
    say("  gpu done; oracle ...")
    rows = None if sample is None else np.linspace(0, cfg.B - 1, sample).round().astype(int)
    bank_h = bank.cpu()
    q_h = queries.cpu()
    del bank
    torch.cuda.empty_cache()
    ties, near = check_route(cfg, res, q_h, bank_h, qual, ln, pl, inst, rows=rows, label=name)
    say(f"  neighbour near-ties {ties}, pick near-ties {near}")
