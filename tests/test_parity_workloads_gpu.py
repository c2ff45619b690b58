"""GPU parity at the workloads' own structure, against the CPU oracle.

* High-load (B=256, N=1,000,000, d=768 bf16): consecutive batches whose
  dead-reckoned state carries forward (1/30 s per request between batches).
  Every batch is replayed teacher-forced from the GPU's own state at its
  start (Alg. 1's greedy loop, with the scores each step saw), and the state
  after the carry is checked against the oracle's carry of the replayed
  state. The first four batches also run free-running: the oracle's own
  neighbour search, predictions, greedy loop and carry, chained.
* Online (B=64, N=100,000, d=768 bf16): one lookup, then the score matrix
  and the greedy loop at every point of the step-0.2 simplex lattice of
  Eq. 1's weights (21 points, corners included) and of the step-0.25
  lattice (15 points), each from a copy of the batch-start state.

Acceptance rules are those of oracle.parity.
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


def say(msg):
    print(msg, flush=True)


def threads():
    return len(os.sched_getaffinity(0))


def workload(name):
    import paper_2606_17949_amd as rb
    cfg = synth.CONFIGS[name]
    centres = synth.make_centres(cfg, DEV)
    bank = synth.make_bank(cfg, DEV, centres)
    qual, ln = synth.make_labels(cfg)
    return dict(rb=rb, cfg=cfg, centres=centres, bank=bank, norms=rb.rb_bank_norms(bank),
                qual=qual, ln=ln, gq=torch.from_numpy(qual).to(DEV),
                gl=torch.from_numpy(ln).to(DEV), inst_h=synth.make_instances(cfg))


def gpu_batch(w, gi, t, weights):
    """One batch on the GPU: lookup with its lists, greedy loop with the
    decided rows, carry. Returns host copies of everything."""
    rb, cfg = w["rb"], w["cfg"]
    B, k, M, I = cfg.B, cfg.k, cfg.M, cfg.I
    q = synth.make_queries(cfg, t, DEV, w["centres"])
    pl = synth.make_prompt_lens(cfg, t)
    p0, a0 = gi.prefill_q.cpu().numpy(), gi.decode_q.cpu().numpy()
    nbr = torch.empty(B, k, dtype=torch.int32, device=DEV)
    nd = torch.empty(B, k, device=DEV)
    qh, lh = rb.rb_knn_predict(q, w["bank"], w["norms"], k, w["gq"], w["gl"], nbr_idx=nbr,
                               nbr_dist=nd)
    decided = torch.empty(B, I, device=DEV)
    asg, ch = rb.rb_assign(qh, lh, torch.from_numpy(pl).to(DEV), gi, weights, decided=decided)
    torch.cuda.synchronize()
    p1, a1 = gi.prefill_q.cpu().numpy(), gi.decode_q.cpu().numpy()
    rb.rb_advance_state(gi, B / 30.0)
    torch.cuda.synchronize()
    return dict(q=q.cpu(), pl=pl, p0=p0, a0=a0, nbr=nbr.cpu().numpy(), nd=nd.cpu().numpy(),
                qh=qh.cpu().numpy(), lh=lh.cpu().numpy(), assign=asg.cpu().numpy(),
                chosen=ch.cpu().numpy(), decided=decided.cpu().numpy(), p1=p1, a1=a1,
                p2=gi.prefill_q.cpu().numpy(), a2=gi.decode_q.cpu().numpy())


def check_state(g, o, label):
    e = par.rel(g, o, par.VAL_FLOOR)
    assert e.max() <= par.VAL_RTOL, f"{label}: state rel err {e.max()}"


@pytest.mark.timeout(600)
def test_highload_carried_batches_teacher_forced():
    w = workload("highload")
    rb, cfg = w["rb"], w["cfg"]
    say(f"highload carried: B={cfg.B} N={cfg.N} d={cfg.d}, 12 batches, dt={cfg.B / 30:.4f} s")
    gi = rb.DeviceInstances.from_host(w["inst_h"], DEV)
    inst = w["inst_h"]
    # the oracle's state chained over the whole run from the GPU's picks
    p_chain = inst.prefill_q.astype(np.float64)
    a_chain = inst.decode_q.astype(np.float64)
    total_near = 0
    for t in range(12):
        g = gpu_batch(w, gi, t, cfg.weights)
        label = f"highload batch {t}"
        par.check_predictions(g["nbr"], g["qh"], g["lh"], w["qual"], w["ln"], label=label)
        st = {}
        near = par.check_assign(g["assign"], g["chosen"], g["qh"], g["lh"], g["pl"], inst,
                                cfg.weights, p0=g["p0"], a0=g["a0"], g_final_p=g["p1"],
                                g_final_a=g["a1"], g_decided=g["decided"], label=label,
                                stats=st)
        # the carry of the replayed state, and of the chained state
        rp = par.replay_state(g["assign"], g["lh"], g["pl"], inst, g["p0"], g["a0"])
        op, oa = oracle.advance(rp[0], rp[1], inst.prefill_rate, inst.decode_rate,
                                np.float32(cfg.B / 30.0))
        check_state(g["p2"], op, f"{label} prefill after the carry")
        check_state(g["a2"], oa, f"{label} decode after the carry")
        cp = par.replay_state(g["assign"], g["lh"], g["pl"], inst, p_chain, a_chain)
        p_chain, a_chain = oracle.advance(cp[0], cp[1], inst.prefill_rate, inst.decode_rate,
                                          np.float32(cfg.B / 30.0))
        check_state(g["p2"], p_chain, f"{label} prefill against the chain from batch 0")
        check_state(g["a2"], a_chain, f"{label} decode against the chain from batch 0")
        total_near += near
        say(f"  batch {t}: near-ties {st}, picks per instance "
            f"{np.bincount(g['assign'], minlength=cfg.I).tolist()}")
    say(f"  12 batches, near-tie events {total_near}")


@pytest.mark.timeout(900)
def test_highload_first_batches_free_running():
    w = workload("highload")
    rb, cfg = w["rb"], w["cfg"]
    say(f"highload free-running: batches 0-3 against the oracle alone ({threads()} threads)")
    gi = rb.DeviceInstances.from_host(w["inst_h"], DEV)
    inst = w["inst_h"]
    bank_h = w["bank"].cpu()
    o_inst = inst.copy()
    clean = True
    for t in range(4):
        g = gpu_batch(w, gi, t, cfg.weights)
        label = f"highload batch {t}"
        oi, od = oracle.knn(g["q"], bank_h, cfg.k + 4, nthreads=threads())
        ties = par.check_neighbours(g["nbr"], g["nd"], oi, od, label=label)
        near = par.check_assign(g["assign"], g["chosen"], g["qh"], g["lh"], g["pl"], inst,
                                cfg.weights, p0=g["p0"], a0=g["a0"], g_final_p=g["p1"],
                                g_final_a=g["a1"], label=label)
        # the oracle alone, from its own chained state
        qh, lh = oracle.predict(oi[:, :cfg.k], w["qual"], w["ln"])
        o = oracle.assign(qh, lh, g["pl"], o_inst, cfg.weights)
        p2, a2 = oracle.advance(o["p"], o["a"], inst.prefill_rate, inst.decode_rate,
                                np.float32(cfg.B / 30.0))
        o_inst.prefill_q, o_inst.decode_q = p2, a2
        clean = clean and ties == 0 and near == 0
        diff = np.flatnonzero(o["assign"] != g["assign"])
        say(f"  batch {t}: neighbour near-ties {ties}, pick near-ties {near}, "
            f"free-running picks differ at {diff.size} requests")
        if clean:
            assert diff.size == 0, f"{label}: free-running picks differ first at {diff[0]}"
            check_state(g["p2"], p2, f"{label} free-running prefill")
            check_state(g["a2"], a2, f"{label} free-running decode")


@pytest.mark.timeout(600)
def test_online_weight_sweep():
    w = workload("online")
    rb, cfg = w["rb"], w["cfg"]
    lattices = synth.simplex_lattice(0.2) + synth.simplex_lattice(0.25)
    assert len(lattices) == 21 + 15
    say(f"online sweep: B={cfg.B} N={cfg.N}, {len(lattices)} weight points")
    B, k, M, I = cfg.B, cfg.k, cfg.M, cfg.I
    q = synth.make_queries(cfg, 0, DEV, w["centres"])
    pl = synth.make_prompt_lens(cfg, 0)
    nbr = torch.empty(B, k, dtype=torch.int32, device=DEV)
    nd = torch.empty(B, k, device=DEV)
    qh, lh = rb.rb_knn_predict(q, w["bank"], w["norms"], k, w["gq"], w["gl"], nbr_idx=nbr,
                               nbr_dist=nd)
    torch.cuda.synchronize()
    g_nbr, g_qh, g_lh = nbr.cpu().numpy(), qh.cpu().numpy(), lh.cpu().numpy()
    oi, od = oracle.knn(q.cpu(), w["bank"].cpu(), k + 4, nthreads=threads())
    ties = par.check_neighbours(g_nbr, nd.cpu().numpy(), oi, od, label="online")
    par.check_predictions(g_nbr, g_qh, g_lh, w["qual"], w["ln"], label="online")
    o_qh, o_lh = oracle.predict(oi[:, :k], w["qual"], w["ln"])
    inst = w["inst_h"]
    g_pl = torch.from_numpy(pl).to(DEV)
    events = 0
    for wt in lattices:
        gi = rb.DeviceInstances.from_host(inst, DEV)     # a copy of the batch-start state
        S0 = rb.rb_score(qh, lh, g_pl, gi, wt)
        decided = torch.empty(B, I, device=DEV)
        asg, ch = rb.rb_assign(qh, lh, g_pl, gi, wt, decided=decided)
        torch.cuda.synchronize()
        label = f"online w={tuple(round(x, 3) for x in wt)}"
        par.check_scores(S0.cpu().numpy(), g_qh, g_lh, pl, inst, wt, label=label)
        near = par.check_assign(asg.cpu().numpy(), ch.cpu().numpy(), g_qh, g_lh, pl, inst, wt,
                                g_final_p=gi.prefill_q.cpu().numpy(),
                                g_final_a=gi.decode_q.cpu().numpy(),
                                g_decided=decided.cpu().numpy(), label=label)
        free = oracle.assign(o_qh, o_lh, pl, inst, wt)
        if ties == 0 and near == 0:
            assert np.array_equal(free["assign"], asg.cpu().numpy()), label
        events += near
        # simplex corners: quality alone picks the best predicted quality,
        # cost alone the cheapest (lowest index among equals)
        if wt == (1.0, 0.0, 0.0):
            qv = g_qh[:, inst.model]
            assert np.array_equal(asg.cpu().numpy(), np.argmax(qv, axis=1)), label
        if wt == (0.0, 0.0, 1.0):
            C = pl[:, None] * inst.price_in[None, :].astype(np.float64) + \
                g_lh[:, inst.model].astype(np.float64) * inst.price_out[None, :]
            Cs = np.sort(C, axis=1)
            apart = Cs[:, 1] - Cs[:, 0] > 1e-5 * Cs[:, 1]   # no near-equal cheapest pair
            assert np.array_equal(asg.cpu().numpy()[apart], np.argmin(C, axis=1)[apart]), label
    say(f"  neighbour near-ties {ties}, pick near-ties over the sweep {events}")
