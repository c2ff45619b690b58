"""The split path (rb_knn_predict, then rb_assign_ex) and the pipelined
schedule that overlaps the lookup of batch t+1 with the greedy pass of batch t
give exactly the results of one rb_route_batch call per batch."""
import numpy as np
import pytest
import torch

import synth

pytestmark = pytest.mark.gpu

DEV = "cuda"


def say(msg):
    print(msg, flush=True)


def setup(cfg):
    import paper_2606_17949_amd as rb
    centres = synth.make_centres(cfg, DEV)
    bank = synth.make_bank(cfg, DEV, centres)
    qual, ln = synth.make_labels(cfg)
    return dict(rb=rb, centres=centres, bank=bank, norms=rb.rb_bank_norms(bank),
                gq=torch.from_numpy(qual).to(DEV), gl=torch.from_numpy(ln).to(DEV),
                inst_h=synth.make_instances(cfg))


@pytest.mark.parametrize("name,over", [
    ("tiny-bf16", dict(dtype="bf16", d=768, N=20000, B=64, clusters=256)),
    ("tiny-f32-multi-tile", dict(B=600, N=30000, d=384)),
])
def test_knn_predict_overlap_flag_changes_nothing(name, over):
    cfg = synth.tiny_config(**over)
    say(f"knn_predict {name}: B={cfg.B} N={cfg.N} d={cfg.d} {cfg.dtype}")
    c = setup(cfg)
    rb = c["rb"]
    q = synth.make_queries(cfg, 0, DEV, c["centres"])
    outs = []
    for flags in (0, rb.RB_FLAG_OVERLAP):
        for wt in (rb.RB_KNN_UNIFORM, rb.RB_KNN_INV_DIST):
            idx = torch.empty(cfg.B, cfg.k, dtype=torch.int32, device=DEV)
            dist = torch.empty(cfg.B, cfg.k, device=DEV)
            qh, lh = rb.rb_knn_predict(q, c["bank"], c["norms"], cfg.k, c["gq"], c["gl"],
                                       rb.options(weighting=wt, flags=flags), nbr_idx=idx,
                                       nbr_dist=dist)
            torch.cuda.synchronize()
            outs.append((flags, wt, idx.cpu().numpy(), dist.cpu().numpy(), qh.cpu().numpy(),
                         lh.cpu().numpy()))
            # the same lookup in two calls on two streams: the scan half, an
            # event, the merge half
            s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
            ws = rb.workspace(cfg.B, cfg.N, cfg.d, rb._dtype_code(c["bank"]), cfg.k, cfg.M, DEV)
            ev = torch.cuda.Event()
            torch.cuda.synchronize()
            rb.rb_knn_predict(q, c["bank"], c["norms"], cfg.k, c["gq"], c["gl"],
                              rb.options(weighting=wt, flags=flags | rb.RB_FLAG_LISTS_ONLY),
                              ws=ws, stream=s1)
            ev.record(s1)
            s2.wait_event(ev)
            idx = torch.empty(cfg.B, cfg.k, dtype=torch.int32, device=DEV)
            dist = torch.empty(cfg.B, cfg.k, device=DEV)
            qh, lh = rb.rb_knn_predict(q, c["bank"], c["norms"], cfg.k, c["gq"], c["gl"],
                                       rb.options(weighting=wt,
                                                  flags=flags | rb.RB_FLAG_FROM_LISTS),
                                       ws=ws, nbr_idx=idx, nbr_dist=dist, stream=s2)
            torch.cuda.synchronize()
            outs.append((flags, wt, idx.cpu().numpy(), dist.cpu().numpy(), qh.cpu().numpy(),
                         lh.cpu().numpy()))
    # the fused route call's own lists and predictions
    gi = rb.DeviceInstances.from_host(c["inst_h"], DEV)
    idx = torch.empty(cfg.B, cfg.k, dtype=torch.int32, device=DEV)
    qh = torch.empty(cfg.B, cfg.M, device=DEV)
    lh = torch.empty(cfg.B, cfg.M, device=DEV)
    rb.rb_route_batch(q, c["bank"], c["norms"], cfg.k, c["gq"], c["gl"],
                      torch.from_numpy(synth.make_prompt_lens(cfg)).to(DEV), gi, cfg.weights,
                      nbr_idx=idx, q_hat=qh, l_hat=lh)
    torch.cuda.synchronize()
    for flags, wt, i, d, a, b in outs:
        ref = [o for o in outs if o[0] == 0 and o[1] == wt][0]
        for x, y in zip((i, d, a, b), ref[2:]):
            assert np.array_equal(x.view(np.uint8), y.view(np.uint8)), (flags, wt)
        if wt == rb.RB_KNN_UNIFORM:
            assert np.array_equal(i, idx.cpu().numpy())
            assert np.array_equal(a.view(np.uint32), qh.cpu().numpy().view(np.uint32))
            assert np.array_equal(b.view(np.uint32), lh.cpu().numpy().view(np.uint32))


@pytest.mark.parametrize("name,batches,split", [("online", 5, False), ("highload", 4, False),
                                                ("online", 5, True), ("highload", 4, True)])
def test_pipelined_schedule_matches_sequential(name, batches, split):
    """split: the scan half of every lookup on one stream, the merge half with
    the greedy pass on the other, each batch with its own workspace."""
    cfg = synth.CONFIGS[name]
    say(f"pipeline {name}: B={cfg.B} N={cfg.N}, {batches} carried batches, split={split}")
    c = setup(cfg)
    rb = c["rb"]
    qs = [synth.make_queries(cfg, t, DEV, c["centres"]) for t in range(batches)]
    pls = [torch.from_numpy(synth.make_prompt_lens(cfg, t)).to(DEV) for t in range(batches)]
    dt = cfg.B / 30.0
    ws = rb.workspace(cfg.B, cfg.N, cfg.d, rb.RB_BF16, cfg.k, cfg.M, DEV)

    # sequential: one fused call per batch, then the carry
    gi = rb.DeviceInstances.from_host(c["inst_h"], DEV)
    seq = []
    for t in range(batches):
        a = rb.rb_route_batch(qs[t], c["bank"], c["norms"], cfg.k, c["gq"], c["gl"], pls[t], gi,
                              cfg.weights, ws=ws)
        rb.rb_advance_state(gi, dt)
        seq.append(a)
    torch.cuda.synchronize()
    seq_state = (gi.prefill_q.cpu().numpy(), gi.decode_q.cpu().numpy())

    # pipelined: lookups on one stream (overlap flag), greedy passes on another
    gi = rb.DeviceInstances.from_host(c["inst_h"], DEV)
    s_knn, s_asg = torch.cuda.Stream(), torch.cuda.Stream()
    torch.cuda.synchronize()
    qh = [torch.empty(cfg.B, cfg.M, device=DEV) for _ in range(2)]
    lh = [torch.empty(cfg.B, cfg.M, device=DEV) for _ in range(2)]
    ev_k = [torch.cuda.Event() for _ in range(batches)]
    ev_a = [torch.cuda.Event() for _ in range(batches)]
    kopt = rb.options(flags=rb.RB_FLAG_OVERLAP)
    aopt = rb.options()
    pip = []

    def lookup(t):
        if t >= 2:
            s_knn.wait_event(ev_a[t - 2])
        rb.rb_knn_predict(qs[t], c["bank"], c["norms"], cfg.k, c["gq"], c["gl"], kopt, ws=ws,
                          q_hat=qh[t % 2], l_hat=lh[t % 2], stream=s_knn)
        ev_k[t].record(s_knn)

    if split:
        wss = [rb.workspace(cfg.B, cfg.N, cfg.d, rb.RB_BF16, cfg.k, cfg.M, DEV)
               for _ in range(batches)]
        lopt = rb.options(flags=rb.RB_FLAG_OVERLAP | rb.RB_FLAG_LISTS_ONLY)
        mopt = rb.options(flags=rb.RB_FLAG_OVERLAP | rb.RB_FLAG_FROM_LISTS)

        def lookup(t):
            rb.rb_knn_predict(qs[t], c["bank"], c["norms"], cfg.k, c["gq"], c["gl"], lopt,
                              ws=wss[t], stream=s_knn)
            ev_k[t].record(s_knn)

    lookup(0)
    for t in range(batches):
        if t + 1 < batches:
            lookup(t + 1)
        s_asg.wait_event(ev_k[t])
        if split:
            rb.rb_knn_predict(qs[t], c["bank"], c["norms"], cfg.k, c["gq"], c["gl"], mopt,
                              ws=wss[t], q_hat=qh[t % 2], l_hat=lh[t % 2], stream=s_asg)
        a, _ = rb.rb_assign_ex(qh[t % 2], lh[t % 2], pls[t], gi, cfg.weights, aopt,
                               stream=s_asg, want_chosen=False)
        rb.rb_advance_state(gi, dt, stream=s_asg)
        ev_a[t].record(s_asg)
        pip.append(a)
    torch.cuda.synchronize()
    for t in range(batches):
        assert np.array_equal(seq[t].cpu().numpy(), pip[t].cpu().numpy()), t
    assert np.array_equal(seq_state[0].view(np.uint32), gi.prefill_q.cpu().numpy().view(np.uint32))
    assert np.array_equal(seq_state[1].view(np.uint32), gi.decode_q.cpu().numpy().view(np.uint32))
