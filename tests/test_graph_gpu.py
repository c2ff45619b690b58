"""One batch of the fused path (rb_route_batch, then rb_advance_state)
captured in a HIP graph: every replay, with eager work and host
synchronisations between replays, gives the assignment and the carried
instance state that the same calls give eagerly. The path enqueues kernels
only (no memset or copy nodes), so callers may capture it."""
import numpy as np
import pytest
import torch

import synth

pytestmark = pytest.mark.gpu

DEV = "cuda"


def say(msg):
    print(msg, flush=True)


@pytest.mark.parametrize("name", ["online", "tiny"])
def test_route_batch_graph_replays_match_eager(name):
    import paper_2606_17949_amd as rb
    cfg = synth.CONFIGS[name]
    say(f"graph {name}: B={cfg.B} N={cfg.N} d={cfg.d} {cfg.dtype}")
    centres = synth.make_centres(cfg, DEV)
    bank = synth.make_bank(cfg, DEV, centres)
    norms = rb.rb_bank_norms(bank)
    qual, ln = synth.make_labels(cfg)
    gq, gl = torch.from_numpy(qual).to(DEV), torch.from_numpy(ln).to(DEV)
    inst_h = synth.make_instances(cfg)
    nb = 4
    queries = [synth.make_queries(cfg, t, DEV, centres) for t in range(nb)]
    plens = [torch.from_numpy(synth.make_prompt_lens(cfg, t)).to(DEV) for t in range(nb)]
    dt = cfg.B / 30.0
    code = rb._dtype_code(bank)
    inst_e = rb.DeviceInstances.from_host(inst_h, DEV)
    inst_g = inst_e.clone()
    ws_e = rb.workspace(cfg.B, cfg.N, cfg.d, code, cfg.k, cfg.M, DEV)
    ws_g = rb.workspace(cfg.B, cfg.N, cfg.d, code, cfg.k, cfg.M, DEV)
    q_s = torch.empty_like(queries[0])
    pl_s = torch.empty_like(plens[0])
    a_g = torch.empty(cfg.B, dtype=torch.int32, device=DEV)
    a_e = torch.empty(cfg.B, dtype=torch.int32, device=DEV)
    # one eager call on a throwaway state first (lazy per-process set-up)
    rb.rb_route_batch(queries[0], bank, norms, cfg.k, gq, gl, plens[0], inst_e.clone(),
                      cfg.weights, ws=ws_g, assign=a_g)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    cap = torch.cuda.Stream()
    with torch.cuda.graph(g, stream=cap, capture_error_mode="thread_local"):
        rb.rb_route_batch(q_s, bank, norms, cfg.k, gq, gl, pl_s, inst_g, cfg.weights, ws=ws_g,
                          assign=a_g, stream=cap)
        rb.rb_advance_state(inst_g, dt, stream=cap)
    torch.cuda.synchronize()
    for t in range(nb):
        q_s.copy_(queries[t])
        pl_s.copy_(plens[t])
        a_g.fill_(-7)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        rb.rb_route_batch(queries[t], bank, norms, cfg.k, gq, gl, plens[t], inst_e, cfg.weights,
                          ws=ws_e, assign=a_e)
        rb.rb_advance_state(inst_e, dt)
        torch.cuda.synchronize()
        ge, gg = a_e.cpu().numpy(), a_g.cpu().numpy()
        say(f"  batch {t}: {int(np.sum(ge == gg))}/{cfg.B} assignments equal")
        assert np.array_equal(ge, gg), f"batch {t}: graph replay differs from eager"
        for f in ("prefill_q", "decode_q"):
            assert torch.equal(getattr(inst_e, f), getattr(inst_g, f)), f"batch {t}: {f}"
