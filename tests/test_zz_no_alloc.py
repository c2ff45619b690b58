"""rb_route_batch_noalloc against rb_route_batch (GPU).

The no-allocation entry point runs the same kernels on the library's static
per-GPU workspace instead of a caller's. Its results must be those of
rb_route_batch on the same inputs, bit for bit: two calls in a row, the
second on a smaller batch (the static array keeps the first call's contents,
none of which may leak into the second), then a third on the query-resident
scan, and sizes past the static maximum must be refused before anything runs.
"""
import numpy as np
import pytest
import torch

import synth

pytestmark = pytest.mark.gpu

DEV = "cuda"


def say(msg):
    print(msg, flush=True)


def inputs(cfg):
    centres = synth.make_centres(cfg, DEV)
    bank = synth.make_bank(cfg, DEV, centres)
    q = synth.make_queries(cfg, 0, DEV, centres)
    qual, ln = synth.make_labels(cfg)
    return dict(bank=bank, q=q, qual=torch.from_numpy(qual).to(DEV),
                ln=torch.from_numpy(ln).to(DEV),
                pl=torch.from_numpy(synth.make_prompt_lens(cfg)).to(DEV),
                inst=synth.make_instances(cfg))


def run(rb, cfg, x, noalloc):
    B, k, M, I = cfg.B, cfg.k, cfg.M, cfg.I
    norms = rb.rb_bank_norms(x["bank"])
    gi = rb.DeviceInstances.from_host(x["inst"], DEV)
    out = dict(assign=torch.full((B,), -5, dtype=torch.int32, device=DEV),
               chosen=torch.empty(B, device=DEV),
               nbr_idx=torch.empty(B, k, dtype=torch.int32, device=DEV),
               nbr_dist=torch.empty(B, k, device=DEV), q_hat=torch.empty(B, M, device=DEV),
               l_hat=torch.empty(B, M, device=DEV), score0=torch.empty(B, I, device=DEV))
    fn = rb.rb_route_batch_noalloc if noalloc else rb.rb_route_batch
    fn(x["q"], x["bank"], norms, k, x["qual"], x["ln"], x["pl"], gi, cfg.weights, **out)
    torch.cuda.synchronize()
    res = {n: t.cpu().numpy() for n, t in out.items()}
    res["p"] = gi.prefill_q.cpu().numpy()
    res["a"] = gi.decode_q.cpu().numpy()
    return res


def same(a, b, label):
    for n in a:
        assert np.array_equal(a[n].view(np.uint8), b[n].view(np.uint8)), f"{label}: {n} differs"


def test_noalloc_matches_route_batch():
    import paper_2606_17949_amd as rb
    cases = [
        ("online batch", synth.CONFIGS["online"]),
        ("smaller fp32 batch", synth.CONFIGS["tiny"]),
        ("query-resident scan", synth.tiny_config(B=200, N=200_000, d=768, dtype="bf16",
                                                 clusters=1024)),
        # more than 128 requests over more than 32 x 32,768 rows: two passes
        ("query-resident scan in two passes",
         synth.tiny_config(B=160, N=1_100_000, d=384, dtype="bf16", clusters=1024)),
    ]
    for label, cfg in cases:
        say(f"noalloc {label}: B={cfg.B} N={cfg.N} d={cfg.d} {cfg.dtype}, "
            f"workspace {rb.rb_workspace_size(cfg.B, cfg.N, cfg.d, rb.RB_BF16 if cfg.dtype == 'bf16' else rb.RB_F32, cfg.k, cfg.M) / 2**20:.1f} MiB")
        x = inputs(cfg)
        got = run(rb, cfg, x, noalloc=True)
        ref = run(rb, cfg, x, noalloc=False)
        same(got, ref, label)
        assert np.all(got["assign"] >= 0)


def test_noalloc_refuses_sizes_past_its_workspace():
    import paper_2606_17949_amd as rb
    # (a batch of 1024 requests of 384 elements goes to the GEMM-structured
    # scan, whose per-wave overflow areas alone exceed the static workspace)
    cfg = synth.tiny_config(B=1024, N=100_000, d=384, dtype="bf16", clusters=256)
    need = rb.rb_workspace_size(cfg.B, cfg.N, cfg.d, rb.RB_BF16, cfg.k, cfg.M)
    say(f"noalloc refusal: B={cfg.B} needs {need / 2**20:.1f} MiB of {rb.RB_SCRATCH_BYTES >> 20}")
    assert need > rb.RB_SCRATCH_BYTES
    x = inputs(cfg)
    norms = rb.rb_bank_norms(x["bank"])
    gi = rb.DeviceInstances.from_host(x["inst"], DEV)
    assign = torch.full((cfg.B,), -5, dtype=torch.int32, device=DEV)
    with pytest.raises(rb.RbError) as e:
        rb.rb_route_batch_noalloc(x["q"], x["bank"], norms, cfg.k, x["qual"], x["ln"], x["pl"],
                                  gi, cfg.weights, assign=assign)
    assert e.value.status == rb.RB_ERR_SCRATCH
    torch.cuda.synchronize()
    assert torch.all(assign == -5)
    assert np.array_equal(gi.prefill_q.cpu().numpy(), x["inst"].prefill_q)
