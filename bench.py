"""Benchmark of the batched routing path on one MI355X.

A step is one pass of the whole hot path over one batch: exact k-NN of the
batch's request embeddings against the reference bank, the KNN-averaged
quality and length predictions, the greedy assignment with dead-reckoned
instance state (one fused rb_route_batch call), then the carry of the state to
the next batch (rb_advance_state, 1/30 s per request). Inputs are synthetic and
already resident in HBM when the timed region starts.

Default workload: the high-load batch, B=256 requests, N=1,000,000 bank rows,
d=768 bf16 (1.5 GB), M=4 models, I=13 instances, k=10, weights (1/3,1/3,1/3),
100 consecutive batches. ``--workload`` selects another of the synthetic
workloads (tiny, online, highload, largebatch, wide). ``--options`` runs the
path through rb_route_batch_ex with any of: ``lpt`` (longest-predicted-first
order), ``inv_dist`` (inverse-distance KNN average), ``budget`` (cost budgets
on 45 % of the requests), ``mask`` (the last model's instances unavailable).

Prints one JSON line with decisions/s (value), the bank-scan bandwidth, the
roofline of the bank-scan kernel (timed with HIP events on its own stream) and
the CPU oracle's rate on a bounded sample of the same workload.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0          # MI355X HBM3E
BF16_PEAK_TFLOPS = 2500.0      # dense bf16 MFMA
FP32_PEAK_TFLOPS = 157.3


# Sources the scan kernels and their plan (chunking, passes) are built from:
# measured traffic is reported only for the build whose sources it was taken
# with.
SCAN_SOURCES = ["paper_2606_17949_amd/csrc/scan.hpp", "paper_2606_17949_amd/csrc/scan_rq.hpp",
                "paper_2606_17949_amd/csrc/scan_gemm.hpp", "paper_2606_17949_amd/csrc/knn.hip",
                "paper_2606_17949_amd/csrc/knn_common.hpp",
                "paper_2606_17949_amd/csrc/kernels.hpp", "paper_2606_17949_amd/csrc/common.hpp"]
TRAFFIC_FILE = "profiles/scan_traffic.json"
# The scan kernel is timed with HIP events on its own stream around every
# SCAN_EVENT_EVERY-th batch of the timed run (each event record adds a few
# microseconds of queue work to the stream it is recorded on).
SCAN_EVENT_EVERY = 8
# Workspaces of the pipelined schedule, used in turn.
WS_RING = 8


def scan_source_digest():
    import hashlib
    h = hashlib.sha256()
    root = os.path.dirname(os.path.abspath(__file__))
    for rel in SCAN_SOURCES:
        with open(os.path.join(root, rel), "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def _load_traffic(path):
    """The per-workload traffic records of a scan_traffic.json ({} if none)."""
    try:
        with open(path) as f:
            t = json.load(f)
    except (OSError, ValueError):
        return {}
    return t.get("workloads", {}) if isinstance(t, dict) else {}


def measured_traffic(workload):
    """HBM bytes per scan launch from the committed rocprofv3 FETCH_SIZE/WRITE_SIZE
    passes (scaled by the copy calibration), or None when they were taken on other
    sources or not for this workload."""
    root = os.path.dirname(os.path.abspath(__file__))
    t = _load_traffic(os.path.join(root, TRAFFIC_FILE)).get(workload)
    if not t or t.get("sources_sha256") != scan_source_digest():
        return None
    return t.get("bytes_per_launch")


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="highload")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--options", default="",
                    help="comma list of lpt, inv_dist, budget, mask (rb_route_batch_ex)")
    ap.add_argument("--schedule", choices=("pipelined", "sequential"), default="pipelined",
                    help="pipelined: the seed and bank scan of batch t+1 run on a second stream "
                         "while batch t is merged, averaged and assigned; sequential: one "
                         "rb_route_batch call per batch")
    ap.add_argument("--cpu-sample", type=int, default=0,
                    help="requests in the CPU oracle sample (0: 8 per host thread)")
    ap.add_argument("--record-traffic", metavar="PMC_DIR",
                    help="turn rocprofv3 FETCH_SIZE/WRITE_SIZE passes over the scan "
                         "(PMC_DIR/<workload>/fetch, PMC_DIR/<workload>/write) and over "
                         "--calibrate-copy (PMC_DIR/copyfetch, PMC_DIR/copywrite) into the "
                         "--workload record of PMC_DIR/scan_traffic.json")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="only run a plain device copy of 1 GiB (counter calibration)")
    ap.add_argument("--ceilings", action="store_true",
                    help="only measure the practical ceilings: a read-only pass over 4 GiB and "
                         "a library bf16 GEMM of the largebatch shape (yardsticks, not the path)")
    ap.add_argument("--clock-warm", type=float, default=1.0, metavar="SECONDS",
                    help="untimed batches of the measured schedule, on a copy of the instance "
                         "state (the timed batches carry the real one), for this long before "
                         "the warm-up batches, so that the timed batches run at the GPU's "
                         "sustained clock, as in a serving loop that never idles (0: none)")
    ap.add_argument("--graph", action="store_true",
                    help="sequential batches, each batch's calls (rb_route_batch, "
                         "rb_advance_state) captured beforehand in a HIP graph of its own; "
                         "times the graph launches (the host-side cost of small batches)")
    ap.add_argument("--cold", action="store_true",
                    help="time each batch alone (sequential) right after reading a 512 MiB "
                         "buffer on the same stream, so that the bank is not resident in the "
                         "last-level cache; prints the per-batch and scan-only median and p10/p90")
    return ap.parse_args()


def ceilings():
    """Practical ceilings on this device, as yardsticks for the roofline
    fractions: a read-only reduction over 4 GiB (torch) and a bf16 GEMM of the
    largebatch shape, 1,000,000 x 1,024 by 1,024 x 1,024 (torch / hipBLASLt)."""
    import torch
    dev = torch.device("cuda:0")
    out = {}
    x = torch.ones(1 << 31, dtype=torch.bfloat16, device=dev)      # 4 GiB
    for _ in range(2):
        x.sum(dtype=torch.float32)
    torch.cuda.synchronize()
    b, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    b.record()
    for _ in range(5):
        x.sum(dtype=torch.float32)
    e.record()
    torch.cuda.synchronize()
    out["read_probe_gbps"] = round(x.numel() * 2 * 5 / (b.elapsed_time(e) / 1e3) / 1e9, 1)
    del x
    bank = torch.randn(1_000_000, 1024, device=dev).to(torch.bfloat16)
    q = torch.randn(1024, 1024, device=dev).to(torch.bfloat16)
    for _ in range(2):
        torch.mm(bank, q)
    torch.cuda.synchronize()
    b.record()
    for _ in range(5):
        torch.mm(bank, q)
    e.record()
    torch.cuda.synchronize()
    flops = 2.0 * 1_000_000 * 1024 * 1024
    out["gemm_bf16_tflops"] = round(flops * 5 / (b.elapsed_time(e) / 1e3) / 1e12, 1)
    out["gemm_shape"] = "1,000,000 x 1,024 @ 1,024 x 1,024 bf16 (fp32 accumulate)"
    print(json.dumps(out), flush=True)


def calibrate_copy():
    import torch
    n = 1 << 30
    a = torch.empty(n, dtype=torch.uint8, device="cuda")
    b = torch.empty(n, dtype=torch.uint8, device="cuda")
    a.fill_(1)
    for _ in range(3):
        b.copy_(a)
    torch.cuda.synchronize()
    print(json.dumps({"calibrate_copy_bytes": n, "launches": 3}), flush=True)


def _counter_means(path, kernel_sub, counter, required=True):
    import csv
    import glob
    vals = []
    for f in glob.glob(os.path.join(path, "**", "*counter_collection.csv"), recursive=True):
        with open(f) as fh:
            for r in csv.DictReader(fh):
                if kernel_sub in r["Kernel_Name"] and r["Counter_Name"] == counter:
                    vals.append(float(r["Counter_Value"]))
    if not vals:
        if not required:
            return 0.0, 0
        raise SystemExit(f"no {counter} values for {kernel_sub} under {path}")
    return sum(vals) / len(vals), len(vals)


def record_traffic(pmc, workload):
    """Scan HBM bytes per launch: counter KiB x (bytes a 1 GiB copy moves / the
    same counter's KiB for that copy). Reads PMC/copyfetch, PMC/copywrite and
    PMC/<workload>/fetch, PMC/<workload>/write; writes PMC/scan_traffic.json,
    the records already there (else the committed ones) with this workload's
    replaced. A scan in two passes (list_bound_kernel dispatches present: the
    counters were collected for kernels matching scan_kernel|list_bound) is
    two scan-kernel dispatches and one list-bound dispatch."""
    copy_bytes = float(1 << 30)
    cf, _ = _counter_means(os.path.join(pmc, "copyfetch"), "copyBuffer", "FETCH_SIZE")
    cw, _ = _counter_means(os.path.join(pmc, "copywrite"), "copyBuffer", "WRITE_SIZE")
    sf, nf = _counter_means(os.path.join(pmc, workload, "fetch"), "scan_kernel", "FETCH_SIZE")
    sw, nw = _counter_means(os.path.join(pmc, workload, "write"), "scan_kernel", "WRITE_SIZE")
    lf, nlf = _counter_means(os.path.join(pmc, workload, "fetch"), "list_bound", "FETCH_SIZE", False)
    lw, _ = _counter_means(os.path.join(pmc, workload, "write"), "list_bound", "WRITE_SIZE", False)
    if nlf:
        sf, sw = 2 * sf + lf, 2 * sw + lw
    kf, kw = copy_bytes / cf, copy_bytes / cw     # bytes per counter unit
    rec = {"sources_sha256": scan_source_digest(),
           "fetch_size_kib": round(sf, 1), "write_size_kib": round(sw, 1), "dispatches": [nf, nw],
           "passes": 2 if nlf else 1,
           "copy_fetch_kib_per_gib": round(cf, 1), "copy_write_kib_per_gib": round(cw, 1),
           "fetch_bytes": round(sf * kf), "write_bytes": round(sw * kw),
           "bytes_per_launch": round(sf * kf + sw * kw)}
    out_path = os.path.join(pmc, "scan_traffic.json")
    recs = _load_traffic(out_path)
    if not recs:
        recs = _load_traffic(os.path.join(os.path.dirname(os.path.abspath(__file__)), TRAFFIC_FILE))
    recs[workload] = rec
    with open(out_path, "w") as f:
        json.dump({"workloads": recs}, f, indent=1, sort_keys=True)
    print(json.dumps({workload: rec}), flush=True)


def main():
    args = parse()
    if args.record_traffic:
        record_traffic(args.record_traffic, args.workload)
        return
    if args.gpus != 1:
        print(f"bench.py measures one GPU only; --gpus {args.gpus} is not supported "
              "(the bank-sharded multi-GPU design is described in DESIGN.md).", file=sys.stderr)
        sys.exit(2)
    if args.calibrate_copy:
        calibrate_copy()
        return
    if args.ceilings:
        ceilings()
        return

    import numpy as np
    import torch

    import paper_2606_17949_amd as rb
    import synth

    cfg = synth.CONFIGS[args.workload]
    opt_names = [o for o in args.options.split(",") if o]
    bad = set(opt_names) - {"lpt", "inv_dist", "budget", "mask"}
    if bad:
        raise SystemExit(f"unknown --options {sorted(bad)}")
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    K, W = args.steps, args.warmup
    nb = K + W
    log(f"workload {cfg.name}: B={cfg.B} N={cfg.N} d={cfg.d} {cfg.dtype} M={cfg.M} I={cfg.I} "
        f"k={cfg.k}, {W} warm-up + {K} timed batches")

    t0 = time.time()
    centres = synth.make_centres(cfg, dev)
    bank = synth.make_bank(cfg, dev, centres)
    queries = [synth.make_queries(cfg, t, dev, centres) for t in range(nb)]
    qual, length = synth.make_labels(cfg)
    plens = [torch.from_numpy(synth.make_prompt_lens(cfg, t)).to(dev) for t in range(nb)]
    inst_h = synth.make_instances(cfg)
    g_qual = torch.from_numpy(qual).to(dev)
    g_len = torch.from_numpy(length).to(dev)
    inst = rb.DeviceInstances.from_host(inst_h, dev)
    norms = rb.rb_bank_norms(bank)
    dt_code = rb.RB_BF16 if cfg.dtype == "bf16" else rb.RB_F32
    ws = rb.workspace(cfg.B, cfg.N, cfg.d, dt_code, cfg.k, cfg.M, dev)
    assign = torch.empty(nb, cfg.B, dtype=torch.int32, device=dev)
    carry_dt = cfg.B / 30.0
    budgets = [torch.from_numpy(synth.make_budgets(cfg, t)).to(dev) if "budget" in opt_names
               else None for t in range(nb)]
    mask_h = synth.make_availability(cfg, lost_models=(cfg.M - 1,)) if "mask" in opt_names \
        else None
    mask = None if mask_h is None else torch.from_numpy(mask_h).to(dev)
    opts = [rb.options(order=rb.RB_ORDER_LPT if "lpt" in opt_names else rb.RB_ORDER_ARRIVAL,
                       weighting=rb.RB_KNN_INV_DIST if "inv_dist" in opt_names
                       else rb.RB_KNN_UNIFORM, budget=budgets[t], instance_mask=mask)
            for t in range(nb)] if opt_names else None
    torch.cuda.synchronize()
    log(f"inputs resident in HBM ({time.time() - t0:.1f}s); bank {cfg.bank_bytes() / 1e9:.3f} GB")

    stream = torch.cuda.current_stream()
    ev_b = [torch.cuda.Event(enable_timing=True) for _ in range(K)]
    ev_e = [torch.cuda.Event(enable_timing=True) for _ in range(K)]
    for ev in ev_b + ev_e:      # torch creates the HIP event on first record
        ev.record(stream)

    def step(t, state=None, out=None):
        state = inst if state is None else state
        out = assign[t] if out is None else out
        if opts is None:
            rb.rb_route_batch(queries[t], bank, norms, cfg.k, g_qual, g_len, plens[t], state,
                              cfg.weights, ws=ws, assign=out, stream=stream)
        else:
            rb.rb_route_batch_ex(queries[t], bank, norms, cfg.k, g_qual, g_len, plens[t], state,
                                 cfg.weights, opts[t], ws=ws, assign=out, stream=stream)
        rb.rb_advance_state(state, carry_dt, stream=stream)

    # pipelined schedule: the first half of each lookup (seed and bank scan,
    # RB_FLAG_LISTS_ONLY) on s_knn; the second half (merge of the chunk lists
    # and label average, RB_FLAG_FROM_LISTS), the greedy pass and the carry in
    # batch order on s_asg, after an event on the first half. A ring of
    # WS_RING workspaces: a lookup waits for the merge WS_RING batches back,
    # which last read its workspace. The greedy stream keeps a few hundred
    # microseconds of slack per batch, but a merge that finds every compute
    # unit taken by the next scan waits for the few units the scan leaves
    # free, so the ring is deep enough that such a late merge never holds up
    # a lookup.
    s_knn = torch.cuda.Stream(device=dev)
    s_asg = torch.cuda.Stream(device=dev) if args.schedule == "pipelined" else stream
    n_ws = WS_RING if args.schedule == "pipelined" else 1
    wss = [ws] + [rb.workspace(cfg.B, cfg.N, cfg.d, dt_code, cfg.k, cfg.M, dev)
                  for _ in range(n_ws - 1)]
    qh = torch.empty(cfg.B, cfg.M, device=dev)
    lh = torch.empty(cfg.B, cfg.M, device=dev)
    order_buf = torch.empty(cfg.B, dtype=torch.int32, device=dev)
    wmode = rb.RB_KNN_INV_DIST if "inv_dist" in opt_names else rb.RB_KNN_UNIFORM
    lists_opts = rb.options(weighting=wmode, flags=rb.RB_FLAG_OVERLAP | rb.RB_FLAG_LISTS_ONLY)
    merge_opts = rb.options(weighting=wmode, flags=rb.RB_FLAG_OVERLAP | rb.RB_FLAG_FROM_LISTS)
    lpt = "lpt" in opt_names
    asg_opts = [rb.options(order=rb.RB_ORDER_LPT if lpt else rb.RB_ORDER_ARRIVAL,
                           budget=budgets[t], instance_mask=mask,
                           order_out=order_buf if lpt else None)
                for t in range(nb)]
    ev_knn = [torch.cuda.Event() for _ in range(nb)]
    ev_mrg = [torch.cuda.Event() for _ in range(nb)]

    def lookup(t, ek=ev_knn, em=ev_mrg, i=None):
        """Lookup of batch t's inputs as the i-th batch of its run (default
        i = t); the event lists are indexed modulo their length (a ring longer
        than the workspace ring keeps every event it waits for unrecorded
        until that wait is enqueued)."""
        i = t if i is None else i
        if i >= n_ws:
            s_knn.wait_event(em[(i - n_ws) % len(em)])
        rb.rb_knn_predict(queries[t], bank, norms, cfg.k, g_qual, g_len, lists_opts,
                          ws=wss[i % n_ws], stream=s_knn)
        ek[i % len(ek)].record(s_knn)

    def decide(t, ek=ev_knn, em=ev_mrg, i=None, state=None, out=None):
        i = t if i is None else i
        state = inst if state is None else state
        out = assign[t] if out is None else out
        s_asg.wait_event(ek[i % len(ek)])
        rb.rb_knn_predict(queries[t], bank, norms, cfg.k, g_qual, g_len, merge_opts,
                          ws=wss[i % n_ws], q_hat=qh, l_hat=lh, stream=s_asg)
        em[i % len(em)].record(s_asg)
        rb.rb_assign_ex(qh, lh, plens[t], state, cfg.weights, asg_opts[t],
                        assign=out, stream=s_asg, want_chosen=False)
        rb.rb_advance_state(state, carry_dt, stream=s_asg)

    def scan_events(j, timed):
        """Scan events j around the j-th batch's scan if it is a sampled one."""
        if timed and j % SCAN_EVENT_EVERY == 0:
            rb.rb_profile_scan_events(ev_b[j], ev_e[j])
        else:
            rb.rb_profile_scan_events(None, None)

    def run(ts, timed=False):
        """Batches ts in order; with `timed`, the scans of every
        SCAN_EVENT_EVERY-th batch are bracketed by HIP events."""
        if args.schedule == "sequential":
            for j, t in enumerate(ts):
                scan_events(j, timed)
                step(t)
        else:
            for j, t in enumerate(ts):
                if j == 0:
                    scan_events(0, timed)
                    lookup(t)
                if j + 1 < len(ts):
                    scan_events(j + 1, timed)
                    lookup(ts[j + 1])
                decide(t)
        rb.rb_profile_scan_events(None, None)

    if args.clock_warm > 0:
        # The GPU settles its clock to the load it runs: after a stretch of
        # lookups alone the batches that followed ran slower than their steady
        # state for about 50 batches (measured with every scan timed: the
        # high-load scan from 450 to 380 us), after a stretch of the batch
        # schedule itself at 390-400 us from the first one. So this untimed
        # warm-up runs the schedule being measured, on a copy of the instance
        # state (the timed batches carry the real one), cycling over the
        # batches' inputs, as one unbroken stretch (no host synchronisation).
        state_w = inst.clone()
        out_w = torch.empty(cfg.B, dtype=torch.int32, device=dev)
        ek = [torch.cuda.Event() for _ in range(2 * n_ws)]
        em = [torch.cuda.Event() for _ in range(2 * n_ws)]

        def warm(n):
            if args.schedule == "sequential":
                for i in range(n):
                    step(i % nb, state_w, out_w)
                return
            for i in range(n):
                lookup(i % nb, ek, em, i)
                if i >= 1:
                    decide((i - 1) % nb, ek, em, i - 1, state_w, out_w)
            decide((n - 1) % nb, ek, em, n - 1, state_w, out_w)
        warm(2)
        torch.cuda.synchronize()
        t_w = time.perf_counter()
        warm(8)
        torch.cuda.synchronize()
        per = (time.perf_counter() - t_w) / 8
        n_w = max(1, int(args.clock_warm / per))
        t_w = time.perf_counter()
        warm(n_w)
        torch.cuda.synchronize()
        log(f"clock warm-up: {n_w} untimed batches in {time.perf_counter() - t_w:.2f} s")
    run(list(range(W)))
    torch.cuda.synchronize()
    log("warm-up done")

    if args.cold:
        # each batch alone, after a 512 MiB write that evicts the bank from
        # the last-level cache (untimed); sequential fused calls
        # the flush READS a 512 MiB buffer (twice the last-level cache), so
        # that it evicts the bank without leaving dirty lines whose write-back
        # would compete with the timed batch's reads; it is enqueued on the
        # batch's own stream right before it, with no host synchronisation in
        # between
        flush = torch.ones(128 << 20, dtype=torch.float32, device=dev)
        times, scans = [], []
        for j in range(K):
            torch.cuda.synchronize()
            with torch.cuda.stream(stream):
                flush.sum()
            b0, b1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            rb.rb_profile_scan_events(ev_b[j], ev_e[j])
            b0.record(stream)
            step(W + j)
            b1.record(stream)
            torch.cuda.synchronize()
            rb.rb_profile_scan_events(None, None)
            times.append(b0.elapsed_time(b1))
            scans.append(ev_b[j].elapsed_time(ev_e[j]))
        med = float(np.median(times))
        smed = float(np.median(scans))

        def pct(v, q):
            return round(float(np.percentile(v, q)), 4)
        print(json.dumps({"metric": "routing decisions/sec, cold bank (per batch, median)",
                          "value": round(cfg.B / (med / 1e3), 1), "unit": "decisions/s",
                          "workload": cfg.name, "batches": K,
                          "ms_per_batch": {"median": round(med, 4), "p10": pct(times, 10),
                                           "p90": pct(times, 90)},
                          "bank_gbps_at_median": round(cfg.bank_bytes() / (med / 1e3) / 1e9, 1),
                          "scan_us": {"median": round(smed * 1e3, 2),
                                      "p10": round(pct(scans, 10) * 1e3, 2),
                                      "p90": round(pct(scans, 90) * 1e3, 2)},
                          "scan_bank_gbps_at_median": round(cfg.bank_bytes() / (smed / 1e3) / 1e9,
                                                            1),
                          "scan_frac_of_8tbs": round(cfg.bank_bytes() / (smed / 1e3) / 1e9 /
                                                     HBM_PEAK_GBS, 4)}),
              flush=True)
        return

    if args.graph:
        if args.schedule != "sequential" or opts is not None:
            raise SystemExit("--graph captures the sequential schedule without --options")
        # the timed batches' calls, one graph per batch (kernel nodes only:
        # the library enqueues no memset or copy)
        cap = torch.cuda.Stream(device=dev)
        graphs = {}
        torch.cuda.synchronize()
        for t in range(W, W + K):
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g, stream=cap, capture_error_mode="thread_local"):
                rb.rb_route_batch(queries[t], bank, norms, cfg.k, g_qual, g_len, plens[t], inst,
                                  cfg.weights, ws=ws, assign=assign[t], stream=cap)
                rb.rb_advance_state(inst, carry_dt, stream=cap)
            graphs[t] = g
        torch.cuda.synchronize()
        b0, b1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        b0.record(stream)
        w0 = time.perf_counter()
        for t in range(W, W + K):
            graphs[t].replay()
        b1.record(stream)
        torch.cuda.synchronize()
        wall = time.perf_counter() - w0
        ms = b0.elapsed_time(b1) / K
        print(json.dumps({"metric": "routing decisions/sec, sequential batches as HIP graphs",
                          "value": round(cfg.B / (ms / 1e3), 1), "unit": "decisions/s",
                          "workload": cfg.name, "batches": K, "ms_per_batch": round(ms, 4),
                          "host_us_per_batch": round(wall / K * 1e6, 1)}), flush=True)
        return

    start = torch.cuda.Event(enable_timing=True)
    end = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    start.record(s_asg)
    s_knn.wait_event(start)
    w0 = time.perf_counter()
    run(list(range(W, W + K)), timed=True)
    end.record(s_asg)
    torch.cuda.synchronize()
    wall = time.perf_counter() - w0
    total_ms = start.elapsed_time(end)
    scan_ms = [ev_b[j].elapsed_time(ev_e[j]) for j in range(0, K, SCAN_EVENT_EVERY)]
    scan_avg = float(np.mean(scan_ms))
    log(f"timed {K} batches: {total_ms:.3f} ms (events), {wall * 1e3:.3f} ms (host wall); "
        f"scan kernel avg {scan_avg * 1e3:.1f} us")

    ms_per_step = total_ms / K
    decisions = cfg.B * K / (total_ms / 1e3)
    bank_bytes = cfg.bank_bytes()
    scan_gbs = bank_bytes / (scan_avg / 1e3) / 1e9
    flops = 2.0 * cfg.B * cfg.N * cfg.d
    ai = flops / bank_bytes
    peak_tf = BF16_PEAK_TFLOPS if cfg.dtype == "bf16" else FP32_PEAK_TFLOPS
    ridge = peak_tf * 1e12 / (HBM_PEAK_GBS * 1e9)
    if ai < ridge:
        roof = {"bound": "hbm", "achieved": round(scan_gbs, 1), "peak": HBM_PEAK_GBS,
                "unit": "GB/s", "frac": round(scan_gbs / HBM_PEAK_GBS, 4),
                "traffic": measured_traffic(cfg.name)}
    else:
        tf = flops / (scan_avg / 1e3) / 1e12
        roof = {"bound": "mfma", "achieved": round(tf, 1), "peak": peak_tf, "unit": "TFLOP/s",
                "frac": round(tf / peak_tf, 4), "traffic": measured_traffic(cfg.name)}
    roof["kernel"] = ("bank scan, scan_kernel or rq_scan_kernel (distance contraction + fused "
                      "per-chunk top-k)")
    roof["per_launch"] = {"bytes": bank_bytes, "flops": flops, "launches_timed": len(scan_ms),
                          "avg_us": round(scan_avg * 1e3, 2),
                          "p10_us": round(float(np.percentile(scan_ms, 10)) * 1e3, 2),
                          "p90_us": round(float(np.percentile(scan_ms, 90)) * 1e3, 2)}
    roof["mfma_tflops"] = round(flops / (scan_avg / 1e3) / 1e12, 1)

    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(cfg, bank, queries[W], qual, length, plens[W].cpu().numpy(), inst_h,
                           args.cpu_sample, opt_names,
                           None if budgets[W] is None else budgets[W].cpu().numpy(), mask_h)

    out = {
        "metric": "routing decisions/sec + bank-scan HBM GB/s (B=256, N=1M, d=768)",
        "value": round(decisions, 1),
        "unit": "decisions/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": W,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": cfg.dtype,
        "data": "synthetic (seeded Gaussian-mixture embeddings, Beta/LogNormal labels)",
        "config": {"workload": f"{cfg.name}: B={cfg.B} N={cfg.N} d={cfg.d} {cfg.dtype} bank, "
                               f"M={cfg.M} I={cfg.I} k={cfg.k}, {K} carried batches",
                   "B": cfg.B, "N": cfg.N, "d": cfg.d, "k": cfg.k, "M": cfg.M, "I": cfg.I,
                   "weights": [round(w, 6) for w in cfg.weights], "carry_dt_s": round(carry_dt, 6),
                   "parallelism": "single GPU"},
        "options": opt_names,
        "schedule": args.schedule if args.schedule == "sequential" else
        "pipelined: the seed and bank scan of batch t+1 (second stream) overlap the merge, "
        "greedy pass and carry of batch t; every batch's lookup, greedy pass and carry are "
        "inside the timed region",
        "bank_scan_gbps": round(scan_gbs, 1),
        "arith_intensity_flop_per_byte": round(ai, 1),
        "roofline": roof,
        "cpu_baseline": cpu,
    }
    print(json.dumps(out), flush=True)


def cpu_model():
    """The host CPU's model name (Linux /proc/cpuinfo), or None."""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return None


def cpu_baseline(cfg, bank, queries, qual, length, plen, inst_h, sample, opt_names=(),
                 budget=None, mask=None):
    """The oracle as it stands on a bounded sample: the first S requests of the
    first timed batch, full k-NN over the whole bank, predictions and the greedy
    assignment (with the same options), on all host threads available to this
    process; for the two small workloads also on one thread."""
    import numpy as np

    import oracle
    threads = len(os.sched_getaffinity(0))
    S = min(cfg.B, sample if sample > 0 else 16 * threads)
    log(f"cpu baseline: oracle on {S} requests, {threads} threads ...")
    bank_h = bank.cpu()
    q_h = queries[:S].cpu()

    def run(nthreads):
        t0 = time.perf_counter()
        idx, dist = oracle.knn(q_h, bank_h, cfg.k, nthreads=nthreads)
        qh, lh = oracle.predict(idx, qual, length, dist=dist,
                                weighting="inv_dist" if "inv_dist" in opt_names else "uniform")
        oracle.assign(qh, lh, plen[:S], inst_h, cfg.weights,
                      order="lpt" if "lpt" in opt_names else "arrival",
                      budget=None if budget is None else budget[:S], mask=mask)
        return time.perf_counter() - t0

    dt = run(threads)
    log(f"cpu baseline: {dt:.1f}s")
    out = {"value": round(S / dt, 3), "unit": "decisions/s", "cores": threads, "kind": "oracle",
           "sample": f"first {S} requests of one {cfg.B}-request batch: exact fp64 k-NN over "
                     f"all {cfg.N} bank rows, predictions, greedy assignment ({dt:.1f} s)",
           "cpu_model": cpu_model()}
    if S == cfg.B:
        out["s_per_batch"] = round(dt, 3)
    if cfg.name in ("tiny", "online"):
        d1 = run(1)
        log(f"cpu baseline, one thread: {d1:.1f}s")
        out["single_thread"] = {"value": round(S / d1, 3), "unit": "decisions/s",
                                "s_for_sample": round(d1, 3)}
    return out


if __name__ == "__main__":
    main()
