"""Benchmark of one SAME Gibbs pass on one MI355X.

Workload (default): the 1000-node random DAG, 2,000,000 columns in eight
250,000-column minibatches, 40% of entries hidden, m = 10 SAME replicas; all
minibatches resident in HBM (20 GB of int8 states + 2 GB of obs masks) when
timing starts.  One step = one pass over all minibatches; per minibatch the
library runs the colour-group sweep, the counts with their exact moving sum
and the Dirichlet resample of every CPT row (the whole hot path).

Prints one JSON line: node-samples/s (every (node, column, replica) slot of a
pass), the sweep kernels' roofline figures measured with HIP events on the
launch stream, and the oracle's rate on a bounded sample of the same workload
timed on the host cores.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
METRIC = "Gibbs node-samples/sec (incl. SAME replicas) + achieved HBM GB/s, 1 GPU"


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=3)
    p.add_argument("--warmup", type=int, default=1)
    p.add_argument("--cfg", type=int, default=5)
    p.add_argument("--n-cols", type=int, default=None, help="override the column count")
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--cpu-sample-cols", type=int, default=32768)
    p.add_argument("--copy-calibration", action="store_true",
                   help="also run a plain 1 GiB device copy (for HBM counter scaling)")
    p.add_argument("--gen-device", choices=["cuda", "cpu"], default="cuda",
                   help="where the synthetic inputs are generated (cpu: only the library's "
                        "kernels run on the GPU, for counter collection)")
    p.add_argument("--table-limit", type=int, default=None,
                   help="threshold-table size limit passed to same_create_ex (0: products only)")
    p.add_argument("--no-stream", action="store_true",
                   help="skip the out-of-core (pinned host memory) timing")
    p.add_argument("--stream-steps", type=int, default=2)
    p.add_argument("--minibatches", type=int, default=None,
                   help="process only the first K minibatches (profiling runs)")
    return p.parse_args()


def main():
    args = parse()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py runs on exactly one GPU: this build has no multi-GPU path "
              "(see the design notes for how the sampler would shard columns)", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    import paper_1511_06416_amd as same
    from workloads import CONFIGS, make_workload

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    same.load_library()

    t0 = time.time()
    probe = make_workload(args.cfg, n_cols=args.n_cols, device="cpu", minibatches=[])
    mbs = list(range(probe.M if args.minibatches is None else min(args.minibatches, probe.M)))
    gen_dev = dev if args.gen_device == "cuda" else torch.device("cpu")
    w = make_workload(args.cfg, n_cols=args.n_cols, device=gen_dev, minibatches=mbs)
    if args.gen_device == "cpu":
        w.states = [s.to(dev) for s in w.states]
        w.obs = [o.to(dev) for o in w.obs]
    torch.cuda.synchronize()
    log("generated %s on %s in %.1f s: n=%d N=%d m=%d nb=%d M=%d ld=%d, timing %d minibatches" % (
        w.name, args.gen_device, time.time() - t0, w.net.n, w.n_cols, w.m, w.nb, w.M, w.ld,
        len(mbs)))
    net = w.net
    # the oracle's sample is taken from the generator's output, before any sweep
    sample = None
    if not args.no_cpu_baseline:
        cols = min(args.cpu_sample_cols, w.mb_cols(0))
        cols4 = (cols + 3) // 4 * 4
        sample = (cols, np.ascontiguousarray(w.states[0][:, :, :cols4].cpu().numpy()),
                  np.ascontiguousarray(w.obs[0][:, :cols4].cpu().numpy()))
    pptr, pidx, card = net.csr()
    if args.table_limit is None:
        ctx = same.same_create(pptr, pidx, card, w.alpha)
    else:
        ctx = same.same_create_ex(pptr, pidx, card, w.alpha, args.table_limit)
    ws = ctx.new_workspace(dev)
    cpts = torch.from_numpy(w.init_theta).to(dev)
    mb = torch.from_numpy(np.zeros((w.M, ctx.cpt_total), dtype=np.int32)).to(dev)
    tot = torch.from_numpy(np.zeros(ctx.cpt_total, dtype=np.int32)).to(dev)
    stream = torch.cuda.current_stream()
    obs_host = [w.obs[b][:, :w.mb_cols(b)].cpu().numpy() for b in mbs]
    latent = sum(int((o == 0).sum()) for o in obs_host)
    cols_timed = sum(w.mb_cols(b) for b in mbs)
    hidden = latent / float(net.n * cols_timed)
    del obs_host

    # count-only pre-pass initialises the per-minibatch counts and their sum
    for b in mbs:
        same.same_counts(ctx, w.states[b], w.m, w.mb_cols(b), w.ld, mb[b], tot, ws)

    def one_pass(s):
        for b in mbs:
            same.same_step(ctx, w.states[b], w.obs[b], cpts, w.m, w.mb_cols(b), w.ld, b * w.nb,
                           w.seed, s, mb[b], tot, s * w.M + b, ws)

    for s in range(args.warmup):
        one_pass(s)
    torch.cuda.synchronize()
    log("warmup done")
    t_start = time.perf_counter()
    ev_start = torch.cuda.Event(enable_timing=True)
    ev_end = torch.cuda.Event(enable_timing=True)
    ev_start.record(stream)
    for s in range(args.warmup, args.warmup + args.steps):
        one_pass(s)
    ev_end.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t_start
    gpu_ms = ev_start.elapsed_time(ev_end)
    elapsed = max(wall, gpu_ms / 1e3)
    log("timed %d passes: wall %.3f s, events %.3f s" % (args.steps, wall, gpu_ms / 1e3))
    node_samples = float(net.n) * cols_timed * w.m * args.steps

    # the sweep kernels alone: HIP events around every same_sweep call of one
    # further pass over the same minibatches (same launches as inside same_step)
    sweep_ev = []
    s_extra = args.warmup + args.steps
    for b in mbs:
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        same.same_sweep(ctx, w.states[b], w.obs[b], cpts, w.m, w.mb_cols(b), w.ld, b * w.nb,
                        w.seed, s_extra, ws)
        e1.record(stream)
        sweep_ev.append((e0, e1))
    torch.cuda.synchronize()

    value = node_samples / elapsed
    sweep_s = sum(a.elapsed_time(b) for a, b in sweep_ev) / 1e3
    launches = sum(same.same_sweep_plan(ctx, w.m, w.mb_cols(b))[1] for b in mbs)
    node_samples_sweep = float(net.n) * cols_timed * w.m
    bytes_per_ns = 1.0 + hidden + 1.0 / w.m   # read each state, write each latent, obs per column
    alg_bytes = node_samples * bytes_per_ns
    achieved = node_samples_sweep * bytes_per_ns / sweep_s / 1e9
    roofline = {
        "kernel": "sweep_main_kernel (every colour-group launch of a sweep)",
        "bound": "hbm",
        "achieved": round(achieved, 1),
        "peak": HBM_PEAK_GBS,
        "unit": "GB/s",
        "frac": round(achieved / HBM_PEAK_GBS, 4),
        "traffic": None,
        "bytes_per_node_sample": round(bytes_per_ns, 4),
        "launches": launches,
        "avg_launch_ms": round(sweep_s * 1e3 / launches, 4),
        "sweep_share_of_step": round(sweep_s * args.steps / elapsed, 3),
        "tile_cols": same.same_sweep_plan(ctx, w.m, w.mb_cols(0))[0],
    }

    if args.copy_calibration:
        # a plain device-to-device copy of exactly 1 GiB (runtime copy kernel)
        a = torch.from_numpy(np.zeros(1 << 30, dtype=np.uint8)).to(dev)
        b2 = torch.from_numpy(np.ones(1 << 30, dtype=np.uint8)).to(dev)
        b2.copy_(a)
        torch.cuda.synchronize()
        del a, b2

    streamed = None
    if not args.no_stream and len(mbs) == w.M:
        streamed = stream_timing(w, ctx, cpts, ws, dev, args.stream_steps)

    cpu = None
    if sample is not None:
        cpu = cpu_baseline(w, *sample)

    spec = CONFIGS[args.cfg]
    out = {
        "metric": METRIC,
        "value": round(value, 1),
        "unit": "node-samples/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(elapsed * 1e3 / args.steps, 3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {
            "workload": "%s: %d-node random DAG, 0-%d parents, K in {%d..%d}, %d columns in "
                        "%d-column minibatches resident in HBM, %.0f%% hidden, SAME m=%d" % (
                            w.name, net.n, spec["graph"][2] if spec["graph"][0] == "random" else 0,
                            int(net.card.min()), int(net.card.max()), w.n_cols, w.nb,
                            100 * w.hidden, w.m) if args.cfg in (3, 5) else w.name,
            "global_batch": cols_timed,
            "minibatches_timed": len(mbs),
            "minibatch_cols": w.nb,
            "replicas": w.m,
            "nodes": net.n,
            "colors": ctx.n_colors,
            "hidden_fraction": round(hidden, 4),
            "parallelism": "single-gpu",
        },
        "latent_draws_per_s": round(value * hidden, 1),
        "hbm_gbs_algorithmic_step": round(alg_bytes / elapsed / 1e9, 1),
        "roofline": roofline,
        "cpu_baseline": cpu,
        "streamed_from_host": streamed,
        "table_nodes": ctx.table_nodes,
    }
    print(json.dumps(out), flush=True)


def stream_timing(w, ctx, cpts, ws, dev, steps):
    """End-to-end out-of-core passes: every minibatch is copied from pinned host
    memory to the device, swept, counted and resampled, and copied back
    (same_stream_pass).  Reported beside the HBM-resident value, never as it."""
    import torch

    import paper_1511_06416_amd as same

    net = w.net
    host_ld = (w.n_cols + 3) // 4 * 4
    t0 = time.time()
    hs = torch.empty((net.n, w.m, host_ld), dtype=w.states[0].dtype, pin_memory=True)
    ho = torch.empty((net.n, host_ld), dtype=torch.uint8, pin_memory=True)
    for b in range(w.M):
        c0, nc = b * w.nb, w.mb_cols(b)
        for i in range(net.n):
            hs[i, :, c0:c0 + nc].copy_(w.states[b][i, :, :nc])
            ho[i, c0:c0 + nc].copy_(w.obs[b][i, :nc])
    torch.cuda.synchronize()
    log("pinned host copy of the data (%.1f GB) in %.1f s" % (
        (hs.numel() * hs.element_size() + ho.numel()) / 1e9, time.time() - t0))
    slots = torch.empty(same.same_stream_slots_size(ctx, w.m, w.nb), dtype=torch.uint8, device=dev)
    mb = torch.zeros((w.M, ctx.cpt_total), dtype=torch.int32, device=dev)
    tot = torch.zeros(ctx.cpt_total, dtype=torch.int32, device=dev)
    same.same_stream_pass(ctx, hs, ho, host_ld, w.n_cols, w.nb, w.m, cpts, mb, tot, w.seed, 0,
                          same.SAME_STREAM_COUNTS_ONLY, slots, ws)
    same.same_stream_pass(ctx, hs, ho, host_ld, w.n_cols, w.nb, w.m, cpts, mb, tot, w.seed, 0, 0,
                          slots, ws)
    torch.cuda.synchronize()
    t = time.perf_counter()
    for s in range(1, 1 + steps):
        same.same_stream_pass(ctx, hs, ho, host_ld, w.n_cols, w.nb, w.m, cpts, mb, tot, w.seed, s,
                              0, slots, ws)
    torch.cuda.synchronize()
    dt = time.perf_counter() - t
    ns = float(net.n) * w.n_cols * w.m * steps
    state_bytes = float(net.n) * w.m * w.n_cols * hs.element_size()
    h2d = state_bytes + float(net.n) * w.n_cols
    log("streamed %d passes in %.3f s" % (steps, dt))
    del hs, ho
    return {"value": round(ns / dt, 1), "unit": "node-samples/s", "passes": steps,
            "ms_per_pass": round(dt * 1e3 / steps, 2),
            "pcie_bytes_per_pass": {"h2d": h2d, "d2h": state_bytes},
            "pcie_gbs_each_way": {"h2d": round(h2d * steps / dt / 1e9, 1),
                                  "d2h": round(state_bytes * steps / dt / 1e9, 1)}}


def cpu_baseline(w, cols, st, ob):
    """The oracle (fp64, OpenMP over columns) on the first `cols` columns of
    minibatch 0 as generated: one sweep, its counts and one Dirichlet resample."""
    import oracle

    net = w.net
    threads = len(os.sched_getaffinity(0))
    color = oracle.graph(net.parents, net.card)["color"]
    t = time.perf_counter()
    oracle.sweep(net.parents, net.card, w.init_theta, color, st, ob, w.m, cols, 0, w.seed, 0,
                 n_threads=threads)
    cnt = oracle.counts(net.parents, net.card, st, w.m, cols, n_threads=threads)
    oracle.dirichlet(net.parents, net.card, cnt, w.alpha, w.seed, 0)
    dt = time.perf_counter() - t
    ns = float(net.n) * cols * w.m
    log("cpu baseline: %d columns, %.2f s, %d threads" % (cols, dt, threads))
    return {"value": round(ns / dt, 1), "unit": "node-samples/s", "cores": threads,
            "kind": "oracle",
            "sample": "first %d columns of minibatch 0 (all %d nodes, m=%d): one sweep + counts "
                      "+ one Dirichlet resample, %.1f s" % (cols, net.n, w.m, dt)}


if __name__ == "__main__":
    main()
