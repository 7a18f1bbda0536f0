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
    p.add_argument("--cpu-sample-cols", type=int, default=250_000,
                   help="columns of minibatch 0 the oracle baseline runs on (all nodes, all replicas)")
    p.add_argument("--cpu-sample-steps", type=int, default=2,
                   help="SAME steps (sweep + counts + resample) of the oracle baseline")
    p.add_argument("--copy-calibration", action="store_true",
                   help="(kept for older profile commands: the 1 GiB copy now always runs)")
    p.add_argument("--state-bits", type=int, default=-1,
                   help="bits per state in the library's state quads: 4 (every K <= 16), 0 for 8/16-bit; "
                        "default: 4 when the network allows it")
    p.add_argument("--graph-steps", type=int, default=8,
                   help="SAME steps per captured graph in the graphed timing (single-minibatch workloads)")
    p.add_argument("--roofline-steps", type=int, default=1,
                   help="instrumented passes after the timed ones, for the per-launch roofline")
    p.add_argument("--parity-cols", type=int, default=32_768,
                   help="columns of minibatch 0 on which the first GPU sweep is compared with the "
                        "oracle's (flagged fraction, mismatch rate; 0 to skip)")
    p.add_argument("--gen-device", choices=["cuda", "cpu"], default="cuda",
                   help="where the synthetic inputs are generated (cpu: only the library's "
                        "kernels run on the GPU, for counter collection)")
    p.add_argument("--table-limit", type=int, default=None,
                   help="threshold-table size limit passed to same_create_ex (0: products only)")
    p.add_argument("--no-m-study", action="store_true",
                   help="skip the KL_avg-vs-time study of the SAME replication factor (two-layer network)")
    p.add_argument("--no-heldout", action="store_true",
                   help="skip the held-out prediction run (two-layer network) and the hit-count timing")
    p.add_argument("--no-ingest", action="store_true",
                   help="skip the timing of the sparse-input expansion and the latent initialisation")
    p.add_argument("--no-stream", action="store_true",
                   help="skip the out-of-core (pinned host memory) timing")
    p.add_argument("--stream-steps", type=int, default=2)
    p.add_argument("--minibatches", type=int, default=None,
                   help="process only the first K minibatches (profiling runs)")
    p.add_argument("--counters-summary", nargs="+", metavar="CSV", default=None,
                   help="summarise rocprofv3 counter_collection CSVs (no GPU work): per-kernel "
                        "averages, and the sweep kernel's HBM traffic scaled by the 1 GiB copy")
    return p.parse_args()


def main():
    args = parse()
    if args.counters_summary:
        counters_summary(args.counters_summary, args.cfg)
        return
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py runs on exactly one GPU: the library has no multi-GPU path (columns would shard "
              "across GPUs with an all-reduce of the int32 count deltas per CPT update)", file=sys.stderr)
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
    bits = args.state_bits if args.state_bits >= 0 else (4 if int(net.card.max()) <= 16 else 0)
    ctx = same.same_create_ex(pptr, pidx, card, w.alpha, -1 if args.table_limit is None else args.table_limit,
                              state_bits=bits)
    w.bits = 4 if ctx.state_bits == 4 else None   # pack_states / unpack_states argument
    ws = ctx.new_workspace(dev)
    cpts = torch.from_numpy(w.init_theta).to(dev)
    cpts0 = cpts.clone()
    mb = torch.from_numpy(np.zeros((w.M, ctx.cpt_total), dtype=np.int32)).to(dev)
    tot = torch.from_numpy(np.zeros(ctx.cpt_total, dtype=np.int32)).to(dev)
    stream = torch.cuda.current_stream()
    obs_host = [w.obs[b][:, :w.mb_cols(b)].cpu().numpy() for b in mbs]
    latent = sum(int((o == 0).sum()) for o in obs_host)
    cols_timed = sum(w.mb_cols(b) for b in mbs)
    hidden = latent / float(net.n * cols_timed)
    del obs_host
    # the library's replica-quad layout of the timed minibatches (input
    # preparation, on the device); the generator's row layout stays for the
    # oracle's sample and the host-side preparations
    w.pk = {b: same.pack_states(w.states[b], w.bits) for b in mbs}
    torch.cuda.synchronize()

    # count-only pre-pass initialises the per-minibatch counts and their sum
    for b in mbs:
        same.same_counts(ctx, w.pk[b], w.m, w.mb_cols(b), w.ld, mb[b], tot, ws)

    def one_pass(s):
        for b in mbs:
            same.same_step(ctx, w.pk[b], w.obs[b], cpts, w.m, w.mb_cols(b), w.ld, b * w.nb,
                           w.seed, s, mb[b], tot, s * w.M + b, ws)

    for s in range(args.warmup):
        one_pass(s)
    torch.cuda.synchronize()
    log("warmup done")
    # the timed passes run without any per-launch instrumentation
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
    value = node_samples / elapsed

    # then more passes of the same loop with every sweep-kernel launch
    # bracketed by HIP events on its launch stream (the library records them)
    # for the per-launch roofline figures
    rsteps = max(1, args.roofline_steps)
    same.same_kernel_timing(ctx, True)
    t_r = time.perf_counter()
    for s in range(args.warmup + args.steps, args.warmup + args.steps + rsteps):
        one_pass(s)
    torch.cuda.synchronize()
    wall_r = time.perf_counter() - t_r
    kt = same.same_kernel_times(ctx)
    same.same_kernel_timing(ctx, False)
    log("instrumented %d passes: %.3f s; sweep kernels per class (ms, launches): %s; colour phases %.2f ms" % (
        rsteps, wall_r, list(zip(kt["ms"], kt["launches"])), kt["phase_ms"]))
    node_samples_r = float(net.n) * cols_timed * w.m * rsteps

    copy_gbs = copy_peak(dev, stream)
    roofline = sweep_roofline(w, net, mbs, hidden, node_samples_r, kt, wall_r, args, copy_gbs, ctx)
    graphed = graph_timing(w, ctx, mbs, cpts, mb, tot, ws, args.warmup + args.steps + rsteps, args.steps, dev,
                           stream, args.graph_steps)
    log("graphed %d passes: %.3f ms per pass" % (args.steps, graphed["ms_per_step"]))



    ingest = None if args.no_ingest else ingest_timing(w, ctx, mbs[0], dev, stream)
    heldout = None if args.no_heldout else heldout_timing(w, ctx, mbs[0], dev, stream)
    m_study = None if args.no_m_study else m_study_run(dev, stream)

    streamed = None
    if not args.no_stream and len(mbs) == w.M:
        streamed = stream_timing(w, ctx, cpts, ws, dev, args.stream_steps)

    cpu = parity = None
    if sample is not None:
        # untimed: the GPU's first sweep of the sample's leading columns
        # against the oracle's, then the timed oracle baseline
        if args.parity_cols > 0:
            parity = first_sweep_parity(w, ctx, cpts0, ws, sample, args.parity_cols, dev)
        cpu = cpu_baseline(w, *sample, args.cpu_sample_steps)

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
            "state_bits": ctx.state_bits,
            "hidden_fraction": round(hidden, 4),
            "parallelism": "single-gpu",
        },
        "latent_draws_per_s": round(value * hidden, 1),
        "hbm_gbs_algorithmic_step": round(node_samples * bytes_per_node_sample(ctx, hidden, w.m) / elapsed / 1e9, 1),
        "roofline": roofline,
        "graphed": graphed,
        "parity": parity,
        "cpu_baseline": cpu,
        "streamed_from_host": streamed,
        "ingest": ingest,
        "heldout": heldout,
        "m_study": m_study,
        "table_nodes": ctx.table_nodes,
    }
    print(json.dumps(out), flush=True)


ALU_PEAK_TOPS = 256 * 64 * 2.4e9 / 1e12   # one 32-bit VALU op per lane per clock
PHILOX_OPS_PER_DRAW = 23                   # 80 ops per Philox4x32-10 block / 4 words + U24


def graph_timing(w, ctx, mbs, cpts, mb, tot, ws, first_pass, passes, dev, stream, per_graph):
    """The timed loop again with every minibatch's step replayed from a
    captured HIP graph (same_step_graph, one per minibatch, ids advanced on the
    device) instead of issued launch by launch; beside `value`, never it.  With
    a single minibatch one graph holds `per_graph` consecutive steps."""
    import torch

    import paper_1511_06416_amd as same
    k = per_graph if len(mbs) == 1 else 1
    passes = (passes + k - 1) // k * k
    ids = torch.tensor([[first_pass, first_pass * w.M + b] for b in mbs], dtype=torch.int32, device=dev)
    graphs = [same.same_step_graph(ctx, w.pk[b], w.obs[b], cpts, w.m, w.mb_cols(b), w.ld, b * w.nb, w.seed,
                                   mb[b], tot, ids[i], w.M, k, ws) for i, b in enumerate(mbs)]
    for g in graphs:
        g.launch(stream)
    torch.cuda.synchronize()
    t = time.perf_counter()
    ev0 = torch.cuda.Event(enable_timing=True)
    ev1 = torch.cuda.Event(enable_timing=True)
    ev0.record(stream)
    for _ in range(passes // k):
        for g in graphs:
            g.launch(stream)
    ev1.record(stream)
    torch.cuda.synchronize()
    el = max(time.perf_counter() - t, ev0.elapsed_time(ev1) / 1e3)
    for g in graphs:
        g.close()
    ns = float(w.net.n) * sum(w.mb_cols(b) for b in mbs) * w.m * passes
    return {"value": round(ns / el, 1), "unit": "node-samples/s", "passes": passes, "steps_per_graph": k,
            "ms_per_step": round(el * 1e3 / passes, 4)}


def alu_ops_per_draw(net):
    """Algorithmic 32-bit operations of one latent draw of each node: one
    multiply-add per blanket state term of the CPT row indices, K * (children)
    multiplications of the conditional, K running sums, K comparisons, and a
    quarter of a Philox4x32-10 block plus the uniform's conversion."""
    import numpy as np
    n = net.n
    kids = [[] for _ in range(n)]
    for h, ps in enumerate(net.parents):
        for p in ps:
            kids[p].append(h)
    ops = np.zeros(n)
    for i in range(n):
        K = int(net.card[i])
        terms = len(net.parents[i]) + sum(len(net.parents[h]) for h in kids[i])
        ops[i] = terms + K * len(kids[i]) + 2 * K + PHILOX_OPS_PER_DRAW
    return ops


def source_hash():
    import hashlib
    h = hashlib.sha256()
    for f in ("kernels.hip", "graph.cpp", "graph.hpp"):
        with open(os.path.join(ROOT, "paper_1511_06416_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def traffic_path(cfg):
    from workloads import CONFIGS
    return os.path.join(ROOT, "profiles", "sweep_fast_kernel.%s.traffic.json" % CONFIGS[cfg]["name"])


def state_type_name(bits):
    return {4: "Nib", 8: "int8", 16: "int16"}[bits]


def measured_traffic(cfg, bits):
    """HBM bytes per sweep-kernel launch from the committed counter summary of
    this workload, if it was taken on the current kernel sources and state
    format (else None)."""
    path = traffic_path(cfg)
    if not os.path.exists(path):
        return None
    with open(path) as fh:
        t = json.load(fh)
    if t.get("sources_sha256") != source_hash() or t.get("state_bits") != bits:
        return None
    return t


def copy_peak(dev, stream, reps=5):
    """Device-to-device copy rate of 1 GiB (torch's copy kernel), GB/s counting
    the bytes read and written: the practical HBM ceiling beside the 8 TB/s
    spec."""
    import torch
    a = torch.zeros(COPY_BYTES, dtype=torch.uint8, device=dev)
    b = torch.ones(COPY_BYTES, dtype=torch.uint8, device=dev)
    b.copy_(a)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(reps):
        b.copy_(a)
    e1.record(stream)
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / reps
    del a, b
    return 2.0 * COPY_BYTES / (ms / 1e3) / 1e9


def first_sweep_parity(w, ctx, cpts0, ws, sample, cols, dev):
    """The library's production sweep (same_sweep) and the oracle's sweep from
    the same generated states of the first `cols` columns of minibatch 0, with
    the starting CPTs, seed and sweep id 0.  A chain (column, replica) may
    differ only from a flagged draw on (a uniform within 1e-6 of a CDF
    boundary) in visit order; reports the flagged fraction of the latent draws
    and the mismatch rate (chains that differ, per latent draw)."""
    import numpy as np
    import torch

    import oracle
    import paper_1511_06416_amd as same
    net = w.net
    _cols, st, ob, = sample
    cols = min(cols, _cols) // 4 * 4
    pre = np.ascontiguousarray(st[:, :, :cols])
    obs = np.ascontiguousarray(ob[:, :cols])
    d_st = torch.from_numpy(same.pack_states(pre, w.bits)).to(dev)
    d_ob = torch.from_numpy(obs).to(dev)
    same.same_sweep(ctx, d_st, d_ob, cpts0, w.m, cols, cols, 0, w.seed, 0, ws)
    torch.cuda.synchronize()
    gpu = same.unpack_states(d_st.cpu().numpy(), w.m, w.bits)
    del d_st, d_ob
    ref = pre.copy()
    color = oracle.graph(net.parents, net.card)["color"]
    res = oracle.sweep(net.parents, net.card, cpts0.cpu().numpy(), color, ref, obs, w.m, cols, 0, w.seed, 0,
                       want_flags=True)
    flags = res["flags"]
    draws = int((obs == 0).sum()) * w.m
    order = np.array(sorted(range(net.n), key=lambda i: (int(color[i]), i)))
    diff = (gpu != ref)[order]
    chains = diff.any(axis=0)
    first = diff.argmax(axis=0)
    fl = np.take_along_axis(flags[order], first[None], axis=0)[0]
    n_chains = int(chains.sum())
    unexcused = int((chains & (fl == 0)).sum())
    n_flag = int(flags.sum())
    return {"sample": "first %d columns of minibatch 0 (all nodes, m=%d), sweep 0 from the generated states"
                      % (cols, w.m),
            "latent_draws": draws, "flagged_draws": n_flag, "flagged_fraction": n_flag / max(draws, 1),
            "mismatched_chains": n_chains, "mismatch_rate": n_chains / max(draws, 1),
            "unexcused_mismatches": unexcused, "ok": unexcused == 0 and n_chains < 1e-5 * draws}


def bytes_per_node_sample(ctx, hidden, m):
    """Algorithmic bytes per (node, column, replica) slot of a sweep: read
    every state once, write every latent state once (bits / 8 bytes each) and
    read the obs byte once per column (shared by the m replicas)."""
    sb = ctx.state_bits / 8.0
    return sb * (1.0 + hidden) + 1.0 / m


def sweep_roofline(w, net, mbs, hidden, node_samples, kt, elapsed, args, copy_gbs, ctx):
    """Roofline of the dominant kernel, the LDS-staged sweep kernel
    (sweep_fast_kernel, LDS-staged, launch class 0), which draws almost
    every node of the workload in one launch per colour group: the algorithmic
    bytes of the (node, column, replica) slots its launches covered per second
    of its own launch time, against HBM peak.  Beside it: algorithmic 32-bit
    operations per second against the VALU peak, the HBM bytes the counters
    measured per launch (when taken on the current kernel sources), the
    global-table launches (class 1, beside class 0 on a second stream) and the
    colour phases (the sweep's own device time, all classes)."""
    import numpy as np
    assert kt["launches"][2] == 0 and kt["launches"][3] == 0, \
        "this workload is expected to run entirely in the fast sweep kernel"
    bytes_per_ns = bytes_per_node_sample(ctx, hidden, w.m)
    alg_bytes = node_samples * bytes_per_ns
    # latent draws per node per step, from the obs masks of the timed minibatches
    lat = np.zeros(net.n)
    for b in mbs:
        lat += (w.obs[b][:, :w.mb_cols(b)] == 0).sum(dim=1).cpu().numpy().astype(np.float64)
    ops = float((alu_ops_per_draw(net) * lat).sum()) * w.m * max(1, args.roofline_steps)
    ms0, n0, ns0 = kt["ms"][0], kt["launches"][0], kt["node_samples"][0]
    bytes0 = ns0 * bytes_per_ns
    ops0 = ops * ns0 / node_samples   # at the workload's mean operations per slot
    secs0 = ms0 / 1e3
    hbm = bytes0 / secs0 / 1e9
    alu = ops0 / secs0 / 1e12
    traffic = measured_traffic(args.cfg, ctx.state_bits)
    avg_ms = ms0 / n0
    phase_s = kt["phase_ms"] / 1e3
    out = {
        "kernel": "sweep_fast_kernel<%s, false, true> (tables staged in LDS, whole or in part; "
                  "every launch of the timed passes)" % state_type_name(ctx.state_bits),
        "bound": "hbm",
        "achieved": round(hbm, 1),
        "peak": HBM_PEAK_GBS,
        "unit": "GB/s",
        "frac": round(hbm / HBM_PEAK_GBS, 4),
        "traffic": None if traffic is None else traffic["hbm_bytes_per_launch"],
        "copy_peak_gbs": round(copy_gbs, 1),
        "frac_of_copy_peak": round(hbm / copy_gbs, 4),
        "algorithmic_bytes_per_launch": round(bytes0 / n0, 1),
        "bytes_per_node_sample": round(bytes_per_ns, 4),
        "node_samples_share": round(ns0 / node_samples, 4),
        "launches": n0,
        "avg_launch_ms": round(avg_ms, 4),
        "alu": {"achieved": round(alu, 3), "peak": round(ALU_PEAK_TOPS, 2), "unit": "TOP/s",
                "frac": round(alu / ALU_PEAK_TOPS, 4),
                "algorithmic_ops_per_launch": round(ops0 / n0, 1)},
        "global_table_launches": {
            "launches": kt["launches"][1], "ms": round(kt["ms"][1], 3),
            "node_samples_share": round(kt["node_samples"][1] / node_samples, 4)},
        # class-1 launches run beside the class-0 launch of their colour (side
        # stream); the colour phases (first launch to joined last launch of a
        # colour) are the sweep's own device time
        "colour_phases": {
            "phases": int(kt["phases"]),
            "ms": round(kt["phase_ms"], 3),
            "achieved": round(alg_bytes / phase_s / 1e9, 1) if phase_s > 0 else None,
            "frac": round(alg_bytes / phase_s / 1e9 / HBM_PEAK_GBS, 4) if phase_s > 0 else None,
            "alu_frac": round(ops / phase_s / 1e12 / ALU_PEAK_TOPS, 4) if phase_s > 0 else None,
        },
        "sweep_share_of_step": round(phase_s / elapsed, 3),
    }
    if traffic is not None:
        out["traffic_gbs"] = round(traffic["hbm_bytes_per_launch"] / (avg_ms / 1e3) / 1e9, 1)
        if traffic.get("valu_insts_per_launch"):
            # executed VALU wave instructions (counters) beside the algorithmic
            # operation count: 64 lanes x 4 cycles each on a 16-lane SIMD
            out["alu"]["valu_insts_per_node_sample"] = round(
                traffic["valu_insts_per_launch"] / (ns0 / n0), 4)
            out["alu"]["valu_issue_frac"] = round(
                traffic["valu_insts_per_launch"] * 4 / 1024 / (avg_ms / 1e3 * 2.4e9), 4)
    out["timing"] = "per-launch figures from %d instrumented pass(es) after the timed ones" % args.roofline_steps
    return out


COPY_BYTES = 1 << 30


def counters_summary(paths, cfg):
    """Per-kernel averages of rocprofv3 counter CSVs (one counter set per run).
    FETCH_SIZE / WRITE_SIZE (KiB per dispatch) of the sweep kernel are scaled by
    what the same counters read for the 1 GiB device copy of --copy-calibration
    (1 GiB read and 1 GiB written), giving HBM bytes per launch; the result is
    written under profiles/ for later runs on the same kernel sources."""
    import collections
    import csv
    import re
    totals = collections.defaultdict(float)   # (kernel, counter) -> sum over dispatches
    seen = collections.defaultdict(set)       # (kernel, counter) -> dispatches
    dur = collections.defaultdict(dict)       # kernel -> dispatch -> microseconds
    per_dispatch = {}
    for path in paths:
        with open(path) as fh:
            for r in csv.DictReader(fh):
                k, c, d = r["Kernel_Name"], r["Counter_Name"], (path, r["Dispatch_Id"])
                totals[(k, c)] += float(r["Counter_Value"])
                seen[(k, c)].add(d)
                # largest value of each (kernel, counter, grid): finds single dispatches
                key = (k, c, r["Grid_Size"])
                per_dispatch[key] = max(per_dispatch.get(key, 0.0), float(r["Counter_Value"]))
                dur[k][d] = (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3

    def avg(k, c):
        return totals[(k, c)] / len(seen[(k, c)]) if (k, c) in seen else None

    kernels = sorted(dur, key=lambda k: -sum(dur[k].values()))
    counters = sorted({c for (_k, c) in totals})
    print("| kernel | dispatches | avg us | " + " | ".join(counters) + " |")
    print("|---|---|---|" + "---|" * len(counters))
    for k in kernels:
        vals = ["-" if avg(k, c) is None else "%.4g" % avg(k, c) for c in counters]
        print("| %s | %d | %.1f | %s |" % (k[:100], len(dur[k]), sum(dur[k].values()) / len(dur[k]),
                                         " | ".join(vals)))
    sweep = [k for k in kernels if re.search(r"sweep_fast_kernel<[^,]+, false, true>", k)]
    # the 1 GiB device copy: the non-library dispatch whose WRITE_SIZE is 1 GiB
    # within 5% and that also reads (the fills that create the buffers read
    # nothing); its FETCH_SIZE is the same kernel and grid in the FETCH_SIZE run
    copy = fetch_copy = None
    for (k, c, grid), v in per_dispatch.items():
        if c == "WRITE_SIZE" and "same::" not in k and abs(v * 1024 - COPY_BYTES) < 0.05 * COPY_BYTES:
            f = per_dispatch.get((k, "FETCH_SIZE", grid))
            if f and f * 1024 > 0.25 * COPY_BYTES:
                copy, fetch_copy = (k, grid, v), f
    if copy is None or not fetch_copy or not sweep:
        print("no copy calibration, FETCH_SIZE run or sweep kernel in these files")
        return
    f_scale = COPY_BYTES / (fetch_copy * 1024)
    w_scale = COPY_BYTES / (copy[2] * 1024)

    def per_launch(c):
        n = sum(len(seen[(k, c)]) for k in sweep if (k, c) in seen)
        return sum(totals.get((k, c), 0.0) for k in sweep) * 1024 / max(n, 1), n

    fb, nf = per_launch("FETCH_SIZE")
    wb, nw = per_launch("WRITE_SIZE")
    fb *= f_scale
    wb *= w_scale
    names = " ".join(sweep)
    bits = 4 if "Nib" in names else (16 if "short" in names else 8)
    out = {
        "kernel": "sweep_fast_kernel<%s, false, true> (LDS-staged, non-debug)" % state_type_name(bits),
        "state_bits": bits,
        "workload_cfg": cfg,
        "copy_kernel": copy[0],
        "copy_counters_kib": {"FETCH_SIZE": fetch_copy, "WRITE_SIZE": copy[2]},
        "scale": {"fetch": round(f_scale, 4), "write": round(w_scale, 4)},
        "fetch_bytes_per_launch": round(fb, 1),
        "write_bytes_per_launch": round(wb, 1),
        "hbm_bytes_per_launch": round(fb + wb, 1),
        "dispatches": {"fetch": nf, "write": nw},
        "valu_insts_per_launch": (round(per_launch("SQ_INSTS_VALU")[0] / 1024, 1)
                                  if any((k, "SQ_INSTS_VALU") in seen for k in sweep) else None),
        "sources_sha256": source_hash(),
    }
    path = traffic_path(cfg)
    os.makedirs(os.path.dirname(path), exist_ok=True)
    with open(path, "w") as fh:
        json.dump(out, fh, indent=1)
    print(json.dumps(out))


def ingest_timing(w, ctx, b, dev, stream, reps=5):
    """Data ingest of minibatch b (Sec. 4 sparse input; Sec. 5.2 random start):
    same_expand_observed from the minibatch's known entries in CSR form (rows =
    nodes), then same_init_latent, each timed with HIP events on the launch
    stream (into scratch copies; the benchmark's states are not touched).  The
    CSR arrays are built with torch from the dense minibatch (input
    preparation).  Algorithmic bytes: expand reads row_ptr, the column indices
    and the values and writes the obs array and m copies of every known value;
    the initialisation reads the obs array and writes every latent state."""
    import numpy as np
    import torch

    import paper_1511_06416_amd as same
    n, m, ld, nc = w.net.n, w.m, w.ld, w.mb_cols(b)
    sb = w.states[b].element_size()
    ob = w.obs[b]
    known = ob[:, :nc].bool()
    rows, cols = torch.nonzero(known, as_tuple=True)
    nnz = int(rows.numel())
    row_ptr = torch.zeros(n + 1, dtype=torch.int64, device=dev)
    row_ptr[1:] = torch.cumsum(torch.bincount(rows, minlength=n), 0)
    col_idx = cols.to(torch.int32)
    values = w.states[b][:, 0, :nc][known].contiguous()
    del rows, cols, known
    st = torch.empty_like(w.pk[b])
    obs = torch.empty_like(ob)
    torch.cuda.synchronize()

    def timed(fn):
        fn()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(reps):
            fn()
        e1.record(stream)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / reps

    t_exp = timed(lambda: same.same_expand_observed(ctx, row_ptr, col_idx, values, nnz, m, nc, ld, st, obs))
    t_init = timed(lambda: same.same_init_latent(ctx, st, obs, m, nc, ld, b * w.nb, w.seed + 1))
    latent = n * nc - nnz
    b_exp = 8 * (n + 1) + (4 + sb) * nnz + n * ld + m * sb * nnz
    b_init = n * ld + m * sb * latent
    del st, obs, row_ptr, col_idx, values
    return {
        "minibatch_cols": nc, "nnz": nnz, "density": round(nnz / float(n * nc), 4),
        "expand": {"ms": round(t_exp, 4), "algorithmic_bytes": b_exp,
                   "gbs": round(b_exp / t_exp / 1e6, 1), "frac": round(b_exp / t_exp / 1e6 / HBM_PEAK_GBS, 4)},
        "init_latent": {"ms": round(t_init, 4), "algorithmic_bytes": b_init,
                        "gbs": round(b_init / t_init / 1e6, 1),
                        "frac": round(b_init / t_init / 1e6 / HBM_PEAK_GBS, 4)},
        "upload_bytes": {"sparse_csr": 8 * (n + 1) + (4 + sb) * nnz, "dense": n * ld * (1 + m * sb)},
    }


def heldout_timing(w, ctx, b, dev, stream, train_steps=60, pred_sweeps=20):
    """Held-out prediction (Sec. 6).  (1) On the two-layer network
    (concepts30-items300-4k, the shape of the paper's MOOC network): 20% of
    the known entries are held out, the sampler trains on the rest for
    train_steps SAME steps, then same_predict samples pred_sweeps sweeps with
    the CPTs frozen; the AUC of the estimated probabilities of the held-out
    states is reported with the prediction pass's time.  (2) On minibatch b
    of the benchmark workload, same_accumulate_hits against a 20% held-out
    target, timed with HIP events; algorithmic bytes: the states once, the
    targets once, the hit counters read and written."""
    import numpy as np
    import torch

    import paper_1511_06416_amd as same
    from paper_1511_06416_amd import evaluate
    from workloads import holdout, make_workload

    h = make_workload(4, device=dev)
    net = h.net
    obs_train, target = holdout(h, 0, 0.2)
    pptr, pidx, card = net.csr()
    hctx = same.same_create(pptr, pidx, card, h.alpha)
    hws = hctx.new_workspace(dev)
    st = same.pack_states(h.states[0])
    ob = torch.from_numpy(obs_train).to(dev)
    tg = torch.from_numpy(target).to(dev)
    same.same_init_latent(hctx, st, ob, h.m, h.n_cols, h.ld, 0, h.seed + 17)
    cpts = torch.from_numpy(h.init_theta).to(dev)
    mbc = torch.zeros(hctx.cpt_total, dtype=torch.int32, device=dev)
    tot = torch.zeros(hctx.cpt_total, dtype=torch.int32, device=dev)
    same.same_counts(hctx, st, h.m, h.n_cols, h.ld, mbc, tot, hws)
    for s in range(train_steps):
        same.same_step(hctx, st, ob, cpts, h.m, h.n_cols, h.ld, 0, h.seed, s, mbc, tot, s, hws)
    hits = torch.zeros(target.shape, dtype=torch.int32, device=dev)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record(stream)
    same.same_predict(hctx, st, ob, cpts, tg, h.m, h.n_cols, h.ld, 0, h.seed, 1 << 20, pred_sweeps, hits, hws)
    e1.record(stream)
    torch.cuda.synchronize()
    t_pred = e0.elapsed_time(e1)
    sc, lab = evaluate.binary_scores(hits.cpu().numpy(), target, pred_sweeps * h.m)
    a = evaluate.auc(sc, lab)
    hctx.close()
    del st, ob, tg, hits, h

    # hit-count kernel on the benchmark minibatch
    n, m, ld, nc = w.net.n, w.m, w.ld, w.mb_cols(b)
    sb = w.states[b].element_size()
    g = torch.Generator(device=dev)
    g.manual_seed(6)
    pick = (torch.rand(w.obs[b].shape, generator=g, device=dev) < 0.2) & (w.obs[b] == 1)
    tgt = torch.where(pick, w.states[b][:, 0, :], torch.full_like(w.states[b][:, 0, :], -1)).contiguous()
    hc = torch.zeros((n, ld), dtype=torch.int32, device=dev)
    same.same_accumulate_hits(ctx, w.pk[b], tgt, m, nc, ld, hc)
    torch.cuda.synchronize()
    reps = 5
    e0.record(stream)
    for _ in range(reps):
        same.same_accumulate_hits(ctx, w.pk[b], tgt, m, nc, ld, hc)
    e1.record(stream)
    torch.cuda.synchronize()
    t_hits = e0.elapsed_time(e1) / reps
    b_hits = n * m * ld * sb + n * ld * sb + 8 * n * ld
    del hc, tgt, pick
    return {
        "two_layer": {"workload": "concepts30-items300-4k, 20% of known entries held out",
                      "train_steps": train_steps, "pred_sweeps": pred_sweeps, "replicas": 20,
                      "test_entries": int(len(lab)), "auc": round(a, 5), "predict_ms": round(t_pred, 3)},
        "hits_kernel": {"ms": round(t_hits, 4), "algorithmic_bytes": b_hits, "gbs": round(b_hits / t_hits / 1e6, 1),
                        "frac": round(b_hits / t_hits / 1e6 / HBM_PEAK_GBS, 4)},
    }


def m_study_run(dev, stream):
    """KL_avg-vs-time studies of the SAME replication factor (m_study_cfg) on
    the student network (identifiable: every node is observed half the time)
    and on the two-layer network (its concepts are never observed, so their
    states may swap labels and KL_avg against the generating CPTs need not
    fall; there the held-out AUC, which is label-invariant, tracks the
    sampler)."""
    return {"student-100k": m_study_cfg(2, dev, stream),
            "concepts30-items300-4k": m_study_cfg(4, dev, stream, heldout=0.2)}


def m_study_cfg(cfg, dev, stream, steps=200, checkpoints=(10, 25, 50, 100, 150, 200), heldout=None,
                pred_sweeps=20):
    """KL_avg (Sec. 5.1) of the sampled CPTs against the generator's true CPTs
    as a function of device time on workload cfg (Secs. 5.1 and 6 plot KL_avg
    against passes and time for m = 1, 2, 5, 20), for fixed m and for an
    annealed run (Sec. 3: m raised during sampling,
    here 1 -> 2 -> 5 -> 20 at equal step intervals with same_grow_replicas and
    a recount).  Each run takes `steps` SAME steps from the same start.
    With heldout (a fraction), that fraction of the known entries is held out
    of training (workloads.holdout), and at every checkpoint a prediction pass
    (Sec. 6: pred_sweeps frozen-CPT sweeps on a copy of the chains) scores the
    held-out entries; their AUC does not depend on how the sampler labels
    states that are never observed.  The prediction passes are not counted
    in the device time."""
    import numpy as np
    import torch

    import paper_1511_06416_amd as same
    from paper_1511_06416_amd import evaluate
    from workloads import make_workload

    from workloads import holdout
    base = make_workload(cfg, m=1, device=dev)
    net = base.net
    pptr, pidx, card = net.csr()
    ctx = same.same_create(pptr, pidx, card, base.alpha)
    ws = ctx.new_workspace(dev)
    off = ctx.cpt_off
    ld, nc = base.ld, base.n_cols
    obs = base.obs[0]
    target_np = tg = None
    if heldout:
        obs_train, target_np = holdout(base, 0, heldout)
        obs = torch.from_numpy(obs_train).to(dev)
        tg = torch.from_numpy(target_np).to(dev)

    def predict_auc(st, m, cpts):
        sc = st.clone()
        hits = torch.zeros((net.n, ld), dtype=torch.int32, device=dev)
        same.same_predict(ctx, sc, obs, cpts, tg, m, nc, ld, 0, base.seed, 1 << 20, pred_sweeps, hits, ws)
        torch.cuda.synchronize()
        scores, labels = evaluate.binary_scores(hits.cpu().numpy(), target_np, pred_sweeps * m)
        return evaluate.auc(scores, labels)

    def run(schedule):
        m = schedule(0)
        st = same.pack_states(base.states[0][:, :1, :].expand(-1, m, -1).contiguous())
        cpts = torch.from_numpy(base.init_theta).to(dev)
        mb = torch.zeros(ctx.cpt_total, dtype=torch.int32, device=dev)
        tot = torch.zeros(ctx.cpt_total, dtype=torch.int32, device=dev)
        same.same_init_latent(ctx, st, obs, m, nc, ld, 0, base.seed + 3)
        same.same_counts(ctx, st, m, nc, ld, mb, tot, ws)
        out, t_ms = [], 0.0
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        for s in range(steps):
            e0.record(stream)
            m2 = schedule(s)
            if m2 != m:  # anneal: more replicas, then the counts over all of them
                grown = torch.empty(same.state_shape(net.n, m2, ld), dtype=st.dtype, device=dev)
                same.same_grow_replicas(ctx, st, m, grown, m2, ld)
                st, m = grown, m2
                mb.zero_()
                tot.zero_()
                same.same_counts(ctx, st, m, nc, ld, mb, tot, ws)
            same.same_step(ctx, st, obs, cpts, m, nc, ld, 0, base.seed, s, mb, tot, s, ws)
            e1.record(stream)
            e1.synchronize()
            t_ms += e0.elapsed_time(e1)
            if s + 1 in checkpoints:
                kl = evaluate.kl_avg(base.true_theta, cpts.cpu().numpy(), off, net.card)
                rec = {"step": s + 1, "device_ms": round(t_ms, 2), "m": m, "kl_avg": round(kl, 5)}
                if heldout:
                    rec["heldout_auc"] = round(predict_auc(st, m, cpts), 5)
                out.append(rec)
        return out

    res = {}
    for m in (1, 2, 5, 20):
        res["m=%d" % m] = run(lambda s, m=m: m)
    res["annealed 1-2-5-20"] = run(lambda s: (1, 2, 5, 20)[min(3, s * 4 // steps)])
    ctx.close()
    what = "KL_avg against the generating CPTs"
    if heldout:
        what += ("; AUC of %d%% of the known entries held out, from %d frozen-CPT sweeps per checkpoint"
                 % (round(100 * heldout), pred_sweeps))
    return {"workload": "%s, %d columns, %.0f%% hidden; %s" % (base.name, nc, 100 * base.hidden, what),
            "runs": res}


def stream_timing(w, ctx, cpts, ws, dev, steps):
    """End-to-end out-of-core passes: every minibatch is copied from pinned host
    memory to the device, swept, counted and resampled, and copied back
    (same_stream_pass).  Reported beside the HBM-resident value, never as it."""
    import torch

    import paper_1511_06416_amd as same

    net = w.net
    host_ld = (w.n_cols + 3) // 4 * 4
    t0 = time.time()
    hs = torch.empty(same.state_shape(net.n, w.m, host_ld, ctx.state_bits), dtype=w.pk[0].dtype, pin_memory=True)
    ho = torch.empty((net.n, host_ld), dtype=torch.uint8, pin_memory=True)
    for b in range(w.M):
        c0, nc = b * w.nb, w.mb_cols(b)
        for i in range(net.n):
            hs[i, :, c0:c0 + nc, ...].copy_(w.pk[b][i, :, :nc, ...])
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
    state_bytes = float(net.n) * ((w.m + 3) // 4) * w.n_cols * (ctx.state_bits // 2)  # quads, padding included
    h2d = state_bytes + float(net.n) * w.n_cols
    log("streamed %d passes in %.3f s" % (steps, dt))
    # the same passes with the exponential moving sum of the counts (Sec. 4
    # footnote): no per-minibatch count storage, decay 1 - 1/M
    decay = 1.0 - 1.0 / w.M
    tot_e = torch.zeros(ctx.cpt_total, dtype=torch.float64, device=dev)
    cp_e = cpts.clone()
    same.same_stream_pass_ema(ctx, hs, ho, host_ld, w.n_cols, w.nb, w.m, cp_e, tot_e, decay, w.seed, 0,
                              same.SAME_STREAM_COUNTS_ONLY, slots, ws)
    torch.cuda.synchronize()
    t = time.perf_counter()
    for s in range(1, 1 + steps):
        same.same_stream_pass_ema(ctx, hs, ho, host_ld, w.n_cols, w.nb, w.m, cp_e, tot_e, decay, w.seed,
                                  100 + s, 0, slots, ws)
    torch.cuda.synchronize()
    dt_e = time.perf_counter() - t
    log("streamed %d moving-sum passes in %.3f s" % (steps, dt_e))
    del hs, ho
    compact = compact_stream_timing(w, ctx, cpts.clone(), ws, dev, steps)
    return {"value": round(ns / dt, 1), "unit": "node-samples/s", "passes": steps,
            "ms_per_pass": round(dt * 1e3 / steps, 2),
            "pcie_bytes_per_pass": {"h2d": h2d, "d2h": state_bytes},
            "pcie_gbs_each_way": {"h2d": round(h2d * steps / dt / 1e9, 1),
                                  "d2h": round(state_bytes * steps / dt / 1e9, 1)},
            "exponential_moving_sum": {"value": round(ns / dt_e, 1), "ms_per_pass": round(dt_e * 1e3 / steps, 2),
                                       "decay": round(decay, 6),
                                       "count_bytes_not_stored": int(w.M * ctx.cpt_total * 4)},
            "compact_host_state": compact}


def compact_stream_timing(w, ctx, cpts, ws, dev, steps):
    """Out-of-core passes with compact host state (same_stream_pass_compact):
    the known data (obs and observed values) stay on the device and only the
    replicas' latent states, compacted, cross PCIe each way.  The compact host
    array is cut from the benchmark's dense minibatches with torch (input
    preparation)."""
    import torch

    import paper_1511_06416_amd as same
    net = w.net
    n, m = net.n, w.m
    ld_dev = (w.n_cols + 3) // 4 * 4
    t0 = time.time()
    obs = torch.ones((n, ld_dev), dtype=torch.uint8, device=dev)
    data = torch.zeros((n, ld_dev), dtype=w.states[0].dtype, device=dev)
    for b in range(w.M):
        c0, nc = b * w.nb, w.mb_cols(b)
        obs[:, c0:c0 + nc] = w.obs[b][:, :nc]
        data[:, c0:c0 + nc] = w.states[b][:, 0, :nc]
    off, slot_bytes = same.same_stream_compact_layout(ctx, obs, ld_dev, w.n_cols, w.nb, m, ws)
    lat = torch.empty(int(off[-1]), dtype=w.states[0].dtype, pin_memory=True)
    for b in range(w.M):
        nc = w.mb_cols(b)
        st = w.states[b]
        for i in range(n):
            o0, o1 = int(off[b * n + i]), int(off[b * n + i + 1])
            if o1 == o0:
                continue
            cols = torch.nonzero(w.obs[b][i, :nc] == 0).flatten()
            lat[o0:o1].copy_(st[i].index_select(1, cols).reshape(-1))
    slots = torch.empty(slot_bytes, dtype=torch.uint8, device=dev)
    mb = torch.zeros((w.M, ctx.cpt_total), dtype=torch.int32, device=dev)
    tot = torch.zeros(ctx.cpt_total, dtype=torch.int32, device=dev)
    torch.cuda.synchronize()
    log("compact host state (%.1f GB) in %.1f s" % (lat.numel() * lat.element_size() / 1e9, time.time() - t0))
    same.same_stream_pass_compact(ctx, lat, off, obs, data, ld_dev, w.n_cols, w.nb, m, cpts, mb, tot, w.seed, 0,
                                  same.SAME_STREAM_COUNTS_ONLY, slots, ws)
    same.same_stream_pass_compact(ctx, lat, off, obs, data, ld_dev, w.n_cols, w.nb, m, cpts, mb, tot, w.seed, 0, 0,
                                  slots, ws)
    torch.cuda.synchronize()
    t = time.perf_counter()
    for s in range(1, 1 + steps):
        same.same_stream_pass_compact(ctx, lat, off, obs, data, ld_dev, w.n_cols, w.nb, m, cpts, mb, tot, w.seed,
                                      s, 0, slots, ws)
    torch.cuda.synchronize()
    dt = time.perf_counter() - t
    ns = float(n) * w.n_cols * m * steps
    moved = float(off[-1]) * lat.element_size()
    log("compact streamed %d passes in %.3f s" % (steps, dt))
    del lat, slots, obs, data
    return {"value": round(ns / dt, 1), "unit": "node-samples/s", "passes": steps,
            "ms_per_pass": round(dt * 1e3 / steps, 2),
            "pcie_bytes_per_pass": {"h2d": moved, "d2h": moved},
            "pcie_gbs_each_way": round(moved * steps / dt / 1e9, 1),
            "device_resident_known_data_bytes": 2 * n * ld_dev}


def cpu_baseline(w, cols, st, ob, steps):
    """The oracle (fp64, OpenMP over columns) on the first `cols` columns of
    minibatch 0 as generated: `steps` SAME steps, each one sweep, its counts
    and one Dirichlet resample."""
    import oracle

    import numpy as np
    net = w.net
    threads = len(os.sched_getaffinity(0))
    color = oracle.graph(net.parents, net.card)["color"]
    # a smaller sample for the one-thread rate, cut before the states change
    cols1 = min(cols, 10_000) // 4 * 4
    st1 = np.ascontiguousarray(st[:, :, :cols1])
    ob1 = np.ascontiguousarray(ob[:, :cols1])

    def run(st, ob, cols, steps, n_threads):
        theta = w.init_theta
        t = time.perf_counter()
        for s in range(steps):
            oracle.sweep(net.parents, net.card, theta, color, st, ob, w.m, cols, 0, w.seed, s,
                         n_threads=n_threads)
            cnt = oracle.counts(net.parents, net.card, st, w.m, cols, n_threads=n_threads)
            theta = oracle.dirichlet(net.parents, net.card, cnt, w.alpha, w.seed, s)
        return time.perf_counter() - t

    dt = run(st, ob, cols, steps, threads)
    ns = float(net.n) * cols * w.m * steps
    log("cpu baseline: %d columns x %d steps, %.2f s, %d threads" % (cols, steps, dt, threads))
    dt1 = run(st1, ob1, cols1, 1, 1) if cols1 > 0 else 0.0
    ns1 = float(net.n) * cols1 * w.m
    log("cpu baseline, one thread: %d columns x 1 step, %.2f s" % (cols1, dt1))
    return {"value": round(ns / dt, 1), "unit": "node-samples/s", "cores": threads,
            "kind": "oracle",
            "sample": "first %d columns of minibatch 0 (all %d nodes, m=%d), %d SAME steps (sweep + "
                      "counts + Dirichlet resample each), %.1f s" % (cols, net.n, w.m, steps, dt),
            "one_thread": None if dt1 <= 0 else {
                "value": round(ns1 / dt1, 1),
                "sample": "first %d columns of minibatch 0, 1 SAME step, %.1f s" % (cols1, dt1)}}


if __name__ == "__main__":
    main()
