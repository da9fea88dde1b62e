"""Benchmark: GDN-shaped speculative verify+commit on one MI355X.

One step = one speculative round of the whole hot path for every layer of
the workload: per layer one fused commit-and-verify call (the previous
round's accepted paths are committed into the state tile, the state is
written back once, the draft trees are verified from the committed tile and
the factor store is written).  Inputs are seeded synthetic tensors that are
already resident in HBM when the timed region starts.

Prints one JSON line: verified tree-nodes/s (one node = one draft token
through one layer, all heads), the achieved HBM bandwidth of the verify
kernel from its algorithmic bytes and HIP-event durations, and the fp64
oracle timed on the host cores on a bounded sample.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0  # MI355X HBM3E peak, GB/s

DEFAULT_WORKLOAD = "batched_tree_serving"
METRIC = "verified tree-nodes/sec + achieved HBM GB/s, GDN-shaped verify+commit"


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def algorithmic_bytes(cfg, pending_len, family="gdn"):
    """Bytes one fused verify call must move for one layer: the state once in
    and once out, the draft's q/k/v, the gates and betas the layer family
    reads, the parent row, the outputs, the factor store, and the pending
    records of the accepted paths."""
    B, H, dk, dv, n = cfg.batch, cfg.heads, cfg.d_k, cfg.d_v, cfg.n_nodes
    w = 2 if cfg.dtype == "bf16" else 4
    bnh = B * n * H
    gate = dk * 4 if family == "gla" else 4            # gate record (alpha, 1, or per-key gates)
    gin = {"gdn": 8, "deltanet": 4, "decay": 4, "gla": dk * 4}[family]  # gate and beta inputs read
    state = 2 * B * H * dk * dv * 4
    draft = bnh * (2 * dk * w + dv * w + gin) + B * n * 4
    out = bnh * dv * 4
    factors = bnh * (dk * w + dv * 4 + gate) + B * n * 4
    A = int(np.sum(pending_len))
    pend = A * H * (dk * w + dv * 4 + gate) + A * 4 + B * 4 * 2 + B * n * 4
    return state + draft + out + factors + pend


def graph_plan(steps, layers, max_launches=48):
    """(steps per captured graph, replays): an even number of steps per graph
    (the factor stores and inputs ping-pong between consecutive steps), as
    many as fit in about max_launches kernel launches, dividing the requested
    step count (rounded up to even) so that exactly that many are timed."""
    k = steps + (steps % 2)
    cap = max(2, (max_launches // max(layers, 1)) // 2 * 2)
    g = max(d for d in range(2, min(cap, k) + 1, 2) if k % d == 0)
    return g, k // g


def cpu_model() -> str:
    """The host CPU's model name (/proc/cpuinfo), or the platform's."""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    import platform
    return platform.processor() or platform.machine()


def _oracle_pass(oracle, cfg, r0, states, gates, family, layer, seqs=None):
    """One verify + commit of one layer of round r0 by the oracle, over all
    sequences or the first `seqs`."""
    sl = slice(None) if seqs is None else slice(0, seqs)
    a, b = gates[layer] if gates is not None else (r0.alpha[layer], r0.beta[layer])
    a = a[sl] if a is not None else None
    b = b[sl] if b is not None else None
    out, st = oracle.verify(states[layer][sl], r0.q32[layer][sl], r0.k32[layer][sl], r0.v32[layer][sl], a, b,
                            r0.parent[sl], family=family)
    S1, st2 = oracle.commit(states[layer][sl], r0.k32[layer][sl], r0.v32[layer][sl], a, b, r0.parent[sl],
                            r0.path[sl], r0.length[sl], family=family)
    assert (st == 0).all() and (st2 == 0).all()


def cpu_baseline(cfg, rounds, states, budget_s=10.0, gates=None, family="gdn", single_s=4.0, single_seqs=4):
    """The fp64 oracle (verify + commit by definition) on the host cores, on
    whole layers of the same workload, cycling through the layers until about
    budget_s of CPU time has passed; then single-threaded on a subset (the
    first `single_seqs` sequences of each layer, all heads) for about
    single_s.  gates: per layer (alpha, beta) inputs of the family."""
    import oracle

    r0 = rounds
    threads = oracle.num_threads()
    # one untimed pass first: the first touches of the fp64 working arrays
    # (page faults) are not the oracle's arithmetic
    _oracle_pass(oracle, cfg, r0, states, gates, family, 0)
    t0 = time.perf_counter()
    passes = 0
    while True:
        _oracle_pass(oracle, cfg, r0, states, gates, family, passes % cfg.layers)
        passes += 1
        if time.perf_counter() - t0 >= budget_s:
            break
    dt = time.perf_counter() - t0
    nodes = passes * cfg.batch * cfg.n_nodes
    # one thread on a subset: the same per-node work, so the rates compare
    seqs = min(single_seqs, cfg.batch)
    oracle.set_num_threads(1)
    try:
        t1 = time.perf_counter()
        sp = 0
        while True:
            _oracle_pass(oracle, cfg, r0, states, gates, family, sp % cfg.layers, seqs=seqs)
            sp += 1
            if time.perf_counter() - t1 >= single_s:
                break
        dt1 = time.perf_counter() - t1
    finally:
        oracle.set_num_threads(threads)
    single = sp * seqs * cfg.n_nodes / dt1
    return {"value": round(nodes / dt, 1), "unit": "nodes/s", "cores": threads, "kind": "oracle",
            "cpu_model": cpu_model(),
            "sample": "%d layer passes over the %d layers of the %s workload (all %d sequences x %d heads each), "
                      "verify + commit of one round, %.1f s on %d threads" % (passes, cfg.layers, cfg.name, cfg.batch,
                                                                               cfg.heads, dt, threads),
            "single_thread": {"value": round(single, 1), "unit": "nodes/s",
                              "sample": "%d layer passes over the first %d sequences (x %d heads) of each layer, "
                                        "verify + commit, %.1f s on 1 thread" % (sp, seqs, cfg.heads, dt1)},
            "thread_scaling": round((nodes / dt) / single, 2)}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default=DEFAULT_WORKLOAD)
    ap.add_argument("--route", default="auto", choices=["auto", "serial", "parallel", "hybrid"])
    ap.add_argument("--family", default="gdn", choices=["gdn", "deltanet", "decay", "gla"],
                    help="layer family of the recurrent core (gdn: gated delta rule, the headline; deltanet: "
                         "no decay; decay: scalar decay without the delta rule; gla: per-key gates)")
    ap.add_argument("--separate", action="store_true",
                    help="time the separate route (verify, then standalone commit) instead of the fused one")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-extra", action="store_true",
                    help="default run only: skip the other batch >= 64 workloads (64-node trees and the 1-node "
                         "decode chain at batch 256)")
    ap.add_argument("--no-copy-ceiling", action="store_true",
                    help="default run only: skip the measured copy ceiling")
    ap.add_argument("--no-graph", dest="graph", action="store_false",
                    help="launch eagerly from Python with HIP events around every launch")
    ap.add_argument("--traffic-json", default=os.path.join(ROOT, "profiles", "traffic.json"),
                    help="measured HBM bytes per launch from rocprofv3 counters (if present)")
    ap.add_argument("--study", default=None, choices=["tree-shapes", "fused-commit"],
                    help="tree-shapes: root-to-leaf replay, serial, parallel and hybrid verification of "
                         "synthetic top-k proposal trees at the paper's target shape (8 heads, d_k = d_v = 256, "
                         "batch 1); "
                         "fused-commit: fused commit-and-verify vs verify plus standalone commit for accepted "
                         "lengths 1..8 at verify length 4 (the same shape)")
    ap.add_argument("--op", default="gdn", choices=["gdn", "conv", "prune", "commit"],
                    help="gdn: the recurrent-state verify+commit (the headline); conv: the layer's short "
                         "causal convolution with its conv-state commit, on the same drafts; prune: draft "
                         "pruning and packing of 64-candidate rollouts down to the workload's tree size; "
                         "commit: the standalone accepted-path commit alone, over rotating states of at least "
                         "1.5 GiB in total (cold: no verification of the same state right before it)")
    args = ap.parse_args()

    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py runs on exactly one GPU: the library has no multi-GPU path "
              "(every (batch, head) unit is independent: a sharded run would give each GPU whole sequences "
              "or a share of the heads, with no exchange inside verification or commit).",
              file=sys.stderr)
        sys.exit(2)

    import torch

    from paper_2607_16673_amd import binding as B
    from paper_2607_16673_amd import inputs

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    B.lib()
    if args.study == "tree-shapes":
        return study_tree_shapes(args, torch, B, inputs, dev)
    if args.study == "fused-commit":
        return study_fused_commit(args, torch, B, inputs, dev)
    cfg = inputs.config(args.workload)
    if args.op == "conv":
        return run_conv(args, cfg, torch, B, inputs, dev)
    if args.op == "prune":
        return run_prune(args, cfg, torch, B, inputs, dev)
    if args.op == "commit":
        return run_commit(args, cfg, torch, B, inputs, dev)
    res = time_gdn(args, cfg, torch, B, inputs, dev, steps=args.steps, warmup=args.warmup,
                   keep_inputs=not args.no_cpu_baseline)
    fam = args.family
    topo = "chain" if cfg.chain else "tree"
    traffic, kernel = lookup_traffic(args, cfg, fam)
    roof = {"bound": "hbm", "achieved": round(res["achieved"], 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
            "frac": round(res["achieved"] / HBM_PEAK_GBS, 4), "traffic": traffic,
            "kernel": kernel or ("sla verify (%s route)%s" % (args.route, " + sla commit" if args.separate else "")),
            "algorithmic_bytes_per_launch": int(res["bytes_launch"]), "avg_launch_ms": round(res["v_ms"], 5)}
    line = {
        "metric": METRIC, "value": round(res["value"], 1), "unit": "nodes/s", "n_gpus": 1, "steps": res["steps"],
        "warmup": args.warmup, "ms_per_step": round(res["ms_per_step"], 4), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None,
        # bf16 q/k/v (the paper's activation precision) against an fp32 state
        # and fp32 gates; the contractions run on the matrix cores with the
        # fp32 operands split into bf16 hi + lo parts, accumulated in fp32
        "dtype": "bf16 q/k/v, f32 state" if cfg.dtype == "bf16" else "f32", "data": "synthetic",
        "config": {"workload": cfg.name, "batch": cfg.batch, "heads": cfg.heads, "d_k": cfg.d_k,
                   "d_v": cfg.d_v, "nodes_per_tree": cfg.n_nodes, "topology": topo,
                   "max_depth": cfg.max_depth, "max_branch": cfg.max_branch, "layers": cfg.layers,
                   "qkv_dtype": cfg.dtype, "state_dtype": "f32", "route": args.route,
                   "commit": "separate" if args.separate else "fused", "family": fam,
                   "parallelism": "single-gpu",
                   "launch": "hip graph" if args.graph else "eager"},
        "hbm_gbps": round(res["achieved"], 1),
        # one token through every layer of the workload (one layer's node is `value`'s unit)
        "tokens_per_s": round(res["tokens_per_s"], 1),
        "roofline": roof,
    }
    if res.get("c_ms") is not None:
        line["commit_avg_launch_ms"] = round(res["c_ms"], 5)
    default_run = (args.workload == DEFAULT_WORKLOAD and fam == "gdn" and args.route == "auto"
                   and not args.separate and args.graph)
    if default_run and not args.no_copy_ceiling:
        log("bench: copy ceiling")
        cc = copy_ceiling(torch, dev)
        line["copy_ceiling"] = cc
        roof["frac_of_copy_ceiling"] = round(res["achieved"] / cc["gbps"], 4)
    if default_run and not args.no_extra:
        # the other batch >= 64 workloads: 64-node trees and the 1-node decode
        # chain at batch 256 (one layer each, same fused route)
        extra = {}
        for name in EXTRA_WORKLOADS:
            xc = inputs.config(name)
            r = time_gdn(args, xc, torch, B, inputs, dev, steps=20, warmup=args.warmup, keep_inputs=False)
            t, _ = lookup_traffic(args, xc, fam)
            e = {"nodes_per_s": round(r["value"], 1), "avg_launch_ms": round(r["v_ms"], 5),
                 "algorithmic_bytes_per_launch": int(r["bytes_launch"]), "achieved_gbps": round(r["achieved"], 1),
                 "frac": round(r["achieved"] / HBM_PEAK_GBS, 4), "traffic": t, "steps": r["steps"],
                 "config": {"batch": xc.batch, "heads": xc.heads, "d_k": xc.d_k, "d_v": xc.d_v,
                            "nodes_per_tree": xc.n_nodes, "topology": "chain" if xc.chain else "tree",
                            "max_depth": xc.max_depth, "max_branch": xc.max_branch, "layers": xc.layers}}
            if "copy_ceiling" in line:
                e["frac_of_copy_ceiling"] = round(r["achieved"] / line["copy_ceiling"]["gbps"], 4)
            extra[name] = e
            log("bench: %s %.1f us per launch, %.1f GB/s (%.1f%% of 8 TB/s)"
                % (name, r["v_ms"] * 1e3, r["achieved"], 100 * r["achieved"] / HBM_PEAK_GBS))
            del r
            torch.cuda.empty_cache()
        line["workloads_batch_ge_64"] = extra
    if not args.no_cpu_baseline:
        log("bench: oracle CPU baseline")
        line["cpu_baseline"] = cpu_baseline(cfg, res["rnd"], res["states_np"], gates=res["gates"], family=fam)
    print(json.dumps(line), flush=True)


EXTRA_WORKLOADS = ["large_batch_tree64", "large_batch_chain1"]


def lookup_traffic(args, cfg, fam):
    """(HBM bytes per launch from the counters, counted kernel) for this
    workload, or (None, None) when none were taken on the current sources."""
    if not os.path.exists(args.traffic_json):
        return None, None
    with open(args.traffic_json) as f:
        tj = json.load(f)
    key = "%s/%s/%s" % (cfg.name, args.route, "separate" if args.separate else "fused")
    if fam != "gdn":
        key += "/" + fam
    # counters taken on other library sources no longer describe this kernel
    from paper_2607_16673_amd.traffic import source_digest
    if key in tj and tj[key].get("source_sha256") == source_digest(tj[key].get("kernel", "verify_tile_kernel")):
        return tj[key].get("bytes_per_launch"), tj[key].get("kernel")
    return None, None


def copy_ceiling(torch, dev, total_bytes=3 << 30, buffers=6, reps=5):
    """A measured ceiling for streaming the state: plain copies (torch's
    elementwise copy) and in-place read-modify-write passes (torch's x *= 1)
    over `buffers` rotating fp32 buffers of total_bytes / buffers each, far
    beyond the 256 MB last-level cache, launched back to back from a HIP
    graph.  GB/s counts every byte read and written once."""
    n = total_bytes // buffers // 4
    src = [torch.empty(n, dtype=torch.float32, device=dev).normal_() for _ in range(buffers)]
    dst = [torch.empty_like(x) for x in src]

    def span(launch):
        launch()
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        sc = torch.cuda.Stream(dev)
        sc.wait_stream(torch.cuda.current_stream(dev))
        with torch.cuda.stream(sc):
            with torch.cuda.graph(g, stream=sc):
                launch()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        cur = torch.cuda.current_stream(dev)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(cur)
        for _ in range(reps):
            g.replay()
        e1.record(cur)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / (reps * buffers)  # ms per buffer pass

    def copy_all():
        for d, x in zip(dst, src):
            d.copy_(x)

    def rmw_all():
        for x in src:
            x.mul_(1.0)

    t_copy = span(copy_all)
    t_rmw = span(rmw_all)
    per = n * 4 * 2
    g_copy = per / (t_copy * 1e-3) / 1e9
    g_rmw = per / (t_rmw * 1e-3) / 1e9
    del src, dst
    torch.cuda.empty_cache()
    return {"gbps": round(max(g_copy, g_rmw), 1), "copy_gbps": round(g_copy, 1), "in_place_rmw_gbps": round(g_rmw, 1),
            "frac_of_peak": round(max(g_copy, g_rmw) / HBM_PEAK_GBS, 4), "bytes_per_pass": int(per),
            "kernel": "torch elementwise copy_ and in-place mul_(1.0), %d rotating %d MiB fp32 buffers, HIP graph"
                      % (buffers, n * 4 >> 20)}


def time_gdn(args, cfg, torch, B, inputs, dev, steps, warmup, keep_inputs=True):
    """Time `steps` speculative rounds of one GDN workload (per layer one fused
    commit-and-verify, or with --separate a verify then a standalone commit).
    Returns a dict of measurements (and the host inputs when keep_inputs)."""
    fam = args.family
    topo = "chain" if cfg.chain else "tree"
    log("bench: generating %s (%d layers)" % (cfg.name, cfg.layers))
    rnd = inputs.draw_round(cfg, 0)
    states_np = [inputs.draw_state(cfg, l) for l in range(cfg.layers)]

    def act(x):
        if cfg.dtype == "bf16":
            return torch.from_numpy(np.ascontiguousarray(x).view(np.int16)).view(torch.bfloat16).to(dev)
        return torch.from_numpy(np.ascontiguousarray(x)).to(dev)

    adt = torch.bfloat16 if cfg.dtype == "bf16" else torch.float32
    gates = [inputs.family_gates(cfg, rnd, l, fam, layer=l) for l in range(cfg.layers)]

    def dev_or_none(x):
        return torch.from_numpy(x).to(dev) if x is not None else None

    layers = []
    for l in range(cfg.layers):
        layers.append(dict(q=act(rnd.q[l]), k=act(rnd.k[l]), v=act(rnd.v[l]),
                           alpha=dev_or_none(gates[l][0]), beta=dev_or_none(gates[l][1])))
    parent = torch.from_numpy(rnd.parent).to(dev)
    path = torch.from_numpy(rnd.path).to(dev)
    length = torch.from_numpy(rnd.length).to(dev)
    states = [torch.from_numpy(s).to(dev) for s in states_np]
    fshape = (cfg.batch, cfg.n_nodes, cfg.heads, cfg.d_k, cfg.d_v)
    fstores = [[B.Factors.empty(*fshape, adt, dev, family=fam) for _ in range(cfg.layers)] for _ in range(2)]
    outs = [torch.empty(cfg.batch, cfg.n_nodes, cfg.heads, cfg.d_v, dtype=torch.float32, device=dev)
            for _ in range(cfg.layers)]
    status = torch.zeros(cfg.batch, dtype=torch.int32, device=dev)
    stream = torch.cuda.current_stream(dev)

    step_no = [0]

    def step(events=None):
        s = step_no[0]
        cur, prev = fstores[s % 2], fstores[(s + 1) % 2]
        for l in range(cfg.layers):
            L = layers[l]
            if events is not None:
                events.append(torch.cuda.Event(enable_timing=True))
                events[-1].record(stream)
            if args.separate:
                B.sla_verify(states[l], L["q"], L["k"], L["v"], L["alpha"], L["beta"], parent, outs[l], cur[l],
                             status=status, topology=topo, route=args.route, family=fam)
                if events is not None:
                    events.append(torch.cuda.Event(enable_timing=True))
                    events[-1].record(stream)
                B.sla_commit(states[l], cur[l], path, length, status=status, family=fam)
            else:
                pend = (prev[l], path, length) if s > 0 else None
                B.sla_verify(states[l], L["q"], L["k"], L["v"], L["alpha"], L["beta"], parent, outs[l], cur[l],
                             pending=pend, status=status, topology=topo, route=args.route, family=fam)
            if events is not None:
                events.append(torch.cuda.Event(enable_timing=True))
                events[-1].record(stream)
        step_no[0] += 1

    log("bench: warmup %d" % warmup)
    for _ in range(max(warmup, 2)):
        step()
    torch.cuda.synchronize()
    assert int(status.abs().max()) == 0, "device reported a data error"

    if args.graph:
        # One graph holds an even number of consecutive steps (the factor
        # stores ping-pong), replayed back to back: no host work between
        # kernel launches.
        gsteps, reps = graph_plan(steps, cfg.layers)
        if step_no[0] % 2:
            step()
        g = torch.cuda.CUDAGraph()
        s_cap = torch.cuda.Stream(dev)
        s_cap.wait_stream(stream)
        with torch.cuda.stream(s_cap):
            with torch.cuda.graph(g, stream=s_cap):
                for _ in range(gsteps):
                    step()
        torch.cuda.synchronize()
        for _ in range(2):
            g.replay()
        torch.cuda.synchronize()
        steps = gsteps * reps
        log("bench: timing %d steps (graph replays)" % steps)
        cur = torch.cuda.current_stream(dev)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        e0.record(cur)
        for _ in range(reps):
            g.replay()
        e1.record(cur)
        torch.cuda.synchronize()
        t1 = time.perf_counter()
        elapsed = t1 - t0
        # launches in a graph run back to back: the mean duration per layer
        # (one verify, or with --separate one verify plus one commit) is the
        # event-timed replay span over the layers it holds
        vdur = [e0.elapsed_time(e1) / (steps * cfg.layers)]
        cdur = []
    else:
        log("bench: timing %d steps" % steps)
        events = []
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(steps):
            step(events)
        torch.cuda.synchronize()
        t1 = time.perf_counter()
        elapsed = t1 - t0
        # verify-kernel durations from the HIP events bracketing each launch
        if args.separate:
            per = 3
            vdur = [events[i].elapsed_time(events[i + 1]) for i in range(0, len(events), per)]
            cdur = [events[i + 1].elapsed_time(events[i + 2]) for i in range(0, len(events), per)]
        else:
            vdur = [events[i].elapsed_time(events[i + 1]) for i in range(0, len(events), 2)]
            cdur = []
    assert int(status.abs().max()) == 0, "device reported a data error"
    ms_per_step = 1e3 * elapsed / steps
    # per layer: the fused call, or with --separate the verify (state read
    # once) plus the standalone commit (state read and written once more)
    v_ms = float(np.mean(vdur)) + (float(np.mean(cdur)) if cdur else 0.0)
    bytes_launch = algorithmic_bytes(cfg, rnd.length, fam)
    if args.separate:
        bytes_launch += cfg.batch * cfg.heads * cfg.d_k * cfg.d_v * 4
    achieved = bytes_launch / (v_ms * 1e-3) / 1e9
    nodes = cfg.batch * cfg.n_nodes * cfg.layers * steps
    res = {"value": nodes / elapsed, "steps": steps, "ms_per_step": ms_per_step, "v_ms": v_ms,
           "c_ms": float(np.mean(cdur)) if cdur else None, "bytes_launch": bytes_launch, "achieved": achieved,
           "tokens_per_s": cfg.batch * cfg.n_nodes * steps / elapsed}
    if keep_inputs:
        res.update(rnd=rnd, states_np=states_np, gates=gates)
    return res


def conv_algorithmic_bytes(cfg, D, K, pending_len, n_prev):
    """Bytes one fused conv call must move for one layer: the draft inputs
    once in, the outputs once out, the conv state once in and once out, the
    weights, the parent row, and of each pending path only the last K-1
    accepted rows (plus the path, its parent row and length)."""
    B, n = cfg.batch, cfg.n_nodes
    w = 2 if cfg.dtype == "bf16" else 4
    rows = int(np.sum(np.minimum(pending_len, K - 1)))
    return (2 * B * n * D * w + 2 * B * (K - 1) * D * 4 + D * K * 4 + B * n * 4
            + rows * D * w + B * n_prev * 4 * 2 + B * 4)


def conv_cpu_baseline(cfg, topo, xs32, Cs, ws, budget_s=10.0):
    """The fp64 oracle's convolution and conv-state commit on whole layers of
    the same workload, cycling through the layers for about budget_s."""
    import oracle

    parent, path, length = topo
    t0 = time.perf_counter()
    passes = 0
    while True:
        layer = passes % cfg.layers
        y, st = oracle.conv_verify(Cs[layer], xs32[layer], ws[layer], None, parent)
        C1, st2 = oracle.conv_commit(Cs[layer], xs32[layer], parent, path, length)
        assert (st == 0).all() and (st2 == 0).all()
        passes += 1
        if time.perf_counter() - t0 >= budget_s:
            break
    dt = time.perf_counter() - t0
    return {"value": passes * cfg.batch * cfg.n_nodes / dt, "unit": "nodes/s", "cores": oracle.num_threads(),
            "kind": "oracle",
            "sample": "%d layer passes over the %d layers of the %s workload (all %d sequences, %d channels "
                      "each), convolution + conv-state commit of one round, %.1f s"
                      % (passes, cfg.layers, cfg.name, cfg.batch, xs32[0].shape[2], dt)}


def run_conv(args, cfg, torch, B, inputs, dev):
    """Timed steps of the short causal convolution: per layer one fused
    sla_conv_verify with the previous round's accepted rows pending."""
    D, K = inputs.conv_channels(cfg), inputs.CONV_KERNEL
    log("bench: generating %s conv inputs (%d layers, %d channels)" % (cfg.name, cfg.layers, D))
    parent_np, path_np, length_np = inputs.draw_topology(cfg, 0)
    parent = torch.from_numpy(parent_np).to(dev)
    path = torch.from_numpy(path_np).to(dev)
    length = torch.from_numpy(length_np).to(dev)

    def act(x):
        if cfg.dtype == "bf16":
            return torch.from_numpy(np.ascontiguousarray(x).view(np.int16)).view(torch.bfloat16).to(dev)
        return torch.from_numpy(np.ascontiguousarray(x)).to(dev)

    xs, xs32, Cs, ws = [], [], [], []
    for l in range(cfg.layers):
        pair = []
        for r in range(2):
            x, x32 = inputs.draw_conv_x(cfg, l, r)
            pair.append(act(x))
            if r == 0:
                xs32.append(x32)
        xs.append(pair)
        Cs.append(inputs.draw_conv_state(cfg, l))
        ws.append(inputs.draw_conv_weight(cfg, l))
    conv_states = [torch.from_numpy(c).to(dev) for c in Cs]
    weights = [torch.from_numpy(w).to(dev) for w in ws]
    ys = [torch.empty_like(xs[l][0]) for l in range(cfg.layers)]
    status = torch.zeros(cfg.batch, dtype=torch.int32, device=dev)
    step_no = [0]

    def step():
        s = step_no[0]
        for l in range(cfg.layers):
            pend = (xs[l][(s + 1) % 2], parent, path, length) if s > 0 else None
            B.sla_conv_verify(conv_states[l], xs[l][s % 2], weights[l], parent, ys[l], pending=pend,
                              status=status)
        step_no[0] += 1

    log("bench: warmup %d" % args.warmup)
    for _ in range(max(args.warmup, 2)):
        step()
    if step_no[0] % 2:
        step()
    torch.cuda.synchronize()
    assert int(status.abs().max()) == 0, "device reported a data error"
    gsteps, reps = graph_plan(args.steps, cfg.layers)
    g = torch.cuda.CUDAGraph()
    s_cap = torch.cuda.Stream(dev)
    s_cap.wait_stream(torch.cuda.current_stream(dev))
    with torch.cuda.stream(s_cap):
        with torch.cuda.graph(g, stream=s_cap):
            for _ in range(gsteps):
                step()
    torch.cuda.synchronize()
    for _ in range(2):
        g.replay()
    torch.cuda.synchronize()
    steps = gsteps * reps
    log("bench: timing %d conv steps (graph replays)" % steps)
    cur = torch.cuda.current_stream(dev)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    e0.record(cur)
    for _ in range(reps):
        g.replay()
    e1.record(cur)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    assert int(status.abs().max()) == 0, "device reported a data error"
    v_ms = e0.elapsed_time(e1) / (steps * cfg.layers)
    bytes_launch = conv_algorithmic_bytes(cfg, D, K, length_np, cfg.n_nodes)
    achieved = bytes_launch / (v_ms * 1e-3) / 1e9
    topo = "chain" if cfg.chain else "tree"
    line = {
        "metric": METRIC, "value": round(cfg.batch * cfg.n_nodes * cfg.layers * steps / elapsed, 1),
        "unit": "nodes/s", "n_gpus": 1, "steps": steps, "warmup": args.warmup,
        "ms_per_step": round(1e3 * elapsed / steps, 4), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "f32", "data": "synthetic",
        "config": {"workload": cfg.name, "op": "short causal conv (K=%d, SiLU) + conv-state commit" % K,
                   "batch": cfg.batch, "channels": D, "nodes_per_tree": cfg.n_nodes, "topology": topo,
                   "layers": cfg.layers, "x_dtype": cfg.dtype, "conv_state_dtype": "f32", "commit": "fused",
                   "parallelism": "single-gpu", "launch": "hip graph"},
        "hbm_gbps": round(achieved, 1),
        "roofline": {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": None, "kernel": "conv_verify_kernel",
                     "algorithmic_bytes_per_launch": int(bytes_launch), "avg_launch_ms": round(v_ms, 5)},
    }
    if os.path.exists(args.traffic_json):
        with open(args.traffic_json) as f:
            tj = json.load(f)
        key = "%s/conv/fused" % cfg.name
        from paper_2607_16673_amd.traffic import source_digest
        if key in tj and tj[key].get("source_sha256") == source_digest(tj[key].get("kernel", "conv_verify_kernel")):
            line["roofline"]["traffic"] = tj[key].get("bytes_per_launch")
    if not args.no_cpu_baseline:
        log("bench: oracle CPU baseline (conv)")
        line["cpu_baseline"] = conv_cpu_baseline(cfg, (parent_np, path_np, length_np), xs32, Cs, ws)
    print(json.dumps(line), flush=True)


def run_commit(args, cfg, torch, B, inputs, dev, min_bytes=3 << 29):
    """Timed standalone commits (sla_commit) of the workload's accepted
    paths, one per state, over max(layers, enough states for min_bytes)
    rotating states, so that no state is in the last-level cache when its
    commit starts and none was just read by a verification.  The factor
    records come from one untimed verification per state."""
    state_bytes = cfg.batch * cfg.heads * cfg.d_k * cfg.d_v * 4
    nst = max(cfg.layers, -(-min_bytes // state_bytes))
    fam = args.family
    log("bench: generating %s (%d rotating states of %d MiB)" % (cfg.name, nst, state_bytes >> 20))
    rnd = inputs.draw_round(cfg, 0, layers=[0])
    adt = torch.bfloat16 if cfg.dtype == "bf16" else torch.float32

    def act(x):
        if cfg.dtype == "bf16":
            return torch.from_numpy(np.ascontiguousarray(x).view(np.int16)).view(torch.bfloat16).to(dev)
        return torch.from_numpy(np.ascontiguousarray(x)).to(dev)

    a_np, b_np = inputs.family_gates(cfg, rnd, 0, fam, layer=0)
    q, k, v = act(rnd.q[0]), act(rnd.k[0]), act(rnd.v[0])
    a = torch.from_numpy(a_np).to(dev) if a_np is not None else None
    bt = torch.from_numpy(b_np).to(dev) if b_np is not None else None
    parent = torch.from_numpy(rnd.parent).to(dev)
    path = torch.from_numpy(rnd.path).to(dev)
    length = torch.from_numpy(rnd.length).to(dev)
    S0 = torch.from_numpy(inputs.draw_state(cfg, 0)).to(dev)
    states = [S0.clone() for _ in range(nst)]
    del S0
    f = B.Factors.empty(cfg.batch, cfg.n_nodes, cfg.heads, cfg.d_k, cfg.d_v, adt, dev, family=fam)
    out = torch.empty(cfg.batch, cfg.n_nodes, cfg.heads, cfg.d_v, dtype=torch.float32, device=dev)
    status = torch.zeros(cfg.batch, dtype=torch.int32, device=dev)
    B.sla_verify(states[0], q, k, v, a, bt, parent, out, f, status=status,
                 topology="chain" if cfg.chain else "tree", family=fam)

    def step():
        for st in states:
            B.sla_commit(st, f, path, length, status=status, family=fam)

    for _ in range(max(args.warmup, 1)):
        step()
    torch.cuda.synchronize()
    assert int(status.abs().max()) == 0, "device reported a data error"
    reps = max(1, args.steps)
    g = torch.cuda.CUDAGraph()
    s_cap = torch.cuda.Stream(dev)
    s_cap.wait_stream(torch.cuda.current_stream(dev))
    with torch.cuda.stream(s_cap):
        with torch.cuda.graph(g, stream=s_cap):
            step()
    torch.cuda.synchronize()
    g.replay()
    torch.cuda.synchronize()
    cur = torch.cuda.current_stream(dev)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0 = time.perf_counter()
    e0.record(cur)
    for _ in range(reps):
        g.replay()
    e1.record(cur)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    assert int(status.abs().max()) == 0, "device reported a data error"
    c_ms = e0.elapsed_time(e1) / (reps * nst)
    w = 2 if cfg.dtype == "bf16" else 4
    gate = cfg.d_k * 4 if fam == "gla" else 4
    A = int(np.sum(rnd.length))
    bytes_launch = (2 * state_bytes + A * cfg.heads * (cfg.d_k * w + cfg.d_v * 4 + gate)
                    + cfg.batch * cfg.n_nodes * 4 * 2 + cfg.batch * 4)
    achieved = bytes_launch / (c_ms * 1e-3) / 1e9
    line = {
        "metric": "accepted-path commits/sec (standalone, cold states)",
        "value": round(cfg.batch * reps * nst / elapsed, 1), "unit": "sequence-layers/s", "n_gpus": 1,
        "steps": reps, "warmup": args.warmup, "ms_per_step": round(1e3 * elapsed / reps, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "f32 state",
        "data": "synthetic",
        "config": {"workload": cfg.name, "op": "standalone commit", "batch": cfg.batch, "heads": cfg.heads,
                   "d_k": cfg.d_k, "d_v": cfg.d_v, "rotating_states": nst, "state_mib": state_bytes >> 20,
                   "mean_accepted": round(float(np.mean(rnd.length)), 3), "family": fam,
                   "parallelism": "single-gpu", "launch": "hip graph"},
        "roofline": {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": None, "kernel": "commit_kernel",
                     "algorithmic_bytes_per_launch": int(bytes_launch), "avg_launch_ms": round(c_ms, 5)},
    }
    print(json.dumps(line), flush=True)


def run_prune(args, cfg, torch, B, inputs, dev, n_cand=64, tau=3.0):
    """Timed steps of draft pruning and packing: per step (one speculative
    round) one sla_prune over every sequence's 64-candidate rollout, margin
    tau and the workload's tree size as the budget."""
    T = cfg.n_nodes
    par_np, lp_np = inputs.draw_rollouts(cfg, 0, n_cand=n_cand)
    par = torch.from_numpy(par_np).to(dev)
    lp = torch.from_numpy(lp_np).to(dev)
    out = {}

    def step():
        out.update(B.sla_prune(par, lp, tau, T))

    for _ in range(max(args.warmup, 2)):
        step()
    torch.cuda.synchronize()
    assert int(out["status"].abs().max()) == 0
    gsteps, reps = graph_plan(args.steps, 1)
    g = torch.cuda.CUDAGraph()
    s_cap = torch.cuda.Stream(dev)
    s_cap.wait_stream(torch.cuda.current_stream(dev))
    with torch.cuda.stream(s_cap):
        with torch.cuda.graph(g, stream=s_cap):
            for _ in range(gsteps):
                step()
    torch.cuda.synchronize()
    g.replay()
    torch.cuda.synchronize()
    steps = gsteps * reps
    cur = torch.cuda.current_stream(dev)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0 = time.perf_counter()
    e0.record(cur)
    for _ in range(reps):
        g.replay()
    e1.record(cur)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    v_ms = e0.elapsed_time(e1) / steps
    kept = float(out["count"].float().mean())
    bytes_launch = cfg.batch * n_cand * (4 + 4 + 4 + 4) + cfg.batch * 8
    achieved = bytes_launch / (v_ms * 1e-3) / 1e9
    line = {
        "metric": "pruned draft sequences/sec", "value": round(cfg.batch * steps / elapsed, 1),
        "unit": "sequences/s", "n_gpus": 1, "steps": steps, "warmup": args.warmup,
        "ms_per_step": round(1e3 * elapsed / steps, 4), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "f32", "data": "synthetic",
        "config": {"workload": cfg.name, "op": "draft pruning + packing", "batch": cfg.batch,
                   "candidates": n_cand, "rollout": "beam top-4", "tau": tau, "budget": T,
                   "mean_kept": round(kept, 2), "parallelism": "single-gpu", "launch": "hip graph"},
        "roofline": {"bound": "hbm", "achieved": round(achieved, 2), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(achieved / HBM_PEAK_GBS, 6), "traffic": None, "kernel": "prune_kernel",
                     "algorithmic_bytes_per_launch": int(bytes_launch), "avg_launch_ms": round(v_ms, 5)},
    }
    if not args.no_cpu_baseline:
        from oracle import prune as P
        t0 = time.perf_counter()
        done = 0
        while time.perf_counter() - t0 < 10.0:
            b = done % cfg.batch
            keep, q, st = P.prune(par_np[b], lp_np[b], tau, T)
            P.pack(par_np[b], keep)
            done += 1
        dt = time.perf_counter() - t0
        line["cpu_baseline"] = {"value": round(done / dt, 1), "unit": "sequences/s", "cores": 1, "kind": "oracle",
                                "sample": "%d sequences of the rollout set, pruned and packed one by one, %.1f s"
                                          % (done, dt)}
    print(json.dumps(line), flush=True)


def study_tree_shapes(args, torch, B, inputs, dev, trees_per_shape=8, reps=20):
    """Per proposal shape of the paper's tree-verification table (top-k,
    configured depth, nodes): mean latency of verifying one synthetic
    proposal tree (a top-k rollout pruned to the node budget; batch 1, 8
    heads, d_k = d_v = 256, bf16 activations, fp32 state, no pending commit)
    by root-to-leaf replay, the serial, parallel and hybrid routes; each
    timed as `reps` replays of a HIP graph holding ten repetitions of one
    tree's launches (per-tree time = total / (reps x 10), the gaps between
    kernels included).  Also checks that the four routes agree."""
    from paper_2607_16673_amd import study

    H, dk, dv = 8, 256, 256
    rng = np.random.default_rng(4242)
    rows = []

    def timed(launch, per_graph=10):
        launch()
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        sc = torch.cuda.Stream(dev)
        sc.wait_stream(torch.cuda.current_stream(dev))
        with torch.cuda.stream(sc):
            with torch.cuda.graph(g, stream=sc):
                for _ in range(per_graph):
                    launch()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        cur = torch.cuda.current_stream(dev)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(cur)
        for _ in range(reps):
            g.replay()
        e1.record(cur)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) * 1e3 / (reps * per_graph)  # us per tree

    for si, (k, depth, n) in enumerate(study.TREE_SHAPES):
        t = {r: [] for r in study.ROUTES}
        worst = 0.0
        shape_stats = []
        for ti in range(trees_per_shape):
            par = study.proposal_tree(rng, k, depth, n)
            topo = B.sla_topology_host(par)
            shape_stats.append((topo["max_depth"], int((par == -1).sum()), len(study.root_to_leaf_paths(par))))
            d = study.Draft(torch, dev, par, H, dk, dv, seed=100 * si + ti)
            for route in study.ROUTES:
                t[route].append(timed(lambda: d.launch(route)))
            ref = d.outputs("serial")
            scale = np.max(np.abs(ref))
            for route in ["r2l", "parallel", "hybrid"]:
                worst = max(worst, float(np.max(np.abs(d.outputs(route) - ref)) / scale))
            del d
        mean = {r: float(np.mean(t[r])) for r in study.ROUTES}
        st = np.array(shape_stats)
        row = {"top_k": k, "config_depth": depth, "nodes": n, "r2l_us": round(mean["r2l"], 2),
               "serial_x": round(mean["r2l"] / mean["serial"], 2),
               "parallel_x": round(mean["r2l"] / mean["parallel"], 2),
               "hybrid_x": round(mean["r2l"] / mean["hybrid"], 2),
               "hybrid_over_serial": round(mean["serial"] / mean["hybrid"], 2),
               "serial_us": round(mean["serial"], 2), "parallel_us": round(mean["parallel"], 2),
               "hybrid_us": round(mean["hybrid"], 2),
               "mean_depth": round(float(st[:, 0].mean()), 2), "mean_roots": round(float(st[:, 1].mean()), 2),
               "mean_root_to_leaf_paths": round(float(st[:, 2].mean()), 2),
               "max_rel_diff_between_routes": worst}
        log("tree shape k=%d depth=%d n=%d: R2L %.1f us, serial %.2fx, parallel %.2fx, hybrid %.2fx "
            "(routes agree to %.1e)" % (k, depth, n, mean["r2l"], row["serial_x"], row["parallel_x"],
                                        row["hybrid_x"], worst))
        rows.append(row)
    print(json.dumps({"study": "tree-shapes", "shape": {"batch": 1, "heads": H, "d_k": dk, "d_v": dv,
                                                        "qkv_dtype": "bf16", "state_dtype": "f32"},
                      "trees": "top-k rollouts of the configured depth pruned to the node budget",
                      "r2l": "one serial chain verification per root-to-leaf path",
                      "trees_per_shape": trees_per_shape, "rows": rows}), flush=True)


def study_fused_commit(args, torch, B, inputs, dev, reps=10, rounds=20):
    """Delayed state update at the paper's target shape (batch 1, 8 heads,
    d_k = d_v = 256, fp32 state, bf16 activations): per accepted length A in
    1..8, the time of one round that commits the previous round's A accepted
    nodes and verifies a 4-node chain, either fused (one sla_verify with the
    path pending: one state read and write) or separate (sla_commit, then
    sla_verify from the committed state).  Each route is a HIP graph of
    `rounds` consecutive rounds, replayed `reps` times (per-round time =
    total / (rounds x reps), the gaps between the kernels of a graph
    included); the state keeps advancing."""
    H, dk, dv, n_prev, n = 8, 256, 256, 8, 4
    rng = np.random.default_rng(4343)

    def bf(x):
        return torch.from_numpy(np.ascontiguousarray(inputs.bf16_bits(x)).view(np.int16)).view(torch.bfloat16).to(dev)

    def unit(shape):
        x = rng.standard_normal(shape)
        return x / np.linalg.norm(x, axis=-1, keepdims=True)

    def draft(m):
        return dict(q=bf(unit((1, m, H, dk))), k=bf(unit((1, m, H, dk))), v=bf(rng.standard_normal((1, m, H, dv))),
                    a=torch.from_numpy((1 / (1 + np.exp(-rng.uniform(2, 5, (1, m, H))))).astype(np.float32)).to(dev),
                    b=torch.from_numpy((1 / (1 + np.exp(-rng.standard_normal((1, m, H))))).astype(np.float32)).to(dev),
                    p=torch.arange(-1, m - 1, dtype=torch.int32, device=dev)[None])

    prev, cur = draft(n_prev), draft(n)
    S = torch.from_numpy((rng.standard_normal((1, H, dk, dv)) * 0.02).astype(np.float32)).to(dev)
    fprev = B.Factors.empty(1, n_prev, H, dk, dv, torch.bfloat16, dev)
    B.sla_verify(S, prev["q"], prev["k"], prev["v"], prev["a"], prev["b"], prev["p"],
                 torch.empty(1, n_prev, H, dv, device=dev), fprev, topology="chain")
    fcur = B.Factors.empty(1, n, H, dk, dv, torch.bfloat16, dev)
    out = torch.empty(1, n, H, dv, device=dev)
    # warm-up: clocks and caches settle before the first timed route
    wpath = torch.arange(n_prev, dtype=torch.int32, device=dev)[None]
    wlen = torch.tensor([4], dtype=torch.int32, device=dev)
    for _ in range(200):
        B.sla_verify(S, cur["q"], cur["k"], cur["v"], cur["a"], cur["b"], cur["p"], out, fcur,
                     pending=(fprev, wpath, wlen), topology="chain")
    torch.cuda.synchronize()
    S.copy_(S / (1.0 + float(S.abs().max())))
    rows = []
    for A in range(1, 9):
        path = torch.full((1, n_prev), -1, dtype=torch.int32, device=dev)
        path[0, :A] = torch.arange(A, dtype=torch.int32, device=dev)
        ln = torch.tensor([A], dtype=torch.int32, device=dev)
        t = {}
        for route in ["fused", "separate"]:
            def launch():
                if route == "fused":
                    B.sla_verify(S, cur["q"], cur["k"], cur["v"], cur["a"], cur["b"], cur["p"], out, fcur,
                                 pending=(fprev, path, ln), topology="chain")
                else:
                    B.sla_commit(S, fprev, path, ln)
                    B.sla_verify(S, cur["q"], cur["k"], cur["v"], cur["a"], cur["b"], cur["p"], out, fcur,
                                 topology="chain")
            launch()
            torch.cuda.synchronize()
            g = torch.cuda.CUDAGraph()
            sc = torch.cuda.Stream(dev)
            sc.wait_stream(torch.cuda.current_stream(dev))
            with torch.cuda.stream(sc):
                with torch.cuda.graph(g, stream=sc):
                    for _ in range(rounds):
                        launch()
            torch.cuda.synchronize()
            g.replay()
            torch.cuda.synchronize()
            cs = torch.cuda.current_stream(dev)
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(cs)
            for _ in range(reps):
                g.replay()
            e1.record(cs)
            torch.cuda.synchronize()
            t[route] = e0.elapsed_time(e1) * 1e3 / (reps * rounds)
            # keep the state in range: S drifts under repeated commits of the same records
            S.copy_(S / (1.0 + float(S.abs().max())))
        rows.append({"accepted": A, "fused_us": round(t["fused"], 2), "separate_us": round(t["separate"], 2),
                     "separate_over_fused": round(t["separate"] / t["fused"], 2)})
        log("accepted %d: fused %.2f us, separate %.2f us (%.2fx)" % (A, t["fused"], t["separate"],
                                                                      t["separate"] / t["fused"]))
    print(json.dumps({"study": "fused-commit", "shape": {"batch": 1, "heads": H, "d_k": dk, "d_v": dv,
                                                         "verify_len": n, "qkv_dtype": "bf16", "state_dtype": "f32"},
                      "rounds_per_graph": rounds, "reps": reps, "rows": rows}), flush=True)


if __name__ == "__main__":
    main()
