#!/usr/bin/env python
"""Throughput of the tree-replay round on one MI355X.

A step is one full round (plan -> replay -> verify, every kernel of the
path) over one batch of R requests, through tsb_step. Default workload: the
batched serving shape, R=16 requests, V=151936, draft block D=16, budget
B=128 (non-root nodes), K=10 planning candidates, bf16 logits, T=1. Inputs
are synthetic (workloads package), resident in HBM before timing starts; a
pool of P distinct input sets is rotated so that no step reuses cached rows.

Prints one JSON line: steps/s as `value`, verified tree nodes/s, the
roofline of the replay scan (the largest throughput-bound kernel: VALU-bound
when the walk reads the target rows of the nodes it enters, as above 128 MiB
of target; HBM-bound when its grid also streams every target row) measured
live with HIP events on the launch stream, the target stream alone, a
per-kernel breakdown with the walk's per-node latency, and the CPU oracle
timed on a bounded sample of the same workload on the host cores.
"""
import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

import workloads as W  # noqa: E402

HBM_PEAK_GBS = 8000.0
# kernels launched by one replay + RRS round (the replay scan's grid also
# streams the target when the rows are streamed), and by one round over
# sparse pools
STEP_KERNELS = ("draft_partials", "plan_tree", "scan_target", "replay_merge", "verify_walk")
POOL_KERNELS = ("pool_partials", "pool_lists", "pool_plan", "pool_replay", "target_partials", "pool_walk")

# Counter passes per launch at the batched workload, valid for the kernel
# source they were taken on: HBM traffic from FETCH_SIZE / WRITE_SIZE (KiB,
# scaled by a plain copy of known size: FETCH x2.0, WRITE x1.0) and VALU
# wave-instructions from SQ_INSTS_VALU.
COUNTERS = {
    # the round's launch at the batched workload, where the walk reads the
    # target rows of the nodes it enters (the grid scans and clears only)
    "scan_target": {"config": 4, "source_sha256_16": "18036137b51afcf4", "fetch_kib": 42238.8, "write_kib": 893.2,
                    "insts_valu": 30225698.1},
    "target_partials": {"config": 4, "source_sha256_16": "fcb4baee469cbe10", "fetch_kib": 311708.5,
                        "write_kib": 520.0, "insts_valu": 35377376.0},
}
FETCH_SCALE, WRITE_SCALE = 2.0, 1.0
# peak VALU issue: 256 CUs x 4 SIMDs x 16 lanes x 2.4 GHz = 39.3e12 lane
# operations/s, i.e. 614.4e9 wave64 instructions/s
VALU_PEAK_WAVE_INSTS = 256 * 2.4e9


def _read(path):
    return open(os.path.join(ROOT, "paper_2609_33652_amd", "csrc", path)).read()


def _section(path, start, end):
    src = _read(path)
    a, b = src.find(start), src.find(end)
    return None if a < 0 or b < 0 else src[a:b]


def source_hash(kernel):
    """Hash of the source a kernel is built from (its device code), to tie counter figures to it."""
    import hashlib
    if kernel == "scan_target":
        parts = [_section("k_replay.hip", "struct ScanArgs {", "__global__ __launch_bounds__(kWave) void replay_merge("),
                 _read("tsb_target.hpp")]
    elif kernel == "target_partials":
        parts = [_section("k_verify.hip", "// ------------------------------------------------------------------ K4",
                          "// ------------------------------------------------------------------ K5"),
                 _read("tsb_target.hpp")]
    else:
        return None
    if any(p is None for p in parts):
        return None
    return hashlib.sha256("".join(parts).encode()).hexdigest()[:16]


def counted(kernel, cfg_id):
    """Counter figures of a kernel at this workload: (traffic bytes or None, VALU wave-instructions or None)."""
    t = COUNTERS.get(kernel)
    if t is None or cfg_id != t["config"] or t["source_sha256_16"] is None or source_hash(kernel) != t["source_sha256_16"]:
        return None, None
    traffic = None
    if t["fetch_kib"] is not None and t["write_kib"] is not None:
        traffic = int(round((t["fetch_kib"] * FETCH_SCALE + t["write_kib"] * WRITE_SCALE) * 1024))
    return traffic, t["insts_valu"]


def parent_rows(h, B):
    """Distinct (request, depth) draft rows that hold at least one parent of a round's tree."""
    import torch
    n = h["n_nodes"].long()
    idx = torch.arange(B + 1).unsqueeze(0)
    par = (idx < n.unsqueeze(1)) & (h["n_children"].long() > 0)
    dep = h["depth"].long().clamp(min=0)
    rows = set()
    for r, u in par.nonzero().tolist():
        rows.add((r, int(dep[r, u])))
    return len(rows)


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def events(n):
    """n pairs of timing events, created up front (torch creates them lazily on first record)."""
    import torch
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(n)]
    for a, b in ev:
        a.record()
        b.record()
    torch.cuda.synchronize()
    return ev


# ---------------------------------------------------------------- CPU oracle
_CPU = {}


def _cpu_task(args):
    r, step = args
    c = _CPU["cfg"]
    if _CPU["path"] == "first_naive":
        from oracle import naive as onaive
        out = onaive.first_naive_request(_CPU["draft"][r], _CPU["target"][r], c["T"], c["K"], c["B"], _CPU["seed"],
                                         step, r)
    elif _CPU["path"] == "traversal":
        from oracle import step as ostep
        out = ostep.step_request(_CPU["draft"][r], _CPU["target"][r], c["T"], c["K"], c["B"], _CPU["seed"], step, r,
                                 verifier="traversal")
    elif _CPU["path"] == "pool":
        from oracle import pool as opool
        out = opool.step_pool_request(_CPU["draft"][r], _CPU["target"][r], _CPU["trans"][r], c["T"], c["K"],
                                      _CPU["P"], c["B"], _CPU["seed"], step, r)
    else:
        from oracle import step as ostep
        out = ostep.step_request(_CPU["draft"][r], _CPU["target"][r], c["T"], c["K"], c["B"], _CPU["seed"], step, r)
    return out["n_acc"]


def host_cores():
    """Worker processes of the CPU baseline: the host's CPUs, at most the 16 a one-GPU share has."""
    return min(16, len(os.sched_getaffinity(0)))


def cpu_baseline(cfg, seed, requests, path="replay_rrs", P=None):
    """Time the oracle over `requests` request-steps of one input set (runs before any GPU use)."""
    import multiprocessing as mp

    import torch
    from oracle import step as ostep
    base, sigma = W.base_rows(cfg, 0, device="cpu")
    draft = W.draft_from_base(cfg, base)
    trans = W.transitions(cfg, P, set_idx=0) if path == "pool" else None
    dep = torch.zeros(cfg["R"], cfg["B"] + 1, dtype=torch.int64)
    for r in range(min(requests, cfg["R"])):
        if path == "pool":
            from oracle import pool as opool
            tree = pool_plan_cpu(opool, draft[r].float().numpy(), trans[r].numpy(), cfg, P)
        else:
            tree = ostep.plan_request(draft[r].float().numpy(), cfg["T"], cfg["K"], cfg["B"])["tree"]
        dep[r, :tree["n_nodes"]] = torch.from_numpy(tree["depth"])
    target = W.target_from_base(cfg, base, sigma, dep)
    del base
    # plain numpy in the workers: no torch (OpenMP) use after fork
    nr = min(requests, cfg["R"])
    _CPU.update(cfg=cfg, draft=draft[:nr].float().numpy(), target=target[:nr].float().numpy(), seed=seed, path=path,
                trans=None if trans is None else trans[:nr].numpy(), P=P)
    del draft, target
    log("cpu baseline: inputs ready")
    tasks = [(r % nr, r // nr) for r in range(requests)]
    cores = min(host_cores(), len(tasks))
    ctx = mp.get_context("fork")
    t0 = time.perf_counter()
    with ctx.Pool(cores) as pool:
        pool.map(_cpu_task, tasks, chunksize=1)
    dt = time.perf_counter() - t0
    _CPU.clear()
    what = "pools of %d tokens" % P if path == "pool" else path.replace("_", " + ")
    return dict(value=(len(tasks) / cfg["R"]) / dt, unit="steps/s", cores=cores, host_cpus=len(os.sched_getaffinity(0)),
                kind="oracle",
                sample="%d request-steps (%g steps) of the %s workload, CPU-generated set 0, %s round; wall %.2f s"
                       % (len(tasks), len(tasks) / cfg["R"], cfg["name"], what, dt))


def pool_plan_cpu(opool, draft, trans, cfg, P):
    """The pool oracle's first pass for one request (only its depths key the target rows)."""
    from oracle.rowstats import inv_temperature
    invT = inv_temperature(cfg["T"])
    pl = opool.pools(draft, P)
    return opool.plan_ctx(opool.pool_logits(draft, invT, pl), opool.scaled_corrections(trans, invT), cfg["K"],
                          cfg["B"])


# ---------------------------------------------------------------- GPU
def first_naive(tsb, c, dev, drafts, targets, args, cfg):
    """The First + Naive baseline on the same inputs: timed rounds, acceptance, and the walk's roofline."""
    import torch
    R, V = cfg["R"], cfg["V"]
    P = len(drafts)
    rnd = tsb.Round(c, dev)
    for s in range(args.warmup):
        rnd.step_first(drafts[s % P], targets[s % P], s)
    torch.cuda.synchronize()
    start = torch.cuda.Event(enable_timing=True)
    stop = torch.cuda.Event(enable_timing=True)
    start.record()
    for i in range(args.first_steps):
        s = args.warmup + i
        rnd.step_first(drafts[s % P], targets[s % P], s)
    stop.record()
    torch.cuda.synchronize()
    ms = start.elapsed_time(stop) / args.first_steps
    # the walk kernel alone, with the rows it visited (one read of each)
    kern_us = {}
    visited = 0
    for name in ("draft_partials", "plan_tree", "verify_naive"):
        kid = tsb.KERNELS.index(name)
        evs = events(args.breakdown_steps)
        for i in range(args.breakdown_steps):
            tsb.profile_kernel(kid, evs[i][0], evs[i][1])
            rnd.step_first(drafts[i % P], targets[i % P], i)
            tsb.profile_kernel(kid, None)
            if name == "verify_naive":
                n_acc = rnd.n_acc.clamp(min=-1)
                visited += int((n_acc + 1).sum())
        torch.cuda.synchronize()
        kern_us[name] = round(1000.0 * sum(a.elapsed_time(b) for a, b in evs) / args.breakdown_steps, 2)
    acc = 0
    for i in range(P):
        rnd.step_first(drafts[i], targets[i], i)
        h = rnd.host()
        acc += int(h["n_acc"].clamp(min=0).sum()) + int((h["n_acc"] >= 0).sum())
    tau = acc / (P * R)
    b = 2 if cfg["dtype"] == "bf16" else 4
    walk_bytes = visited / args.breakdown_steps * V * b
    achieved = walk_bytes / (kern_us["verify_naive"] * 1e-6) / 1e9
    return {
        "steps_per_s": round(1000.0 / ms, 2), "ms_per_step": round(ms, 4), "steps": args.first_steps,
        "tau": round(tau, 4), "accepted_tokens_per_s": round(tau * R * 1000.0 / ms, 1),
        "kernels_us": kern_us,
        "roofline": {"kernel": "verify_naive", "bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS,
                     "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": None,
                     "bytes_per_launch": int(walk_bytes), "avg_launch_us": kern_us["verify_naive"],
                     "rows_per_launch": round(visited / args.breakdown_steps, 2),
                     "note": "one cross-workgroup exchange per visited row; latency, not bandwidth, sets its time"},
    }


def traversal_block(tsb, c, dev, drafts, targets, args, cfg):
    """Replay + traversal verification on the same inputs: timed rounds, the walk's time and acceptance."""
    import torch
    R = cfg["R"]
    P = len(drafts)
    rnd = tsb.Round(c, dev)
    for s in range(args.warmup):
        rnd.step_traversal(drafts[s % P], targets[s % P], s)
    torch.cuda.synchronize()
    start = torch.cuda.Event(enable_timing=True)
    stop = torch.cuda.Event(enable_timing=True)
    start.record()
    for i in range(args.first_steps):
        s = args.warmup + i
        rnd.step_traversal(drafts[s % P], targets[s % P], s)
    stop.record()
    torch.cuda.synchronize()
    ms = start.elapsed_time(stop) / args.first_steps
    kid = tsb.KERNELS.index("traversal_walk")
    evs = events(args.breakdown_steps)
    for i in range(args.breakdown_steps):
        tsb.profile_kernel(kid, evs[i][0], evs[i][1])
        rnd.step_traversal(drafts[i % P], targets[i % P], i)
        tsb.profile_kernel(kid, None)
    torch.cuda.synchronize()
    walk_us = 1000.0 * sum(a.elapsed_time(b) for a, b in evs) / args.breakdown_steps
    acc, tests = 0, 0
    trnd = tsb.Round(c, dev, trace=True)
    for i in range(P):
        trnd.step_traversal(drafts[i], targets[i], i)
        h = trnd.host()
        acc += int(h["n_acc"].clamp(min=0).sum()) + int((h["n_acc"] >= 0).sum())
        tests += int((h["trace"][:, :, 0] >= 0).sum())
    tau = acc / (P * R)
    return {"steps_per_s": round(1000.0 / ms, 2), "ms_per_step": round(ms, 4), "steps": args.first_steps,
            "tau": round(tau, 4), "accepted_tokens_per_s": round(tau * R * 1000.0 / ms, 1),
            "walk_kernel": "traversal_walk", "walk_avg_launch_us": round(walk_us, 2),
            "tests_per_request": round(tests / (P * R), 2),
            "note": "one vocabulary-wide pass and one cross-workgroup exchange per rejected node and per internal "
                    "node entered; latency, not bandwidth, sets the walk's time"}


def planner_ep(tsb, c, dev, drafts, targets, args, cfg, frontier=10):
    """The expand-then-prune first pass (frontier 10) on the same inputs: planner latency and acceptance."""
    import torch
    R = cfg["R"]
    P = len(drafts)
    rnd = tsb.Round(c, dev)
    kid = tsb.KERNELS.index("plan_tree")
    for s in range(3):
        rnd.plan_ep(drafts[s % P], frontier)
    evs = events(args.breakdown_steps)
    for i in range(args.breakdown_steps):
        tsb.profile_kernel(kid, evs[i][0], evs[i][1])
        rnd.plan_ep(drafts[i % P], frontier)
        tsb.profile_kernel(kid, None)
    torch.cuda.synchronize()
    us = 1000.0 * sum(a.elapsed_time(b) for a, b in evs) / args.breakdown_steps
    acc = 0
    for i in range(P):
        rnd.plan_ep(drafts[i], frontier)
        rnd.replay(drafts[i], i)
        rnd.verify(drafts[i], targets[i], i)
        h = rnd.host()
        acc += int(h["n_acc"].clamp(min=0).sum()) + int((h["n_acc"] >= 0).sum())
    return {"frontier": frontier, "kernel": "plan_ep", "avg_launch_us": round(us, 2),
            "tau_replay_rrs": round(acc / (P * R), 4)}


def pool_block(tsb, c, dev, drafts, args, cfg, P):
    """The round over sparse pools of P tokens with transition-score corrections: its own targets (keyed by
    the pool plan's depths), timed rounds, per-kernel times, acceptance."""
    import torch
    R = cfg["R"]
    NS = len(drafts)
    rnd = tsb.Round(c, dev, pool=P)
    trans, targets = [], []
    for p in range(NS):
        base, sigma = W.base_rows(cfg, p, device=dev)
        tr = W.transitions(cfg, P, set_idx=p, device=dev)
        rnd.pool_plan(drafts[p], tr)
        dep = rnd.tree["depth"].long().clamp(min=0)
        targets.append(W.target_from_base(cfg, base, sigma, dep, set_idx=p))
        trans.append(tr)
        del base
    torch.cuda.synchronize()
    for s in range(args.warmup):
        rnd.pool_step(drafts[s % NS], trans[s % NS], targets[s % NS], s)
    torch.cuda.synchronize()
    start = torch.cuda.Event(enable_timing=True)
    stop = torch.cuda.Event(enable_timing=True)
    start.record()
    for i in range(args.first_steps):
        s = args.warmup + i
        rnd.pool_step(drafts[s % NS], trans[s % NS], targets[s % NS], s)
    stop.record()
    torch.cuda.synchronize()
    ms = start.elapsed_time(stop) / args.first_steps
    kern_us = {}
    for name in POOL_KERNELS:
        kid = tsb.KERNELS.index(name)
        evs = events(args.breakdown_steps)
        for i in range(args.breakdown_steps):
            tsb.profile_kernel(kid, evs[i][0], evs[i][1])
            rnd.pool_step(drafts[i % NS], trans[i % NS], targets[i % NS], i)
            tsb.profile_kernel(kid, None)
        torch.cuda.synchronize()
        kern_us[name] = round(1000.0 * sum(a.elapsed_time(b) for a, b in evs) / args.breakdown_steps, 2)
    acc, flagged = 0, 0
    for i in range(NS):
        rnd.pool_step(drafts[i], trans[i], targets[i], i)
        h = rnd.host()
        acc += int(h["n_acc"].clamp(min=0).sum()) + int((h["n_acc"] >= 0).sum())
        flagged += int(h["req_status"].ne(0).logical_and(h["n_acc"] < 0).sum())
    tau = acc / (NS * R)
    del targets, trans
    torch.cuda.empty_cache()
    return {"pool_size": P, "steps_per_s": round(1000.0 / ms, 2), "ms_per_step": round(ms, 4),
            "steps": args.first_steps, "tau": round(tau, 4), "accepted_tokens_per_s": round(tau * R * 1000.0 / ms, 1),
            "kernels_us": kern_us, "flagged_requests": flagged,
            "transitions": "i.i.d. 1.5 * N(0, 1) binary32 scores [R, D-1, P, P]"}


def latency_block(tsb, cfg_id, args, n=200):
    """Latency of one replay + RRS round of a small workload (one request): back-to-back rounds launched
    eagerly, the same round captured once as a graph and replayed, and eager rounds each followed by a
    synchronisation (what a caller waiting on every round sees)."""
    import torch
    cfg = W.config(cfg_id)
    c = tsb.make_config(cfg["R"], cfg["D"], cfg["V"], cfg["B"], cfg["K"], cfg["T"], cfg["dtype"],
                        W.replay_seed(cfg_id))
    dev = torch.device("cuda:0")
    rnd = tsb.Round(c, dev)
    base, sigma = W.base_rows(cfg, 0, device=dev)
    draft = W.draft_from_base(cfg, base)
    rnd.plan(draft)
    dep = rnd.tree["depth"].long().clamp(min=0)
    target = W.target_from_base(cfg, base, sigma, dep)
    del base
    for s in range(20):
        rnd.step(draft, target, s)
    torch.cuda.synchronize()
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record()
    for s in range(n):
        rnd.step(draft, target, s)
    b.record()
    torch.cuda.synchronize()
    eager_us = 1000.0 * a.elapsed_time(b) / n
    t0 = time.perf_counter()
    for s in range(n):
        rnd.step(draft, target, s)
        torch.cuda.synchronize()
    sync_us = 1e6 * (time.perf_counter() - t0) / n
    # one round captured as a graph (the step index is fixed in it); its outputs must equal the eager round's
    rnd.step(draft, target, 7)
    ref = {k: rnd.host()[k].clone() for k in ("node_tok", "n_acc", "bonus", "acc_tok")}
    g = torch.cuda.CUDAGraph()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        rnd.step(draft, target, 7)  # warm-up on the capture stream
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    with torch.cuda.graph(g):
        rnd.step(draft, target, 7)
    g.replay()
    torch.cuda.synchronize()
    h = rnd.host()
    same = all(torch.equal(h[k], ref[k]) for k in ref)
    a.record()
    for s in range(n):
        g.replay()
    b.record()
    torch.cuda.synchronize()
    graph_us = 1000.0 * a.elapsed_time(b) / n
    t0 = time.perf_counter()
    for s in range(n):
        g.replay()
        torch.cuda.synchronize()
    gsync_us = 1e6 * (time.perf_counter() - t0) / n
    del g
    return {"workload": W.describe(cfg), "eager_us_per_round": round(eager_us, 2),
            "graph_us_per_round": round(graph_us, 2), "eager_synced_us": round(sync_us, 2),
            "graph_synced_us": round(gsync_us, 2), "graph_matches_eager": bool(same), "rounds": n}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--config", type=int, default=4)
    ap.add_argument("--pool", type=int, default=4)
    ap.add_argument("--cpu-requests", type=int, default=None, help="oracle request-steps in the CPU baseline")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--breakdown-steps", type=int, default=20)
    ap.add_argument("--sample", type=int, default=8, help="time the target kernel on every n-th timed step")
    ap.add_argument("--first-steps", type=int, default=100, help="timed steps of the First + Naive baseline")
    ap.add_argument("--pool-size", type=int, default=64, help="tokens per pool in the sparse-pool round (0: skip)")
    ap.add_argument("--latency", type=int, default=1, help="per-round latency of the small workloads, eager and "
                                                               "as a captured graph (0: skip)")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py measures one GPU only: this build has no multi-GPU path (requests shard with no "
              "exchange; see the design notes). Run with --gpus 1.", file=sys.stderr)
        sys.exit(2)

    cfg = W.config(args.config)
    seed = W.replay_seed(args.config)
    R, D, V, B, K = cfg["R"], cfg["D"], cfg["V"], cfg["B"], cfg["K"]

    cpu = None
    if not args.no_cpu_baseline:
        nreq = args.cpu_requests if args.cpu_requests is not None else max(R, host_cores())
        log("cpu baseline: %d oracle request-steps" % nreq)
        cpu = cpu_baseline(cfg, seed, nreq)
        log("cpu baseline:", cpu)
        cpu_first = cpu_baseline(cfg, seed, nreq, path="first_naive")
        log("cpu baseline (first + naive):", cpu_first)
        cpu_trav = cpu_baseline(cfg, seed, nreq, path="traversal")
        log("cpu baseline (traversal):", cpu_trav)
        cpu_pool = cpu_baseline(cfg, seed, nreq, path="pool", P=args.pool_size) if args.pool_size else None
        log("cpu baseline (pools):", cpu_pool)
    else:
        cpu_first = cpu_pool = cpu_trav = None

    import torch
    import paper_2609_33652_amd as tsb
    tsb.load()
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    c = tsb.make_config(R, D, V, B, K, cfg["T"], cfg["dtype"], seed)
    rnd = tsb.Round(c, dev)

    # input pool, resident in HBM
    drafts, targets = [], []
    for p in range(args.pool):
        base, sigma = W.base_rows(cfg, p, device=dev)
        draft = W.draft_from_base(cfg, base)
        rnd.plan(draft)
        dep = rnd.tree["depth"].long().clamp(min=0)
        targets.append(W.target_from_base(cfg, base, sigma, dep, set_idx=p))
        drafts.append(draft)
        del base
    torch.cuda.synchronize()
    log("pool ready: %d sets, %.1f GB" % (args.pool, sum(d.numel() * d.element_size() + t.numel() *
                                                           t.element_size() for d, t in zip(drafts, targets)) / 1e9))

    P = args.pool
    for s in range(args.warmup):
        rnd.step(drafts[s % P], targets[s % P], s)
    torch.cuda.synchronize()

    # above 128 MiB of target the walk reads the rows of the nodes it enters
    # and the scan's grid streams no target row
    streams = not tsb.walk_reads_rows(c)
    K4 = tsb.KERNELS.index("scan_target")
    # the replay scan (with the target stream in its grid when the rows are
    # streamed) is bracketed by events
    # on every `sample`-th timed step (each event pair costs a few
    # microseconds of idle GPU)
    sampled = list(range(0, args.steps, args.sample))
    ev = events(len(sampled))
    start = torch.cuda.Event(enable_timing=True)
    stop = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t_host0 = time.perf_counter()
    start.record()
    for i in range(args.steps):
        s = args.warmup + i
        if i % args.sample == 0:
            a, b = ev[i // args.sample]
            tsb.profile_kernel(K4, a, b)
        rnd.step(drafts[s % P], targets[s % P], s)
        if i % args.sample == 0:
            tsb.profile_kernel(K4, None)
    stop.record()
    torch.cuda.synchronize()
    t_host1 = time.perf_counter()
    ms = start.elapsed_time(stop) / args.steps
    k4_ms = sum(a.elapsed_time(b) for a, b in ev) / len(ev)

    # untimed passes: per-kernel breakdown and acceptance statistics
    kern_us = {}
    for name in STEP_KERNELS:
        kid = tsb.KERNELS.index(name)
        evs = events(args.breakdown_steps)
        for i in range(args.breakdown_steps):
            tsb.profile_kernel(kid, evs[i][0], evs[i][1])
            rnd.step(drafts[i % P], targets[i % P], i)
        torch.cuda.synchronize()
        tsb.profile_kernel(kid, None)
        kern_us[name] = round(1000.0 * sum(a.elapsed_time(b) for a, b in evs) / args.breakdown_steps, 2)
    # untimed pass with the work counters on: replay pruning, walk and planner
    tsb.stats_read(reset=True)
    tsb.stats_enable(True)
    for i in range(args.breakdown_steps):
        rnd.step(drafts[i % P], targets[i % P], i)
    work = tsb.stats_read(reset=True)
    tsb.stats_enable(False)
    acc, nodes, flagged, trows, drows = 0, 0, 0, 0, 0
    for i in range(P):
        rnd.step(drafts[i], targets[i], i)
        h = rnd.host()
        acc += int(h["n_acc"].clamp(min=0).sum()) + int((h["n_acc"] >= 0).sum())
        nodes += int((h["n_nodes"] - 1).sum())
        flagged += int((h["req_status"] & (tsb.REQ_NONFINITE | tsb.REQ_WALK_TIMEOUT)).ne(0).sum())
        trows += int(h["n_nodes"].sum())
        drows += parent_rows(h, B)
    tau = acc / (P * R)
    nodes_per_step = nodes / P
    # the target stream alone (the verification entry point launches it on
    # its own grid when the normaliser output is asked for), for its own
    # roofline
    KT = tsb.KERNELS.index("target_partials")
    trnd = tsb.Round(c, dev, target_lse=True)
    evt = events(args.breakdown_steps)
    for i in range(args.breakdown_steps):
        trnd.step(drafts[i % P], targets[i % P], i)
        tsb.profile_kernel(KT, evt[i][0], evt[i][1])
        trnd.verify(drafts[i % P], targets[i % P], i)
        tsb.profile_kernel(KT, None)
    torch.cuda.synchronize()
    del trnd
    kt_us = 1000.0 * sum(a.elapsed_time(b) for a, b in evt) / args.breakdown_steps

    first = first_naive(tsb, c, dev, drafts, targets, args, cfg)
    first["cpu_baseline"] = cpu_first
    trav = traversal_block(tsb, c, dev, drafts, targets, args, cfg)
    trav["cpu_baseline"] = cpu_trav
    ep = planner_ep(tsb, c, dev, drafts, targets, args, cfg)
    del targets
    torch.cuda.empty_cache()
    pool = None
    if args.pool_size:
        pool = pool_block(tsb, c, dev, drafts, args, cfg, args.pool_size)
        pool["cpu_baseline"] = cpu_pool

    latency = None
    if args.latency:
        del drafts
        torch.cuda.empty_cache()
        latency = {W.config(i)["name"]: latency_block(tsb, i, args) for i in (1, 2, 3)}

    b = 2 if cfg["dtype"] == "bf16" else 4
    # algorithmic bytes of one scan_target launch: every draft row that holds
    # parents and, when the rows are streamed, every target row of the tree,
    # each read once
    t_bytes = trows * V * b // P
    d_bytes = drows * V * b // P
    k4_bytes = (t_bytes if streams else 0) + d_bytes
    nst = max(1, args.breakdown_steps)
    traffic, insts = counted("scan_target", args.config)
    replay = {
        "kernel": "scan_target", "bound": "alu", "avg_launch_us": kern_us["scan_target"],
        "items_per_launch": round(work["replay_items"] / nst, 1),
        "tokens_per_launch": round(work["replay_tokens"] / nst, 1),
        "live_fraction": round(4 * work["replay_groups_live"] / max(1, work["replay_tokens"]), 5),
        "keyed_fraction": round(4 * work["replay_groups_keyed"] / max(1, work["replay_tokens"]), 5),
        "valu_insts_per_launch": insts,
        "achieved": None if insts is None else round(insts / (kern_us["scan_target"] * 1e-6) / 1e9, 1),
        "peak": VALU_PEAK_WAVE_INSTS / 1e9, "unit": "G wave64 VALU instructions/s",
        "frac": None if insts is None else round(insts / (kern_us["scan_target"] * 1e-6) / VALU_PEAK_WAVE_INSTS, 4),
        "note": "VALU issue of the whole launch (the scan, and the target stream when the rows are streamed); "
                "fractions are of the scanned tiles' tokens, in groups of four: live = the group's largest key "
                "bound reaches the parent's threshold (its Philox words are drawn), keyed = a word passes the "
                "floor (its Gumbel keys are evaluated)"}
    t_traffic, t_insts = counted("target_partials", args.config)
    target_stream = {"kernel": "target_partials", "bound": "hbm",
                     "achieved": round(t_bytes / (kt_us * 1e-6) / 1e9, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(t_bytes / (kt_us * 1e-6) / 1e9 / HBM_PEAK_GBS, 4), "traffic": t_traffic,
                     "bytes_per_launch": t_bytes, "avg_launch_us": round(kt_us, 2),
                     "source": "tsb_verify after each round, untimed pass"}
    wr = max(1, work["walk_requests"])
    walk = {"kernel": "verify_walk", "avg_launch_us": kern_us["verify_walk"],
            "nodes_per_request": round(work["walk_nodes"] / wr, 3),
            "tests_per_request": round(work["walk_tests"] / wr, 3),
            "exchanges_per_request": round(work["walk_exchanges"] / wr, 3),
            "us_per_node": round(kern_us["verify_walk"] / max(1e-9, work["walk_nodes"] / wr), 2),
            "us_per_exchange": round(kern_us["verify_walk"] / max(1e-9, work["walk_exchanges"] / wr), 2),
            "target_rows_read": "entered nodes only" if not streams else "none (streamed before the walk)",
            "note": "per-node and per-exchange times divide the launch time by the mean count of one request "
                    "(the requests run side by side); the walk is bound by the latency of its exchanges and "
                    "row reads, one node after another, not by bandwidth"}
    pr = max(1, work["plan_requests"])
    plan = {"kernel": "plan_tree", "avg_launch_us": kern_us["plan_tree"],
            "merge_us": round(work["plan_merge_ticks"] / pr * 0.01, 2),
            "search_us": round(work["plan_search_ticks"] / pr * 0.01, 2),
            "emit_us": round(work["plan_emit_ticks"] / pr * 0.01, 2),
            "rounds_per_request": round(work["plan_rounds"] / pr, 2),
            "note": "phase times of one request's workgroup from the 100 MHz real-time counter"}
    k1_bytes = R * D * V * b        # every draft row, read once
    achieved = k4_bytes / (k4_ms * 1e-3) / 1e9
    if streams:
        roofline = {"kernel": "scan_target", "bound": "hbm", "achieved": round(achieved, 1),
                    "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4),
                    "traffic": traffic, "bytes_per_launch": k4_bytes, "target_bytes": t_bytes,
                    "draft_bytes": d_bytes, "avg_launch_us": round(k4_ms * 1000, 2), "timed_launches": len(ev),
                    "note": "one grid streams every target row of the tree (row normalisers for the walk) and "
                            "scans the draft rows of the parents' depths (replay); bytes count each row once"}
    else:
        va = None if insts is None else insts / (k4_ms * 1e-3)
        roofline = {"kernel": "scan_target", "bound": "alu",
                    "achieved": None if va is None else round(va / 1e9, 1),
                    "peak": VALU_PEAK_WAVE_INSTS / 1e9, "unit": "G wave64 VALU instructions/s",
                    "frac": None if va is None else round(va / VALU_PEAK_WAVE_INSTS, 4),
                    "traffic": traffic, "valu_insts_per_launch": insts, "bytes_per_launch": k4_bytes,
                    "hbm_gbs": round(achieved, 1), "avg_launch_us": round(k4_ms * 1000, 2),
                    "timed_launches": len(ev),
                    "note": "the replay scan of the draft rows of the parents' depths (Gumbel-top-k over every "
                            "token, Philox words drawn where the key bound allows): VALU-bound; the target rows "
                            "are read by the walk as it enters their nodes. verify_walk takes longer per round but "
                            "is latency-bound (walk_breakdown)"}
    steps_per_s = 1000.0 / ms
    out = {
        "metric": "tree-replay steps/sec + verified nodes/sec at V=151936,B=128,bs=16; % HBM peak",
        "value": round(steps_per_s, 2),
        "unit": "steps/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": cfg["dtype"],
        "data": "synthetic",
        "config": {"workload": "%s: %s" % (cfg["name"], W.describe(cfg)), "requests": R, "vocab": V,
                   "draft_depth": D, "budget": B, "topk": K, "temperature": cfg["T"], "pool": P,
                   "seed": seed},
        "nodes_verified_per_s": round(nodes_per_step * steps_per_s, 1),
        "accepted_tokens_per_s": round(tau * R * steps_per_s, 1),
        "tau": round(tau, 4),
        "roofline": roofline,
        "kernels_us": kern_us,
        "roofline_target_stream": target_stream,
        # the other logit-streaming kernel, from the untimed per-kernel pass
        "roofline_draft": {"kernel": "draft_partials", "bound": "hbm (VALU-bound: a table lookup and a binary64 add per logit)",
                           "achieved": round(k1_bytes / (kern_us["draft_partials"] * 1e-6) / 1e9, 1),
                           "peak": HBM_PEAK_GBS, "unit": "GB/s",
                           "frac": round(k1_bytes / (kern_us["draft_partials"] * 1e-6) / 1e9 / HBM_PEAK_GBS, 4),
                           "bytes_per_launch": k1_bytes, "avg_launch_us": kern_us["draft_partials"],
                           "source": "per-kernel pass after the timed region"},
        "replay_roofline": replay,
        "walk_breakdown": walk,
        "plan_breakdown": plan,
        "latency": latency,
        "host_wall_s": round(t_host1 - t_host0, 3),
        "flagged_requests": flagged,
        "cpu_baseline": cpu,
        "first_naive": first,
        "traversal": trav,
        "planner_expand_prune": ep,
        "sparse_pools": pool,
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
