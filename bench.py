"""Decode-step throughput of segment-tree attention on one MI355X.

A step is one ``treepo_tree_decode`` call: every active leaf's query (all Hq
heads) attends over its root-to-leaf chain of segments, with inputs already
resident in HBM.  The default workload is the single 7B-style tree (1 prompt
of 512 tokens, segment length 512, binary forks at the first 4 boundaries, 16
leaves of 7680 tokens, Hq=28 Hkv=4 D=128, bf16 N(0,1) data).

Timing protocol: ``--replicas`` copies of the pools are built and the steps
rotate over them, so that no step finds its KV in the 256 MB Infinity Cache
(the whole working set of this tree is ~200 MB).  W untimed warm-up steps,
then exactly K timed steps between two device synchronisations (after half
a second of untimed steps in both modes, so that the GPU's clocks have
settled before the first timed mode).  A second pass of the K steps runs
with library profiling on: every launch records HIP events at its kernel's
own start and end, which gives the dominant kernel's average duration.  The
same protocol times the per-leaf paged-decode baseline, and a streaming-read
probe gives the attainable HBM read bandwidth.  The fp64 oracle is timed on
the host cores on the same workload.

Other modes: ``--config N`` (another workload), ``--segment-loop``
(segment-level decoding over several layers), ``--advantage`` (the TreePO
advantage) and ``--prefill`` (prompt prefill).  Prints one JSON line.
"""

from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

PEAK_HBM_GBPS = 8000.0
# HBM bytes per partial-kernel launch measured with rocprofv3 counters
# (FETCH_SIZE and WRITE_SIZE passes, calibrated on a plain copy kernel); the
# summary records the hash of the kernel source it was taken on.
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "partial_kernel_config2_traffic.txt")
KERNEL_SOURCE = os.path.join(ROOT, "paper_2508_17445_amd", "csrc", "kernels.hip")
METRIC = "tree-decode leaf-token-steps/sec + achieved HBM GB/s on unique KV (1 MI355X)"


def _parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--config", type=int, default=2)
    ap.add_argument("--replicas", type=int, default=0, help="pool copies rotated over (0: auto)")
    ap.add_argument("--no-naive", action="store_true")
    ap.add_argument("--no-cpu", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=10.0)
    ap.add_argument("--segment-loop", action="store_true",
                    help="instead of the default line: segment-level decoding after a fork, every step one "
                         "append per leaf then a decode, over --layers layers, steady state over the segment")
    ap.add_argument("--seg-len", type=int, default=512, help="segment capacity for --segment-loop")
    ap.add_argument("--layers", type=int, default=4, help="layers (each its own pools) for --segment-loop")
    ap.add_argument("--advantage", action="store_true",
                    help="TreePO advantage (Sec. 2.3, Eq. tree_ae) over the config's decoded leaves: one JSON line")
    ap.add_argument("--prefill", action="store_true",
                    help="prompt prefill (causal attention of every prompt of the config, written once into the "
                         "pools for all of its rollouts): one JSON line")
    ap.add_argument("--profile-pass", action="store_true",
                    help="short run for hardware counters: a few decode steps of the workload, then one "
                         "1 GiB device copy whose byte counters calibrate the kernels'")
    return ap.parse_args()


def _warm_gpu(reps, seconds=0.5):
    """Decode steps in both modes for about `seconds`, untimed, so that the
    first timed mode does not run while the GPU is still raising its clocks
    (without this the first mode measured its steps up to 10% slower)."""
    import torch
    bufs = {m: [(r.outputs(), r.workspace(m)) for r in reps] for m in (0, 1)}
    t0 = time.perf_counter()
    i = 0
    while time.perf_counter() - t0 < seconds:
        for m in (0, 1):
            j = i % len(reps)
            fn = reps[j].ctx.tree_decode if m == 0 else reps[j].ctx.paged_decode_naive
            (out, lse), ws = bufs[m][j]
            fn(reps[j].leaves, reps[j].q, reps[j].cfg.scale, out, lse, ws)
        i += 1
        if i % 64 == 0:
            torch.cuda.synchronize()
    torch.cuda.synchronize()


def _measured_traffic(config_id):
    """Counter-measured HBM bytes per partial-kernel launch, or None when no
    summary exists for this workload or the kernel source changed since."""
    import hashlib
    try:
        kv = dict(line.split(":", 1) for line in open(TRAFFIC_FILE).read().splitlines() if ":" in line)
        kv = {k.strip(): v.strip() for k, v in kv.items()}
        src = hashlib.sha256(open(KERNEL_SOURCE, "rb").read()).hexdigest()
        if kv.get("kernels.hip sha256") != src or int(kv.get("config", -1)) != config_id:
            return None
        return int(kv["traffic bytes per launch"])
    except (OSError, KeyError, ValueError):
        return None


def _ensure_built():
    from paper_2508_17445_amd.treepo import LIB_PATH
    if not os.path.exists(LIB_PATH):
        import __graft_entry__
        __graft_entry__.build()


def _unique_kv(dt):
    """Tokens per KV head over the nodes of the leaves' chains, each counted once."""
    model_len = {}
    nodes = dt.ctx.export_nodes()
    used = set()
    for x in dt.leaves:
        y = x
        while y != -1 and y not in used:
            used.add(y)
            y = int(nodes[y][0])
    tok = sum(int(nodes[n][3]) for n in used)
    logical = 0
    for x in dt.leaves:
        y = x
        while y != -1:
            logical += int(nodes[y][3])
            y = int(nodes[y][0])
    return tok, logical


def _time_mode(reps, mode, steps, warmup, kernel_kind):
    """Times `steps` decode steps rotating over the replicas.

    Two timed passes of the same length: the first without instrumentation
    gives the step time; the second brackets every kernel launch with HIP
    events on the launch stream (library profiling) and gives the average
    duration of each kernel.
    """
    import torch
    from paper_2508_17445_amd import KERNEL_COMBINE
    bufs = []
    for r in reps:
        out, lse = r.outputs()
        bufs.append((out, lse, r.workspace(mode)))
    fn = [(r.ctx.tree_decode if mode == 0 else r.ctx.paged_decode_naive) for r in reps]

    def run(n):
        for i in range(n):
            j = i % len(reps)
            fn[j](reps[j].leaves, reps[j].q, reps[j].cfg.scale, bufs[j][0], bufs[j][1], bufs[j][2])

    run(warmup)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    run(steps)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    for r in reps:
        r.ctx.set_profiling(True)
    torch.cuda.synchronize()
    t2 = time.perf_counter()
    run(steps)
    torch.cuda.synchronize()
    t3 = time.perf_counter()
    kms, kn, cms, cn = 0.0, 0, 0.0, 0
    for r in reps:
        a, b = r.ctx.profile_read(kernel_kind)
        c, d = r.ctx.profile_read(KERNEL_COMBINE)
        kms += a; kn += b; cms += c; cn += d
        r.ctx.set_profiling(False)
    return {"ms": (t1 - t0) * 1e3 / steps, "ms_instrumented": (t3 - t2) * 1e3 / steps,
            "kernel_ms": kms / max(kn, 1), "combine_ms": cms / max(cn, 1), "launches": kn // max(steps, 1)}


def _probe_read(nbytes=4 << 30, iters=10):
    import torch
    from paper_2508_17445_amd import bench_read
    src = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
    sink = torch.empty(4096, dtype=torch.float32, device="cuda")
    bench_read(src, nbytes, sink)
    torch.cuda.synchronize()
    st, en = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    st.record()
    for _ in range(iters):
        bench_read(src, nbytes, sink)
    en.record()
    torch.cuda.synchronize()
    ms = st.elapsed_time(en) / iters
    del src
    return nbytes / (ms * 1e-3) / 1e9


def _blas_threads():
    try:
        from threadpoolctl import threadpool_info
        return max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:
        return 1


def _cpu_baseline(cfg_id, seconds):
    import numpy as np
    from oracle import attention as A
    from oracle import metadata as M
    from workloads import CONFIGS, build_call_log, query_bits
    from workloads.device import NodeData
    try:
        from threadpoolctl import threadpool_info
        blas_threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:
        blas_threads = 1
    cfg, log = CONFIGS[cfg_id], build_call_log(cfg_id)
    model = M.replay(log, cfg.block_tokens, 1 << 30, 1 << 30)
    data = NodeData(cfg, log)
    data.prefetch(sorted({n for x in log.leaves for n in model.chain(x)}))
    q = query_bits(cfg.seed, 0, len(log.leaves), cfg.hq, cfg.d)
    reps, t0 = 0, time.perf_counter()
    while True:
        A.tree_decode(model, data, log.leaves, q, cfg.scale)
        reps += 1
        if time.perf_counter() - t0 >= seconds:
            break
    dt = time.perf_counter() - t0
    cores = min(len(os.sched_getaffinity(0)), blas_threads)
    return {"value": len(log.leaves) * reps / dt, "unit": "leaf-token-steps/s", "cores": cores,
            "kind": "oracle",
            "sample": f"{reps} full decode step(s) of the same workload ({len(log.leaves)} leaves, fp64 numpy, "
                      f"chains materialised per leaf) in {dt:.1f} s; host has "
                      f"{len(os.sched_getaffinity(0))} cores, BLAS threads {blas_threads}"}


def _profile_pass(dt, args):
    """A few decode steps (tree, then naive) and a 1 GiB copy, nothing else on the GPU."""
    import torch
    from paper_2508_17445_amd import bench_copy
    for mode in (0, 1):
        out, lse = dt.outputs()
        ws = dt.workspace(mode)
        fn = dt.ctx.tree_decode if mode == 0 else dt.ctx.paged_decode_naive
        for _ in range(args.steps):
            fn(dt.leaves, dt.q, dt.cfg.scale, out, lse, ws)
        torch.cuda.synchronize()
    nbytes = 1 << 30
    src = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
    dst = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
    bench_copy(dst, src, nbytes)
    torch.cuda.synchronize()
    print(json.dumps({"profile_pass": True, "steps_per_mode": args.steps, "copy_bytes": nbytes}), flush=True)


def _advantage(args):
    """TreePO advantage over the config's decoded leaves, 0/1 rewards: the
    kernel's duration (events attached to it), a whole call's time (host index
    arrays + upload + kernel, calls back to back), and the fp64 oracle on the
    host."""
    import numpy as np
    import torch
    from paper_2508_17445_amd import KERNEL_ADVANTAGE, Context
    from workloads import CONFIGS, build_call_log
    cfg, log = CONFIGS[args.config], build_call_log(args.config)
    dummy = torch.empty(256, dtype=torch.uint8, device="cuda")  # the advantage never reads the pools
    ctx = Context(cfg.hq, cfg.hkv, cfg.d, 1 << 30, max(log.n_nodes, 1), dummy, dummy, cfg.block_tokens)
    parents = []
    for op in log.ops:
        if op[0] == "root":
            ctx.new_root(op[1])
            parents.append(-1)
        elif op[0] == "fork":
            ctx.fork(op[1], op[2], op[3])
            parents += [op[1]] * op[2]
        elif op[0] == "fork_at":
            x = op[1]
            ctx.fork_at(x, op[2], op[3], op[4])
            t = len(parents)
            parents = [t if q == x else q for q in parents] + [x] + [x] * op[3]
        else:
            ctx.kv_commit(op[1], op[2])
    leaves = log.leaves
    n = len(leaves)
    R = np.random.default_rng(args.config).integers(0, 2, size=n).astype(np.float32)
    rw = torch.tensor(R, device="cuda")
    out = torch.empty(n, dtype=torch.float32, device="cuda")
    ws = torch.empty(max(ctx.advantage_workspace_size(leaves), 256), dtype=torch.uint8, device="cuda")
    for _ in range(args.warmup):
        ctx.tree_advantage(leaves, rw, out, ws)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        ctx.tree_advantage(leaves, rw, out, ws)
    torch.cuda.synchronize()
    call_ms = (time.perf_counter() - t0) * 1e3 / args.steps
    ctx.set_profiling(True)
    for _ in range(args.steps):
        ctx.tree_advantage(leaves, rw, out, ws)
    torch.cuda.synchronize()
    tot, cnt = ctx.profile_read(KERNEL_ADVANTAGE)
    kern_ms = tot / max(cnt, 1)
    ctx.set_profiling(False)
    pairs = sum(len(_chain(parents, x)) - 1 for x in leaves)
    line = {"metric": "TreePO advantage: trajectories/s (one call per batch of decoded leaves)",
            "value": round(n / (call_ms * 1e-3), 1), "unit": "trajectories/s", "n_gpus": 1,
            "steps": args.steps, "warmup": args.warmup, "higher_is_better": True, "dtype": "f64",
            "data": "synthetic (seeded 0/1 rewards on the config's call-log-built forest)",
            "config": {"workload": f"config {args.config}: {cfg.name}", "trajectories": n,
                       "queries": sum(1 for p in parents if p < 0), "subgroup_pairs": pairs},
            "call_ms": round(call_ms, 5), "kernel_avg_ms": round(kern_ms, 5),
            "roofline": {"bound": "latency", "note": "one workgroup over a few thousand sub-groups; the kernel "
                         "moves ~KiB, far from any throughput roof"}}
    if not args.no_cpu:
        from oracle import advantage as ADV
        reps, t0 = 0, time.perf_counter()
        while True:
            ADV.tree_advantage(parents, leaves, R.astype(np.float64))
            reps += 1
            if time.perf_counter() - t0 >= min(args.cpu_seconds, 5.0):
                break
        dt = time.perf_counter() - t0
        line["cpu_baseline"] = {"value": round(n * reps / dt, 1), "unit": "trajectories/s", "cores": 1,
                                "kind": "oracle", "sample": f"{reps} full batch(es) of {n} trajectories in {dt:.1f} s"}
    print(json.dumps(line), flush=True)


def _prefill(args):
    """Every prompt of the config prefilled in one call (fresh root nodes per
    step, the same work each time): prompt tokens/s, the kernel's duration
    (events attached to it) against the bf16 MFMA peak on the algorithmic
    FLOPs of causal attention, the per-rollout baseline (each of a prompt's w
    rollouts prefills its own copy), and the fp64 oracle on a sample."""
    import numpy as np
    import torch
    from paper_2508_17445_amd import KERNEL_PREFILL, Context
    from workloads import CONFIGS, build_call_log, node_kv_bits, query_bits
    cfg, log = CONFIGS[args.config], build_call_log(args.config)
    plens = [op[1] for op in log.ops if op[0] == "root"]
    n_p, tokens = len(plens), sum(plens)
    width = max(1, round(len(log.leaves) / n_p))           # rollouts per prompt
    blocks = sum(-(-p // 64) for p in plens)

    def dev(bits):
        return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).cuda().view(torch.bfloat16)

    kb, vb, qb = [], [], []
    for i, p in enumerate(plens):
        k, v = node_kv_bits(cfg.seed, 900_000 + i, p, cfg.hkv, cfg.d)
        kb.append(k); vb.append(v)
        qb.append(query_bits(cfg.seed, 900_000 + i, p, cfg.hq, cfg.d))
    k_all, v_all, q_all = dev(np.concatenate(kb)), dev(np.concatenate(vb)), dev(np.concatenate(qb))
    out = torch.empty((tokens, cfg.hq, cfg.d), dtype=torch.float32, device="cuda")
    lse = torch.empty((tokens, cfg.hq), dtype=torch.float32, device="cuda")

    def rig(copies):
        elems = cfg.hkv * blocks * copies * 64 * cfg.d
        kp = torch.empty(elems, dtype=torch.bfloat16, device="cuda")
        vp = torch.empty(elems, dtype=torch.bfloat16, device="cuda")
        return Context(cfg.hq, cfg.hkv, cfg.d, blocks * copies, n_p * copies, kp, vp, 64), kp, vp

    reps = args.warmup + args.steps
    ctx, kp, vp = rig(reps + 1)
    sets = [[ctx.new_root(p) for p in plens] for _ in range(reps + 1)]
    ws = torch.empty(ctx.prefill_workspace_size(sets[0], plens), dtype=torch.uint8, device="cuda")
    for i in range(args.warmup):
        ctx.prefill(sets[i], plens, q_all, k_all, v_all, cfg.scale, out, lse, ws)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.warmup, reps):
        ctx.prefill(sets[i], plens, q_all, k_all, v_all, cfg.scale, out, lse, ws)
    torch.cuda.synchronize()
    call_ms = (time.perf_counter() - t0) * 1e3 / args.steps
    ctx.set_profiling(True)
    ctx.prefill(sets[reps], plens, q_all, k_all, v_all, cfg.scale, out, lse, ws)
    torch.cuda.synchronize()
    tot, cnt = ctx.profile_read(KERNEL_PREFILL)
    kern_ms = tot / max(cnt, 1)
    # algorithmic FLOPs: token p of a prompt scores p + 1 keys (QK) and sums
    # p + 1 values (PV), 2 D flops each, for every query head
    flops = sum(p * (p + 1) // 2 for p in plens) * 4 * cfg.d * cfg.hq
    achieved = flops / (kern_ms * 1e-3) / 1e12
    del ctx, kp, vp, sets
    torch.cuda.empty_cache()
    # per-rollout baseline: each prompt prefilled once per rollout
    naive = None
    if not args.no_naive:
        nrep = 3
        ctx, kp, vp = rig(width * nrep)
        plw = plens * width
        kw, vw, qw = k_all.repeat(width, 1, 1), v_all.repeat(width, 1, 1), q_all.repeat(width, 1, 1)
        ow = torch.empty((tokens * width, cfg.hq, cfg.d), dtype=torch.float32, device="cuda")
        lw = torch.empty((tokens * width, cfg.hq), dtype=torch.float32, device="cuda")
        setw = [[ctx.new_root(p) for p in plw] for _ in range(nrep)]
        wsw = torch.empty(ctx.prefill_workspace_size(setw[0], plw), dtype=torch.uint8, device="cuda")
        ctx.prefill(setw[0], plw, qw, kw, vw, cfg.scale, ow, lw, wsw)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for i in range(1, nrep):
            ctx.prefill(setw[i], plw, qw, kw, vw, cfg.scale, ow, lw, wsw)
        torch.cuda.synchronize()
        naive = (time.perf_counter() - t0) * 1e3 / (nrep - 1)
        del ctx, kp, vp, setw, kw, vw, qw, ow, lw
        torch.cuda.empty_cache()
    line = {"metric": "prompt prefill: prompt tokens/s (causal attention + KV written once per prompt, 1 MI355X)",
            "value": round(tokens / (call_ms * 1e-3), 1), "unit": "prompt-tokens/s", "n_gpus": 1,
            "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(call_ms, 5),
            "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
            "data": "synthetic (seeded N(0,1) bf16 q/K/V, the config's prompt lengths)",
            "config": {"workload": f"config {args.config}: {cfg.name} prompts", "prompts": n_p,
                       "prompt_tokens": tokens, "rollouts_per_prompt": width, "hq": cfg.hq, "hkv": cfg.hkv,
                       "head_dim": cfg.d},
            "kernel_avg_ms": round(kern_ms, 5),
            "roofline": {"bound": "mfma", "achieved": round(achieved, 1), "peak": 2500.0, "unit": "TFLOP/s",
                         "frac": round(achieved / 2500.0, 4), "traffic": None, "kernel": "prefill_kernel",
                         "kernel_avg_ms": round(kern_ms, 5), "launches_per_step": 1,
                         "algorithmic_flops_per_launch": flops}}
    if naive is not None:
        line["per_rollout_baseline"] = {"ms_per_step": round(naive, 5), "prompt_copies": width,
                                        "speedup_shared_vs_per_rollout": round(naive / call_ms, 3)}
    if not args.no_cpu:
        from oracle import metadata as M
        from oracle import prefill as PF
        m = M.TreeModel(64, blocks, n_p)
        nodes = [m.new_root(p) for p in plens]
        m.append(nodes, plens)
        kv = {x: (kb[x], vb[x]) for x in nodes}
        q_np = np.concatenate(qb)
        budget = min(args.cpu_seconds, 10.0)
        rows_done, t0 = 0, time.perf_counter()
        rng = np.random.default_rng(0)
        while time.perf_counter() - t0 < budget:
            r = [int(x) for x in rng.integers(0, tokens, size=16)]
            PF.prefill(m, kv.__getitem__, nodes, plens, q_np, cfg.scale, rows=r)
            rows_done += len(r)
        dt = time.perf_counter() - t0
        line["cpu_baseline"] = {"value": round(rows_done / dt, 1), "unit": "prompt-tokens/s", "cores": _blas_threads(),
                                "kind": "oracle",
                                "sample": f"{rows_done} uniformly drawn prompt rows in {dt:.1f} s (fp64 numpy, "
                                          "chains materialised per call)"}
    print(json.dumps(line), flush=True)


def _chain(parents, x):
    c = []
    while x >= 0:
        c.append(x)
        x = parents[x]
    return c


def _segment_loop(args):
    """Segment-level decoding (the paper's Sec. 2.2 step loop): the config's
    tree gets a new --seg-len segment under every leaf; each step appends one
    token per leaf and decodes, on every layer.  Modes: cascade with device
    lengths (one plan for the whole segment), per-leaf baseline with device
    lengths, cascade without them (a new plan and upload every step)."""
    import torch
    from workloads import CONFIGS, CallLog, build_call_log
    from workloads.device import DeviceTree
    cfg = CONFIGS[args.config]
    base = build_call_log(args.config)
    ops, rows, nid, leaves = list(base.ops), dict(base.rows), base.n_nodes, []
    for x in base.leaves:
        ops.append(("fork", x, 1, args.seg_len))
        rows[nid] = 0
        leaves.append(nid)
        nid += 1
    log = CallLog(ops=ops, step_append=None, leaves=leaves, rows=rows, n_nodes=nid)
    n = len(leaves)
    if args.warmup + args.steps > args.seg_len:
        args.steps = args.seg_len - args.warmup
    g = torch.Generator(device="cuda").manual_seed(7)
    k_step = torch.randn(n, cfg.hkv, cfg.d, device="cuda", generator=g).to(torch.bfloat16)
    v_step = torch.randn(n, cfg.hkv, cfg.d, device="cuda", generator=g).to(torch.bfloat16)
    ones = [1] * n
    res = {}
    for name, mode, live in (("tree_live", 0, True), ("naive_live", 1, True), ("tree_replan", 0, False)):
        first = DeviceTree(cfg=cfg, log=log, live=live)
        layers = [first] + [first.clone() for _ in range(args.layers - 1)]
        bufs = [(L.outputs(), L.workspace(mode)) for L in layers]

        def step():
            for i, L in enumerate(layers):
                L.ctx.kv_append(leaves, ones, k_step, v_step)
                ws = bufs[i][1] if live else L.workspace(mode)
                fn = L.ctx.tree_decode if mode == 0 else L.ctx.paged_decode_naive
                fn(leaves, L.q, cfg.scale, bufs[i][0][0], bufs[i][0][1], ws)

        for _ in range(args.warmup):
            step()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(args.steps):
            step()
        torch.cuda.synchronize()
        ms = (time.perf_counter() - t0) * 1e3 / args.steps
        res[name] = {"ms_per_step": round(ms, 4), "ms_per_layer": round(ms / args.layers, 4),
                     "value": round(n / (ms * 1e-3), 1)}
        del layers, bufs, first
        torch.cuda.empty_cache()
    line = {
        "metric": "segment decode loop: leaf-token-steps/sec (one append + one decode per leaf, all layers)",
        "value": res["tree_live"]["value"], "unit": "leaf-token-steps/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": res["tree_live"]["ms_per_step"],
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic (seeded N(0,1) bf16 tree; random bf16 appended rows)",
        "config": {"workload": f"config {args.config}: {cfg.name} + a {args.seg_len}-token segment per leaf",
                   "leaves": n, "layers": args.layers, "hq": cfg.hq, "hkv": cfg.hkv, "head_dim": cfg.d,
                   "segment_tokens": args.seg_len},
        "modes": res,
        "speedup_live_vs_replan": round(res["tree_replan"]["ms_per_step"] / res["tree_live"]["ms_per_step"], 3),
        "speedup_tree_vs_naive": round(res["naive_live"]["ms_per_step"] / res["tree_live"]["ms_per_step"], 3),
    }
    print(json.dumps(line), flush=True)


def main():
    args = _parse()
    if args.gpus != 1:
        print(json.dumps({"error": "the decode path runs on one GPU only; it has no multi-GPU mode",
                          "n_gpus": args.gpus}))
        sys.exit(2)
    import torch
    _ensure_built()
    from paper_2508_17445_amd import KERNEL_PARTIAL
    from workloads import CONFIGS
    from workloads.device import DeviceTree

    if args.advantage:
        _advantage(args)
        return
    if args.prefill:
        _prefill(args)
        return
    if args.segment_loop:
        _segment_loop(args)
        return
    cfg = CONFIGS[args.config]
    base = DeviceTree(cfg_id=args.config)
    if args.profile_pass:
        _profile_pass(base, args)
        return
    uniq_tok, logical_tok = _unique_kv(base)
    kv_bytes_per_tok = cfg.hkv * cfg.d * 2 * 2
    uniq_bytes = uniq_tok * kv_bytes_per_tok
    n_rep = args.replicas or max(1, math.ceil(1.2e9 / uniq_bytes))
    reps = [base] + [base.clone() for _ in range(n_rep - 1)]

    _warm_gpu(reps)
    tm = _time_mode(reps, 0, args.steps, args.warmup, KERNEL_PARTIAL)
    ms, kern_ms, comb_ms, launches = tm["ms"], tm["kernel_ms"], tm["combine_ms"], tm["launches"]
    n_leaves = len(base.leaves)
    value = n_leaves / (ms * 1e-3)
    achieved_step = uniq_bytes / (ms * 1e-3) / 1e9
    achieved_kern = uniq_bytes / (kern_ms * 1e-3) / 1e9
    line = {
        "metric": METRIC,
        "value": round(value, 1),
        "unit": "leaf-token-steps/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 5),
        "ms_per_step_with_kernel_events": round(tm["ms_instrumented"], 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded N(0,1) bf16 q/K/V; call-log-built tree)",
        "config": {
            "workload": f"config {args.config}: {cfg.name}", "leaves": n_leaves, "hq": cfg.hq, "hkv": cfg.hkv,
            "head_dim": cfg.d, "unique_kv_tokens": uniq_tok, "logical_kv_tokens": logical_tok,
            "unique_kv_bytes": uniq_bytes, "share_ratio": round(logical_tok / uniq_tok, 4),
            "pool_replicas": n_rep,
        },
        "achieved_unique_kv_GBps_step": round(achieved_step, 1),
        "roofline": {"bound": "hbm", "achieved": round(achieved_kern, 1), "peak": PEAK_HBM_GBPS, "unit": "GB/s",
                     "frac": round(achieved_kern / PEAK_HBM_GBPS, 4), "traffic": _measured_traffic(args.config),
                     "kernel": "partial_kernel<128>", "kernel_avg_ms": round(kern_ms, 5),
                     "launches_per_step": launches,
                     "algorithmic_bytes_per_launch": uniq_bytes},
        "combine_avg_ms": round(comb_ms, 5),
    }
    if not args.no_naive:
        tn = _time_mode(reps, 1, args.steps, args.warmup, KERNEL_PARTIAL)
        nms = tn["ms"]
        line["naive_baseline"] = {"ms_per_step": round(nms, 5), "value": round(n_leaves / (nms * 1e-3), 1),
                                  "kernel_avg_ms": round(tn["kernel_ms"], 5),
                                  "combine_avg_ms": round(tn["combine_ms"], 5),
                                  "speedup_tree_vs_naive": round(nms / ms, 4)}
    line["probe_read_GBps"] = round(_probe_read(), 1)
    del reps, base
    torch.cuda.empty_cache()
    if not args.no_cpu:
        line["cpu_baseline"] = _cpu_baseline(args.config, args.cpu_seconds)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
