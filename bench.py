"""Decode-step throughput of segment-tree attention on one MI355X.

A step is one pass of the decode path over a batch: ``treepo_tree_decode``
(node partials + log-sum-exp combine) for every active leaf of the workload,
and, on workloads whose decode step fuses an append (config 5: one new token
per leaf), the ``treepo_kv_append`` of that token first.  Inputs are resident
in HBM when timing starts.  The default workload is the single 7B-style tree
(1 prompt of 512 tokens, segment length 512, binary forks at the first 4
boundaries, 16 leaves of 7680 tokens, Hq=28 Hkv=4 D=128, bf16 N(0,1) data).

Timing protocol: ``--replicas`` copies of the pools are built and the steps
rotate over them, so that no step finds its KV in the 256 MB Infinity Cache
(config 2's working set is ~200 MB).  After half a second of untimed
decode steps (the GPU's clocks settle), W untimed warm-up steps, then exactly
K timed steps between two device synchronisations give ``ms_per_step`` and
``value``.  A second pass of the K steps runs with library profiling on
(events at every kernel's own start and end) and gives each kernel's average
duration; a third pass of max(K, 50) steps records an event between
consecutive steps and gives the median, p10 and p90 step time.  The same
protocol times the per-leaf paged-decode baseline.  Two probes give the
attainable HBM read bandwidth (plain 16-byte loads, and the decode kernels'
own global->LDS staging), and the fp64 oracle is timed on the host cores on
the same workload (and on one core for configs 1 and 2).

A fused-append workload grows: each step appends one token to every leaf
(the plan, built once with device-resident lengths, serves every step), so
the leaves are built with room for every step of the run and the bytes of a
step are counted at that step's lengths.

Other modes: ``--config N`` (another workload), ``--segment-loop``
(segment-level decoding over several layers), ``--advantage`` (the TreePO
advantage), ``--prefill`` (prompt prefill), ``--profile-pass`` (a short run
for hardware counters) and ``--summarize`` (writes the rocprofv3 summaries
under profiles/ from a run's output).  Prints one JSON line.
"""

from __future__ import annotations

import argparse
import csv
import dataclasses
import glob
import hashlib
import json
import math
import os
import statistics
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

PEAK_HBM_GBPS = 8000.0
PROFILES = os.path.join(ROOT, "profiles")
# the decode kernels' sources: their hash gates the stored counter summaries
KERNEL_SOURCES = [os.path.join(ROOT, "paper_2508_17445_amd", "csrc", f) for f in ("kernels.hip", "partial_format.h")]
KERNEL_SHA_LABEL = "kernels.hip + partial_format.h sha256"
METRIC = "tree-decode leaf-token-steps/sec + achieved HBM GB/s on unique KV (1 MI355X)"
DIST_MIN_STEPS = 50


def _parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--config", type=int, default=2)
    ap.add_argument("--replicas", type=int, default=0, help="pool copies rotated over (0: auto)")
    ap.add_argument("--no-naive", action="store_true")
    ap.add_argument("--no-cpu", action="store_true")
    ap.add_argument("--no-probes", action="store_true")
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
    ap.add_argument("--overlap", action="store_true",
                    help="how matrix-core and vector-ALU work share a SIMD (treepo_bench_overlap): one JSON line")
    ap.add_argument("--profile-pass", action="store_true",
                    help="short run for hardware counters: --steps steps of the workload in each mode (tree, "
                         "then per-leaf), then one 1 GiB device copy whose byte counters calibrate the kernels'")
    ap.add_argument("--summarize", choices=("trace", "traffic", "mfma", "prefill", "advantage"),
                    help="write a profiles/ summary from the rocprofv3 output under --dir (the commands are in "
                         "each file): trace, traffic, mfma -> partial_kernel_config<N>_*; prefill -> "
                         "prefill_kernel_config<N>_{kernel_trace.md,counters.txt}; advantage -> "
                         "advantage_kernel_config<N>_kernel_trace.md")
    ap.add_argument("--dir", default="", help="rocprofv3 output directory for --summarize")
    return ap.parse_args()


def _ensure_built():
    from paper_2508_17445_amd.treepo import LIB_PATH
    if not os.path.exists(LIB_PATH):
        import __graft_entry__
        __graft_entry__.build()


def _kernel_sha():
    h = hashlib.sha256()
    for f in KERNEL_SOURCES:
        h.update(open(f, "rb").read())
    return h.hexdigest()


def _traffic_file(cfg_id):
    return os.path.join(PROFILES, f"partial_kernel_config{cfg_id}_traffic.txt")


def _measured_traffic(cfg_id):
    """Counter-measured HBM bytes per partial-kernel launch (tree schedule), or
    None when no summary exists for this workload or the kernel source changed
    since it was taken."""
    try:
        kv = dict(line.split(":", 1) for line in open(_traffic_file(cfg_id)).read().splitlines() if ":" in line)
        kv = {k.strip(): v.strip() for k, v in kv.items()}
        if kv.get(KERNEL_SHA_LABEL) != _kernel_sha() or int(kv.get("config", -1)) != cfg_id:
            return None
        return int(kv["traffic bytes per launch"])
    except (OSError, KeyError, ValueError):
        return None


# ---- the workload on the device --------------------------------------------------

def _with_room(log, room):
    """The call log with every node that is a decoded leaf reserving `room`
    more tokens, so that every leaf can take one more token per step for
    `room` steps (segment-level decoding: the step's token joins its path)."""
    leaves = set(log.leaves)
    ops, nid = [], 0
    for op in log.ops:
        if op[0] == "root":
            ops.append(("root", op[1] + (room if nid in leaves else 0)))
            nid += 1
        elif op[0] == "fork":
            kids = range(nid, nid + op[2])
            ops.append(("fork", op[1], op[2], op[3] + (room if any(k in leaves for k in kids) else 0)))
            nid += op[2]
        elif op[0] == "fork_at":
            raise ValueError("room for step appends is not supported on logs with fork_at")
        else:
            ops.append(op)
    return dataclasses.replace(log, ops=ops)


class Workload:
    """The config's forest on the device (and replicas of it), and one decode
    step per mode.  On a fused-append config every step first appends one
    token to every leaf (device-resident lengths: one plan serves the run);
    every timing pass then starts from a fresh copy of the forest as built
    (leaves at their configured lengths), made by ``reset``."""

    def __init__(self, cfg_id, args, room):
        from workloads import CONFIGS, build_call_log
        from workloads.device import DeviceTree
        self.cfg = CONFIGS[cfg_id]
        self.cfg_id = cfg_id
        self.no_naive = args.no_naive
        log = build_call_log(cfg_id)
        self.fused = log.step_append is not None
        if self.fused:
            base = DeviceTree(cfg=self.cfg, log=_with_room(log, room), apply_step_append=False, live=True)
        else:
            base = DeviceTree(cfg_id=cfg_id)
        self.base = base
        self.leaves = list(base.leaves)
        self.n_leaves = len(self.leaves)
        c = self.cfg
        self.kv_bytes_per_tok = c.hkv * c.d * 2 * 2
        self.uniq_tok, self.logical_tok = self._tokens(base)
        self.chain0 = self._chain_tokens(base, self.leaves[0])
        if self.fused:  # the first step's append is part of the step: count its token
            self.uniq_tok += self.n_leaves
            self.logical_tok += self.n_leaves
        uniq_bytes = self.uniq_tok * self.kv_bytes_per_tok
        self.n_rep = args.replicas or min(16, max(1, math.ceil(1.2e9 / uniq_bytes)))
        self.reps = {}
        self.bufs = {}
        self.appended = {0: 0, 1: 0}
        if self.fused:
            self.reset(0)
            self.reset(1)
        else:
            reps = [base] + [base.clone() for _ in range(self.n_rep - 1)]
            for m in (0, 1):
                self.reps[m] = reps
                self.bufs[m] = [(r.outputs(), r.workspace(m)) for r in reps]

    def reset(self, mode):
        """Fused-append workloads: fresh copies of the forest for `mode`."""
        if not self.fused:
            return
        import torch
        self.reps.pop(mode, None)
        self.bufs.pop(mode, None)
        torch.cuda.empty_cache()
        if mode == 1 and self.no_naive:
            return
        self.reps[mode] = [self.base.clone() for _ in range(self.n_rep)]
        self.bufs[mode] = [(r.outputs(), r.workspace(mode)) for r in self.reps[mode]]
        self.appended[mode] = 0

    @staticmethod
    def _tokens(dt):
        nodes = dt.ctx.export_nodes()
        used = set()
        logical = 0
        for x in dt.leaves:
            y = x
            while y != -1:
                logical += int(nodes[y][3])
                if y not in used:
                    used.add(y)
                y = int(nodes[y][0])
        return sum(int(nodes[n][3]) for n in used), logical

    @staticmethod
    def _chain_tokens(dt, x):
        nodes = dt.ctx.export_nodes()
        t = 0
        while x != -1:
            t += int(nodes[x][3])
            x = int(nodes[x][0])
        return t

    def step(self, mode, i, decode_only=False):
        """Step i of `mode` (replica i mod replicas)."""
        reps = self.reps[mode]
        j = i % len(reps)
        r = reps[j]
        if self.fused and not decode_only:
            nodes, ntok = r.log.step_append
            r.ctx.kv_append(nodes, ntok, r.step_k, r.step_v)
            if j == len(reps) - 1:
                self.appended[mode] += 1
        (out, lse), ws = self.bufs[mode][j]
        fn = r.ctx.tree_decode if mode == 0 else r.ctx.paged_decode_naive
        fn(r.leaves, r.q, r.cfg.scale, out, lse, ws)

    def step_bytes(self, first_append, count):
        """Unique KV bytes per step, averaged over `count` steps whose first
        appends the `first_append`-th token (1-based) of the pass."""
        if not self.fused:
            return self.uniq_tok * self.kv_bytes_per_tok
        extra = first_append - 1 + (count - 1) / 2.0
        return (self.uniq_tok + extra * self.n_leaves) * self.kv_bytes_per_tok


def _warm_gpu(w, seconds=0.5):
    """Decode steps (no appends) in both modes for about `seconds`, untimed,
    so that the first timed mode does not run while the GPU is still raising
    its clocks (without this the first mode measured its steps up to 10%
    slower)."""
    import torch
    t0 = time.perf_counter()
    i = 0
    modes = (0,) if w.no_naive else (0, 1)
    while time.perf_counter() - t0 < seconds:
        for m in modes:
            w.step(m, i, decode_only=True)
        i += 1
        if i % 16 == 0:
            torch.cuda.synchronize()
    torch.cuda.synchronize()


def _pct(v, q):
    v = sorted(v)
    if not v:
        return float("nan")
    k = (len(v) - 1) * q
    lo, hi = math.floor(k), math.ceil(k)
    return v[lo] + (v[hi] - v[lo]) * (k - lo)


def _time_mode(w, mode, steps, warmup):
    """Times `steps` steps of `mode` rotating over the replicas.

    Pass 1 (uninstrumented) gives the step time.  Pass 2 (same length) runs
    with library profiling: events at every kernel's own start and end give
    each kernel's average duration.  Pass 3 (max(steps, 50) steps) records a
    torch event between consecutive steps on the launch stream and gives the
    distribution of the step time.
    """
    import torch
    from paper_2508_17445_amd import KERNEL_APPEND, KERNEL_COMBINE, KERNEL_PARTIAL
    w.reset(mode)
    for i in range(warmup):
        w.step(mode, i)
    torch.cuda.synchronize()
    first = w.appended[mode] + 1
    t0 = time.perf_counter()
    for i in range(steps):
        w.step(mode, i)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    nbytes = w.step_bytes(first, steps)
    w.reset(mode)
    for r in w.reps[mode]:
        r.ctx.set_profiling(True)
    torch.cuda.synchronize()
    for i in range(steps):
        w.step(mode, i)
    torch.cuda.synchronize()
    kern = {}
    for kind, name in ((KERNEL_PARTIAL, "partial"), (KERNEL_COMBINE, "combine"), (KERNEL_APPEND, "append")):
        tot, n = 0.0, 0
        for r in w.reps[mode]:
            a, b = r.ctx.profile_read(kind)
            tot += a
            n += b
        kern[name] = (tot / n if n else None, n // max(steps, 1))
    for r in w.reps[mode]:
        r.ctx.set_profiling(False)
    nd = max(steps, DIST_MIN_STEPS)
    w.reset(mode)
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(nd + 1)]
    torch.cuda.synchronize()
    for i in range(nd):
        ev[i].record()
        w.step(mode, i)
    ev[nd].record()
    torch.cuda.synchronize()
    per = [ev[i].elapsed_time(ev[i + 1]) for i in range(nd)]
    return {"ms": (t1 - t0) * 1e3 / steps, "bytes": nbytes, "kern": kern, "first": first,
            "dist": {"steps": nd, "median_ms": round(_pct(per, 0.5), 5), "p10_ms": round(_pct(per, 0.1), 5),
                     "p90_ms": round(_pct(per, 0.9), 5)}}


# ---- probes and the oracle -------------------------------------------------------

def _timed(fn, iters):
    import torch
    fn()
    torch.cuda.synchronize()
    st, en = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    st.record()
    for _ in range(iters):
        fn()
    en.record()
    torch.cuda.synchronize()
    return st.elapsed_time(en) / iters


def _probes(work_bytes):
    """Attainable HBM read bandwidth: a plain 16-byte-load read of 4 GiB, and
    the decode kernels' staging (16-byte non-temporal global->LDS loads into a
    ring of four 16 KiB buffers, three in flight, a barrier per chunk; 512
    workgroups, one contiguous share each) on 4 GiB and on rotating buffers
    the size of the workload."""
    import torch
    from paper_2508_17445_amd import bench_read, bench_stream
    wgs, chunk = 512, 16384
    big = 4 << 30
    src = torch.empty(big, dtype=torch.uint8, device="cuda")
    sink = torch.empty(8192, dtype=torch.float32, device="cuda")
    res = {"plain_read_4GiB_GBps": round(big / (_timed(lambda: bench_read(src, big, sink), 10) * 1e-3) / 1e9, 1),
           "staging_4GiB_GBps": round(big / (_timed(lambda: bench_stream(src, big, sink, 3, wgs), 10) * 1e-3)
                                      / 1e9, 1)}
    step = wgs * chunk
    # rotating buffers of the workload's size (at most the 4 GiB source; at
    # most 20 of them), every one inside the source
    size = min(big // step, max(1, int(work_bytes) // step)) * step
    n = max(1, min(big // size, 20))
    assert size % step == 0 and 0 < n * size <= big

    it = [0]

    def rot():
        off = (it[0] % n) * size
        assert off + size <= big
        bench_stream(src[off:off + size], size, sink, 3, wgs)
        it[0] += 1
    res["staging_workload_size_GBps"] = round(size / (_timed(rot, 4 * n) * 1e-3) / 1e9, 1)
    res["staging_workload_bytes"] = size
    del src
    torch.cuda.empty_cache()
    return res


def _blas_threads():
    try:
        from threadpoolctl import threadpool_info
        return max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:
        return 1


def _oracle_rate(cfg_id, seconds, one_core=False):
    """The fp64 oracle over whole decode steps of the workload: leaf-token-steps/s."""
    import contextlib
    from oracle import attention as A
    from oracle import metadata as M
    from workloads import CONFIGS, build_call_log, query_bits
    from workloads.device import NodeData
    cfg, log = CONFIGS[cfg_id], build_call_log(cfg_id)
    model = M.replay(log, cfg.block_tokens, 1 << 30, 1 << 30)
    # workloads of many trees: the leaves of the first tree (a bounded sample)
    pos = list(range(len(log.leaves)))
    if len(pos) > 64:
        first = model.nodes[log.leaves[0]]["tree_id"]
        pos = [p for p, x in enumerate(log.leaves) if model.nodes[x]["tree_id"] == first]
    data = NodeData(cfg, log)
    data.prefetch(sorted({n for p in pos for n in model.chain(log.leaves[p])}))
    q = query_bits(cfg.seed, 0, len(log.leaves), cfg.hq, cfg.d)
    ctx = contextlib.nullcontext()
    if one_core:
        from threadpoolctl import threadpool_limits
        ctx = threadpool_limits(limits=1)
    with ctx:
        threads = _blas_threads()
        reps, t0 = 0, time.perf_counter()
        while True:
            A.tree_decode(model, data, log.leaves, q, cfg.scale,
                          positions=None if len(pos) == len(log.leaves) else pos)
            reps += 1
            if time.perf_counter() - t0 >= seconds:
                break
        dt = time.perf_counter() - t0
    return len(pos) * reps / dt, reps, dt, threads, len(pos), len(log.leaves)


def _cpu_baseline(cfg_id, seconds):
    rate, reps, dt, threads, n_pos, n_all = _oracle_rate(cfg_id, seconds)
    host = len(os.sched_getaffinity(0))
    what = "full decode step(s) of the same workload" if n_pos == n_all else \
        f"decode(s) of the {n_pos} leaves of its first tree (of {n_all} leaves)"
    out = {"value": round(rate, 2), "unit": "leaf-token-steps/s", "cores": min(host, threads), "kind": "oracle",
           "sample": f"{reps} {what} (fp64 numpy, chains materialised per leaf) in {dt:.1f} s; host has "
                     f"{host} cores, BLAS threads {threads}"}
    if cfg_id in (1, 2):
        one = {}
        for c in (1, 2):
            r1, n1, d1, _, _, _ = _oracle_rate(c, min(seconds, 4.0), one_core=True)
            one[f"config{c}"] = {"value": round(r1, 2), "steps": n1, "seconds": round(d1, 2)}
        out["one_core"] = one
    return out


# ---- hardware-counter runs and their summaries -----------------------------------

def _profile_pass(cfg_id, args):
    """--steps steps of the workload in each mode (tree, then per-leaf), then
    one 1 GiB device copy, nothing else on the GPU (fused-append workloads
    append in every step, as in the bench)."""
    import torch
    from paper_2508_17445_amd import bench_copy
    w = Workload(cfg_id, args, args.steps + 8)
    for mode in (0, 1):
        for i in range(args.steps):
            w.step(mode, i)
        torch.cuda.synchronize()
    nbytes = 1 << 30
    src = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
    dst = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
    bench_copy(dst, src, nbytes)
    torch.cuda.synchronize()
    print(json.dumps({"profile_pass": True, "config": cfg_id, "steps_per_mode": args.steps,
                      "copy_bytes": nbytes}), flush=True)


def _csv_rows(d, suffix):
    files = sorted(glob.glob(os.path.join(d, "**", f"*{suffix}"), recursive=True))
    if not files:
        raise SystemExit(f"no *{suffix} under {d}")
    rows = []
    for f in files:
        rows += list(csv.DictReader(open(f)))
    return rows


def _bench_line(d):
    for f in sorted(glob.glob(os.path.join(d, "*.json"))):
        for line in open(f).read().splitlines()[::-1]:
            if line.startswith("{") and '"metric"' in line:
                return json.loads(line)
    raise SystemExit(f"no bench JSON line under {d}")


def _workload_name(cfg_id):
    from workloads import CONFIGS
    return CONFIGS[cfg_id].name


def _summarize_trace(cfg_id, d):
    """profiles/partial_kernel_config<N>_kernel_trace.md from a kernel trace
    of one bench run (its JSON line saved as a .json file in the same dir)."""
    b = _bench_line(d)
    rows = _csv_rows(d, "kernel_trace.csv")
    rows.sort(key=lambda r: int(r["Start_Timestamp"]))

    def dur(r):
        return (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3

    steps, warm = b["steps"], b["warmup"]
    per_mode = warm + 2 * steps + max(steps, DIST_MIN_STEPS)   # the launches of _time_mode per mode
    modes = 2 if "naive_baseline" in b else 1
    lines, avg = [], {}
    names = ("partial_kernel", "combine_kernel") + (("kv_append_kernel",) if "append_avg_ms" in b else ())
    for kname in names:
        ks = [r for r in rows if kname in r["Kernel_Name"]]
        if not ks:
            continue
        ks = ks[-modes * per_mode:]
        for m in range(modes):
            blk = ks[m * per_mode:(m + 1) * per_mode][warm:]
            v = [dur(r) for r in blk]
            label = ("tree schedule", "per-leaf baseline")[m]
            avg[(kname, m)] = statistics.mean(v)
            lines.append(f"| {kname}, {label} | {blk[0]['Grid_Size_X'] if 'Grid_Size_X' in blk[0] else blk[0].get('Grid_Size', '')} "
                         f"| {len(v)} | {statistics.mean(v):.2f} | {statistics.median(v):.2f} | "
                         f"{_pct(v, 0.1):.2f} | {_pct(v, 0.9):.2f} | {min(v):.2f} | {max(v):.2f} |")
    stats = []
    try:
        for r in _csv_rows(d, "kernel_stats.csv"):
            if any(k in r["Name"] for k in names):
                stats.append(f"| {r['Name'][:60]} | {r['Calls']} | {float(r['AverageNs']) / 1e3:.2f} | "
                             f"{float(r['MinNs']) / 1e3:.2f} | {float(r['MaxNs']) / 1e3:.2f} |")
    except SystemExit:
        pass
    alg = b["roofline"]["algorithmic_bytes_per_launch"]
    t_avg = avg[("partial_kernel", 0)]
    txt = f"""# Kernel trace: decode step on config {cfg_id} ({_workload_name(cfg_id)})

Command (repository root `$R` on the MI355X host):

```
cd /tmp && export TMPDIR=/tmp && rocprofv3 --kernel-trace --stats --output-format csv -d $R/gpurun_out/prof/c{cfg_id}/trace -o run -- python3 -u $R/bench.py --config {cfg_id} --steps {steps} --warmup {warm} --no-cpu --no-probes --no-naive > $R/gpurun_out/prof/c{cfg_id}/trace/bench.json
python3 bench.py --summarize trace --config {cfg_id} --dir gpurun_out/prof/c{cfg_id}/trace
```

Per-dispatch durations from the kernel trace (microseconds), the launches of
the bench's timing passes after the W = {warm} warm-up steps of each mode
(uninstrumented pass, events pass, distribution pass: {per_mode - warm} per mode).

| kernel, schedule | grid (threads) | dispatches | avg | median | p10 | p90 | min | max |
|---|---|---|---|---|---|---|---|---|
""" + "\n".join(lines) + f"""

rocprofv3 `--stats` summary of the same run (every dispatch of the kernel,
the untimed warm-up steps included; microseconds):

| kernel | calls | avg | min | max |
|---|---|---|---|---|
""" + "\n".join(stats) + f"""

Algorithmic bytes per tree launch (unique KV of the decoded chains at the
timed steps): {alg} -> {alg / t_avg / 1e6:.3f} TB/s = {alg / t_avg / 1e6 / 8:.3f} of 8 TB/s on the
kernel-trace average ({t_avg:.2f} us).  The same run's bench line: partial kernel
{b['roofline']['kernel_avg_ms'] * 1e3:.2f} us on events attached to the kernel (frac {b['roofline']['frac']}),
step {b['ms_per_step'] * 1e3:.2f} us (median {b['step_distribution']['median_ms'] * 1e3:.2f} us over
{b['step_distribution']['steps']} steps).

{KERNEL_SHA_LABEL}: {_kernel_sha()}
"""
    path = os.path.join(PROFILES, f"partial_kernel_config{cfg_id}_kernel_trace.md")
    open(path, "w").write(txt)
    print(txt)


def _summarize_traffic(cfg_id, d):
    """profiles/partial_kernel_config<N>_traffic.txt from two counter runs of
    --profile-pass (FETCH_SIZE in <dir>/fetch, WRITE_SIZE in <dir>/write)."""
    from workloads import CONFIGS, build_call_log
    cfg = CONFIGS[cfg_id]

    def agg(sub, counter):
        rows = [r for r in _csv_rows(os.path.join(d, sub), "counter_collection.csv") if r["Counter_Name"] == counter]
        rows.sort(key=lambda r: int(r["Dispatch_Id"]))
        part = [float(r["Counter_Value"]) for r in rows if "partial_kernel" in r["Kernel_Name"]]
        copy = [float(r["Counter_Value"]) for r in rows if "copy_kernel" in r["Kernel_Name"]]
        n = len(part) // 2   # tree decodes first, then the per-leaf ones
        return statistics.mean(part[:n]), statistics.mean(part[n:]), statistics.mean(copy), n

    ft, fn, fc, n = agg("fetch", "FETCH_SIZE")
    wt, wn, wc, _ = agg("write", "WRITE_SIZE")
    fs, ws = 1048576 / fc, 1048576 / wc
    fb, wb = round(ft * 1024 * fs), round(wt * 1024 * ws)
    from workloads.device import DeviceTree  # noqa: F401  (same workload definition)
    log = build_call_log(cfg_id)
    alg = _algorithmic_bytes(cfg_id, log)
    txt = f"""HBM traffic of the node-partial kernel, decode workload config {cfg_id} ({cfg.name}, Hq={cfg.hq} Hkv={cfg.hkv} D={cfg.d})
Commands (repository root $R on the MI355X host; each counter in its own run):
  cd /tmp && export TMPDIR=/tmp
  rocprofv3 --pmc FETCH_SIZE --output-format csv -d $R/gpurun_out/prof/c{cfg_id}/pmc/fetch -o run -- python3 $R/bench.py --profile-pass --config {cfg_id} --steps {n}
  rocprofv3 --pmc WRITE_SIZE --output-format csv -d $R/gpurun_out/prof/c{cfg_id}/pmc/write -o run -- python3 $R/bench.py --profile-pass --config {cfg_id} --steps {n}
  python3 bench.py --summarize traffic --config {cfg_id} --dir gpurun_out/prof/c{cfg_id}/pmc
The profile pass runs {n} tree decode steps, {n} per-leaf decode steps and one 1 GiB device copy.
Calibration on the 1 GiB copy kernel: FETCH_SIZE reads {fc:.1f} KiB for 1048576 KiB read (scale {fs:.4f}); WRITE_SIZE reads {wc:.1f} KiB for 1048576 KiB written (scale {ws:.4f}).
partial_kernel<128>, tree schedule, mean of {n} dispatches:
  FETCH_SIZE {ft:.1f} KiB -> {fb} bytes read
  WRITE_SIZE {wt:.1f} KiB -> {wb} bytes written (partial rows)
partial_kernel<128>, per-leaf baseline: FETCH_SIZE {fn:.1f} KiB ({round(fn * 1024 * fs)} bytes), WRITE_SIZE {wn:.1f} KiB ({round(wn * 1024 * ws)} bytes)
Algorithmic bytes per launch (unique KV of the decoded chains): {alg}; measured traffic / algorithmic = {(fb + wb) / alg:.4f}
config: {cfg_id}
{KERNEL_SHA_LABEL}: {_kernel_sha()}
fetch bytes per launch: {fb}
write bytes per launch: {wb}
traffic bytes per launch: {fb + wb}
"""
    open(_traffic_file(cfg_id), "w").write(txt)
    print(txt)


def _host_plan_ctx(cfg_id):
    """A host-only context holding the workload's tree (metadata appends; the
    pools are never touched), for exporting the plans the GPU ran."""
    from paper_2508_17445_amd import Context
    from workloads import CONFIGS, build_call_log
    cfg, log = CONFIGS[cfg_id], build_call_log(cfg_id)
    from workloads.device import pool_blocks
    fake = 0x10000
    ctx = Context(cfg.hq, cfg.hkv, cfg.d, pool_blocks(log, cfg.block_tokens) + 1, max(log.n_nodes, 1), fake,
                  fake + 64, cfg.block_tokens)
    for op in log.ops:
        if op[0] == "root":
            ctx.new_root(op[1])
        elif op[0] == "fork":
            ctx.fork(op[1], op[2], op[3])
        elif op[0] == "fork_at":
            ctx.fork_at(op[1], op[2], op[3], op[4])
        else:
            ctx.kv_commit(op[1], op[2])
    if log.step_append is not None:
        ctx.kv_commit(*log.step_append)
    return ctx, cfg, log


def _summarize_mfma(cfg_id, d):
    """profiles/partial_kernel_config<N>_mfma.txt from one SQ counter pass of
    --profile-pass (MFMA instructions, MFMA busy cycles) and the plans the
    library makes for the workload (predicted MFMA count, MFMA row fill)."""
    ctx, cfg, log = _host_plan_ctx(cfg_id)
    rows = [r for r in _csv_rows(d, "counter_collection.csv") if "partial_kernel" in r["Kernel_Name"]]
    disp = sorted({int(r["Dispatch_Id"]) for r in rows})
    first = set(disp[:len(disp) // 2])   # the profile pass runs the tree decodes first, then the per-leaf ones
    by = {0: {}, 1: {}}
    for r in rows:
        by[0 if int(r["Dispatch_Id"]) in first else 1].setdefault(r["Counter_Name"], []).append(
            float(r["Counter_Value"]))
    D = cfg.d

    def per_tile(n_rows):
        # MFMAs per KV tile of a piece: column-split pieces (<= 32 rows) run
        # 8 QK MFMAs on each of the 4 waves and split the PV d-blocks over
        # them; larger pieces run 8 QK + 2 (hi, lo) x D/16 PV MFMAs per 16-row block
        if n_rows <= 16:
            return 4 * (8 + 2 * (D // 16 // 4))
        if n_rows <= 32:
            return 4 * (8 + 2 * (D // 16 // 2))
        return math.ceil(n_rows / 16) * (8 + 2 * (D // 16))

    out = []
    for mode, name in ((0, "tree schedule"), (1, "per-leaf baseline")):
        pieces, _, _, ns = ctx.export_plan(log.leaves, mode)
        m = {k: statistics.mean(v) for k, v in by[mode].items()}
        exp = sum(int(p[5]) * per_tile(int(p[2])) for p in pieces)

        def cls(ps):
            t = sum(int(p[5]) for p in ps)
            mf = sum(int(p[5]) * per_tile(int(p[2])) for p in ps)
            rb = sum(int(p[5]) * 16 * math.ceil(int(p[2]) / 16) for p in ps)
            useful = sum(int(p[5]) * int(p[2]) for p in ps)
            return t, mf, (useful / rb if rb else 0.0)

        ts, ms_, fs = cls([p for p in pieces if p[1] > 1])
        t1, m1, f1 = cls([p for p in pieces if p[1] == 1])
        gui = m["GRBM_GUI_ACTIVE"] / 8   # summed over the 8 XCDs
        util = m["SQ_VALU_MFMA_BUSY_CYCLES"] / (gui * 1024)
        out.append(
            f"partial_kernel<{D}>, {name} (grid {ns} x 256), mean of {len(by[mode]['GRBM_GUI_ACTIVE'])} dispatches:\n"
            f"  SQ_INSTS_VALU_MFMA_BF16      {m['SQ_INSTS_VALU_MFMA_BF16']:.0f} MFMA instructions "
            f"(v_mfma_f32_16x16x32_bf16); the plan predicts {exp}\n"
            f"  SQ_INSTS_VALU_MFMA_MOPS_BF16 {m['SQ_INSTS_VALU_MFMA_MOPS_BF16']:.0f} -> "
            f"{m['SQ_INSTS_VALU_MFMA_MOPS_BF16'] * 512 / 1e9:.3f} GFLOP issued per launch\n"
            f"  SQ_VALU_MFMA_BUSY_CYCLES     {m['SQ_VALU_MFMA_BUSY_CYCLES']:.0f}; GRBM_GUI_ACTIVE "
            f"{m['GRBM_GUI_ACTIVE']:.0f} (8 XCDs) -> MFMA busy {100 * util:.1f}% of 1024 SIMDs x {gui:.0f} cycles\n"
            f"  SQ_INSTS_VALU {m['SQ_INSTS_VALU']:.0f}, SQ_WAVES {m['SQ_WAVES']:.0f}, "
            f"SQ_BUSY_CU_CYCLES {m['SQ_BUSY_CU_CYCLES']:.0f}\n"
            f"  KV tiles of shared-node pieces (more than one leaf): {ts} tiles, {ms_} MFMAs "
            f"({100 * ms_ / max(exp, 1):.1f}% of the launch), MFMA row fill {100 * fs:.1f}%\n"
            f"  KV tiles of one-leaf pieces: {t1} tiles, {m1} MFMAs, MFMA row fill {100 * f1:.1f}%")
    ctx.close()
    counters = ("SQ_INSTS_VALU_MFMA_BF16 SQ_INSTS_VALU_MFMA_MOPS_BF16 SQ_VALU_MFMA_BUSY_CYCLES SQ_BUSY_CU_CYCLES "
                "SQ_WAVES SQ_INSTS_VALU GRBM_GUI_ACTIVE")
    txt = f"""MFMA use of the node-partial kernel, decode workload config {cfg_id} ({cfg.name}, Hq={cfg.hq} Hkv={cfg.hkv} D={cfg.d})
Commands (repository root $R on the MI355X host; one counter pass):
  cd /tmp && export TMPDIR=/tmp
  rocprofv3 --pmc {counters} --output-format csv -d $R/gpurun_out/prof/c{cfg_id}/mfma -o run -- python3 $R/bench.py --profile-pass --config {cfg_id} --steps 10
  python3 bench.py --summarize mfma --config {cfg_id} --dir gpurun_out/prof/c{cfg_id}/mfma
The profile pass runs 10 tree decodes, 10 per-leaf decodes and one 1 GiB device copy.
Prediction from the plan (treepo_export_plan): per KV tile, a piece of <= 16 query rows issues 4 waves x (8 QK + {2 * (D // 64)} PV) MFMAs,
17-32 rows 4 x (8 + {2 * (D // 32)}), more rows {8 + 2 * (D // 16)} per 16-row block (8 QK + {2 * (D // 16)} PV; PV runs twice, on the hi and lo bf16 parts of P).
Row fill = query rows / (16 x row blocks) of the MFMA tiles, weighted by KV tiles.

""" + "\n".join(out) + f"""

{KERNEL_SHA_LABEL}: {_kernel_sha()}
"""
    path = os.path.join(PROFILES, f"partial_kernel_config{cfg_id}_mfma.txt")
    open(path, "w").write(txt)
    print(txt)


def _summarize_prefill(cfg_id, d):
    """profiles/prefill_kernel_config<N>_{kernel_trace.md,counters.txt} from a
    kernel trace of `bench.py --prefill` (<dir>/trace, its JSON line saved
    there) and two SQ counter passes (<dir>/sq, <dir>/mfma)."""
    from workloads import CONFIGS, build_call_log
    cfg, log = CONFIGS[cfg_id], build_call_log(cfg_id)
    plens = [op[1] for op in log.ops if op[0] == "root"]
    b = _bench_line(os.path.join(d, "trace"))
    rows = _csv_rows(os.path.join(d, "trace"), "kernel_trace.csv")
    rows.sort(key=lambda r: int(r["Start_Timestamp"]))

    def dur(r):
        return (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3

    def stats(v):
        return f"{len(v)} | {statistics.mean(v):.2f} | {statistics.median(v):.2f} | {min(v):.2f} | {max(v):.2f}"

    pf = [r for r in rows if "prefill_kernel" in r["Kernel_Name"]]
    ap = [dur(r) for r in rows if "kv_append_dev_kernel" in r["Kernel_Name"]]
    warm, steps = b["warmup"], b["steps"]
    timed = pf[warm:warm + steps]
    flops = b["roofline"]["algorithmic_flops_per_launch"]
    avg = statistics.mean(dur(r) for r in timed)
    grid = timed[0].get("Grid_Size_X", timed[0].get("Grid_Size", ""))
    head = f"prefill of the config-{cfg_id} prompts ({len(plens)} prompts, {sum(plens):,} tokens, " \
           f"Hq={cfg.hq} Hkv={cfg.hkv} D={cfg.d})"
    naive = b.get("per_rollout_baseline")
    txt = f"""# Kernel trace: {head}

Commands (repository root `$R` on the MI355X host):

```
cd /tmp && export TMPDIR=/tmp && rocprofv3 --kernel-trace --stats --output-format csv -d $R/gpurun_out/pfprof/c{cfg_id}/trace -o run -- python3 -u $R/bench.py --prefill --config {cfg_id} --steps {steps} --warmup {warm} --no-cpu > $R/gpurun_out/pfprof/c{cfg_id}/trace/bench.json
python3 bench.py --summarize prefill --config {cfg_id} --dir gpurun_out/pfprof/c{cfg_id}
```

Each step is one `treepo_prefill` call over all {len(plens)} prompts (fresh root nodes
every step): one KV-append launch (pieces read from the uploaded tables), then one prefill launch.
Prefill dispatches in order: {warm} warm-up, {steps} timed, 1 with events attached (then the
per-rollout baseline's).

| kernel | grid (threads) | dispatches | avg us | median us | min us | max us |
|---|---|---|---|---|---|---|
| prefill_kernel<{cfg.d}>, timed steps | {grid} | {stats([dur(r) for r in timed])} |
| kv_append_dev_kernel<{cfg.d}> (all calls) | - | {stats(ap)} |

Algorithmic FLOPs per launch (causal QK and PV, 4 D flops per query-key pair
and query head): {flops} -> {flops / (avg * 1e-6) / 1e12:.1f} TFLOP/s on the
trace average = {flops / (avg * 1e-6) / 1e12 / 2500:.3f} of the 2.5 PFLOP/s
bf16 dense peak.  The same run's bench line: the kernel at
{b["kernel_avg_ms"] * 1e3:.1f} us with events attached to it
({b["roofline"]["achieved"]} TFLOP/s), the whole call (append + host tables
+ upload + prefill) at {b["ms_per_step"] * 1e3:.1f} us""" + (f""", and prefilling every
prompt once per rollout ({naive["prompt_copies"]} copies) at {naive["ms_per_step"] * 1e3:.0f} us
({naive["speedup_shared_vs_per_rollout"]}x).""" if naive else ".") + f"""

{KERNEL_SHA_LABEL}: {_kernel_sha()}
"""
    open(os.path.join(PROFILES, f"prefill_kernel_config{cfg_id}_kernel_trace.md"), "w").write(txt)
    print(txt)
    agg = {}
    for sub in ("sq", "mfma"):
        for r in _csv_rows(os.path.join(d, sub), "counter_collection.csv"):
            if "prefill_kernel" in r["Kernel_Name"]:
                agg.setdefault(r["Counter_Name"], []).append(float(r["Counter_Value"]))
    m = {k: statistics.mean(v) for k, v in agg.items()}
    busy = m["SQ_BUSY_CU_CYCLES"]
    sq = ("SQ_VALU_MFMA_BUSY_CYCLES SQ_BUSY_CU_CYCLES SQ_INSTS_VALU SQ_INSTS_LDS SQ_LDS_BANK_CONFLICT "
          "SQ_ACTIVE_INST_VALU SQ_ACTIVE_INST_LDS SQ_WAVE_CYCLES")
    mf = "SQ_INSTS_VALU_MFMA_BF16 SQ_INSTS_VALU_MFMA_MOPS_BF16 SQ_WAVES GRBM_GUI_ACTIVE"
    txt2 = f"""SQ counters of the {head}
Commands (repository root $R on the MI355X host; each pass its own run):
  cd /tmp && export TMPDIR=/tmp
  rocprofv3 --pmc {sq} --output-format csv -d $R/gpurun_out/pfprof/c{cfg_id}/sq -o run -- python3 $R/bench.py --prefill --config {cfg_id} --steps 3 --warmup 1 --no-cpu --no-naive
  rocprofv3 --pmc {mf} --output-format csv -d $R/gpurun_out/pfprof/c{cfg_id}/mfma -o run -- python3 $R/bench.py --prefill --config {cfg_id} --steps 3 --warmup 1 --no-cpu --no-naive
  python3 bench.py --summarize prefill --config {cfg_id} --dir gpurun_out/pfprof/c{cfg_id}
Means over the prefill dispatches of each run ({len(agg.get("SQ_BUSY_CU_CYCLES", []))} and {len(agg.get("SQ_WAVES", []))}):
""" + "".join(f"  {k}: {v:.0f}\n" for k, v in sorted(m.items())) + f"""Derived (per CU, 256 CUs; MFMA busy counted per SIMD, 4 per CU):
  MFMA pipe busy: {m["SQ_VALU_MFMA_BUSY_CYCLES"] / 4 / busy:.3f} of the CU busy cycles
  VALU active: {m["SQ_ACTIVE_INST_VALU"] / busy:.3f}; LDS active: {m["SQ_ACTIVE_INST_LDS"] / busy:.3f}; LDS bank-conflict cycles: {m["SQ_LDS_BANK_CONFLICT"] / busy:.3f}
  MFMA instructions per launch {m["SQ_INSTS_VALU_MFMA_BF16"]:.0f} -> {m["SQ_INSTS_VALU_MFMA_BF16"] * 16384 / flops:.2f} x the algorithmic FLOPs executed
{KERNEL_SHA_LABEL}: {_kernel_sha()}
"""
    open(os.path.join(PROFILES, f"prefill_kernel_config{cfg_id}_counters.txt"), "w").write(txt2)
    print(txt2)


def _summarize_advantage(cfg_id, d):
    """profiles/advantage_kernel_config<N>_kernel_trace.md from the kernel
    statistics of one `bench.py --advantage` run (its JSON line saved in
    <dir>)."""
    b = _bench_line(d)
    stats = [r for r in _csv_rows(d, "kernel_stats.csv") if "advantage_kernel" in r["Name"]]
    s0 = stats[0]
    txt = f"""# Kernel trace: TreePO advantage over config {cfg_id}'s decoded leaves ({_workload_name(cfg_id)})

Commands (repository root `$R` on the MI355X host):

```
cd /tmp && export TMPDIR=/tmp && rocprofv3 --kernel-trace --stats --output-format csv -d $R/gpurun_out/advprof/c{cfg_id} -o run -- python3 -u $R/bench.py --advantage --config {cfg_id} --steps {b["steps"]} --warmup {b["warmup"]} --no-cpu > $R/gpurun_out/advprof/c{cfg_id}/bench.json
python3 bench.py --summarize advantage --config {cfg_id} --dir gpurun_out/advprof/c{cfg_id}
```

rocprofv3 `--stats` ({b["warmup"]} warm-up + {b["steps"]} timed calls + the calls with the
library's events attached to the kernel):

| kernel | calls | avg us | min us | max us |
|---|---|---|---|---|
| advantage_kernel | {s0["Calls"]} | {float(s0["AverageNs"]) / 1e3:.2f} | {float(s0["MinNs"]) / 1e3:.2f} | {float(s0["MaxNs"]) / 1e3:.2f} |

The bench line of the same run: {b["call_ms"] * 1e3:.1f} us per call back to back (host index
arrays cached for the tree shape and leaf list, their upload through pinned
staging, the kernel), {b.get("kernel_avg_ms", float("nan")) * 1e3:.1f} us on the kernel's attached events,
{b["value"] / 1e6:.1f} M trajectories/s.  One workgroup; the time is dependent global
loads (sub-group members, each pair's sub-group mean), not bandwidth.

advantage.hip sha256: {hashlib.sha256(open(os.path.join(ROOT, "paper_2508_17445_amd", "csrc", "advantage.hip"), "rb").read()).hexdigest()}
"""
    open(os.path.join(PROFILES, f"advantage_kernel_config{cfg_id}_kernel_trace.md"), "w").write(txt)
    print(txt)


def _algorithmic_bytes(cfg_id, log):
    """Unique KV bytes of a decode step of the workload (with its fused append)."""
    from workloads import CONFIGS
    cfg = CONFIGS[cfg_id]
    parent = {}
    nid = 0
    for op in log.ops:
        if op[0] == "root":
            parent[nid] = -1
            nid += 1
        elif op[0] == "fork":
            for k in range(op[2]):
                parent[nid + k] = op[1]
            nid += op[2]
        elif op[0] == "fork_at":
            t = nid
            for y, p in list(parent.items()):
                if p == op[1]:
                    parent[y] = t
            parent[t] = op[1]
            for k in range(op[3]):
                parent[t + 1 + k] = op[1]
            nid += 1 + op[3]
    used = set()
    for x in log.leaves:
        while x != -1 and x not in used:
            used.add(x)
            x = parent[x]
    return sum(log.rows[n] for n in used) * cfg.hkv * cfg.d * 4


# ---- the decode line ---------------------------------------------------------------

def _decode_line(args):
    import torch
    cfg_id = args.config
    w = Workload(cfg_id, args, max(args.warmup + args.steps, DIST_MIN_STEPS) + 8)
    cfg = w.cfg
    _warm_gpu(w)
    tm = _time_mode(w, 0, args.steps, args.warmup)
    ms, nbytes = tm["ms"], tm["bytes"]
    kern_ms, launches = tm["kern"]["partial"]
    comb_ms = tm["kern"]["combine"][0]
    value = w.n_leaves / (ms * 1e-3)
    achieved_kern = nbytes / (kern_ms * 1e-3) / 1e9
    achieved_step = nbytes / (ms * 1e-3) / 1e9
    line = {
        "metric": METRIC,
        "value": round(value, 1),
        "unit": "leaf-token-steps/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded N(0,1) bf16 q/K/V; call-log-built tree)",
        "config": {
            "workload": f"config {cfg_id}: {cfg.name}" + (" (append of one token per leaf + decode per step)"
                                                          if w.fused else ""),
            "leaves": w.n_leaves, "hq": cfg.hq, "hkv": cfg.hkv, "head_dim": cfg.d,
            "unique_kv_tokens": w.uniq_tok, "logical_kv_tokens": w.logical_tok,
            "unique_kv_bytes_per_step": round(nbytes), "share_ratio": round(w.logical_tok / w.uniq_tok, 4),
            "pool_replicas": len(w.reps[0]),
        },
        "achieved_unique_kv_GBps_step": round(achieved_step, 1),
        "call_level_frac": round(achieved_step / PEAK_HBM_GBPS, 4),
        "step_distribution": tm["dist"],
        "roofline": {"bound": "hbm", "achieved": round(achieved_kern, 1), "peak": PEAK_HBM_GBPS, "unit": "GB/s",
                     "frac": round(achieved_kern / PEAK_HBM_GBPS, 4), "traffic": _measured_traffic(cfg_id),
                     "kernel": "partial_kernel<128>", "kernel_avg_ms": round(kern_ms, 5),
                     "launches_per_step": launches, "algorithmic_bytes_per_launch": round(nbytes)},
        "combine_avg_ms": round(comb_ms, 5),
    }
    if w.fused:
        line["config"]["leaf_chain_tokens_timed"] = [w.chain0 + tm["first"], w.chain0 + tm["first"] + args.steps - 1]
        ap_ms = tm["kern"]["append"][0]
        line["append_avg_ms"] = round(ap_ms, 5) if ap_ms is not None else None
    if not args.no_naive:
        tn = _time_mode(w, 1, args.steps, args.warmup)
        nms = tn["ms"]
        line["naive_baseline"] = {"ms_per_step": round(nms, 5), "value": round(w.n_leaves / (nms * 1e-3), 1),
                                  "kernel_avg_ms": round(tn["kern"]["partial"][0], 5),
                                  "combine_avg_ms": round(tn["kern"]["combine"][0], 5),
                                  "step_distribution": tn["dist"],
                                  "speedup_tree_vs_naive": round(nms / ms, 4),
                                  "speedup_median": round(tn["dist"]["median_ms"] / tm["dist"]["median_ms"], 4)}
    uniq = w.uniq_tok * w.kv_bytes_per_tok
    w.reps.clear()
    w.bufs.clear()
    del w
    torch.cuda.empty_cache()
    if not args.no_probes:
        pr = _probes(uniq)
        line["probes"] = pr
        line["roofline"]["frac_of_staging_probe"] = round(achieved_kern / pr["staging_workload_size_GBps"], 4)
    if not args.no_cpu:
        line["cpu_baseline"] = _cpu_baseline(cfg_id, args.cpu_seconds)
    print(json.dumps(line), flush=True)


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


def _overlap():
    """Clock units (s_memtime) per round of 8 independent MFMAs, of 24
    independent FMAs, and of both interleaved, per wave, at 1, 2 and 4 waves
    per SIMD (one workgroup on one CU).  The FMA-alone time at 4 waves per
    SIMD gives the vector ALU's cost per FMA when saturated.  For 1 and 2
    waves per SIMD the line sets the time of both against full overlap (the
    slower of the two alone) and against serial issue (one wave: the sum of
    the two alone; two waves: the MFMA time plus the saturated cost of both
    waves' FMAs)."""
    import numpy as np
    import torch
    from paper_2508_17445_amd import bench_overlap
    sink = torch.empty(1024, dtype=torch.float32, device="cuda")
    cyc = torch.zeros(16, dtype=torch.int64, device="cuda")
    iters = 4000
    res = {}
    for w in (1, 2, 4):
        for mode, name in ((0, "mfma"), (1, "fma"), (2, "both")):
            bench_overlap(mode, w, iters, sink, cyc)            # warm-up (clocks ramp)
            bench_overlap(mode, w, iters, sink, cyc)
            torch.cuda.synchronize()
            c = cyc[:4 * w].cpu().numpy().astype(np.float64)
            res[f"{name}_w{w}"] = round(float(c.mean()) / iters, 2)
    fma_unit = res["fma_w4"] / (4 * 24)
    line = {"metric": "matrix/vector overlap on one SIMD (clock units per round per wave)", "rounds": iters,
            "per_round": res, "fma_saturated_units": round(fma_unit, 3)}
    for w in (1, 2):
        serial = res["mfma_w1"] + res["fma_w1"] if w == 1 else res["mfma_w2"] + 2 * 24 * fma_unit
        line[f"w{w}"] = {"both": res[f"both_w{w}"], "full_overlap": max(res[f"mfma_w{w}"], res[f"fma_w{w}"]),
                         "serial": round(serial, 2)}
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
    if args.summarize:
        if not args.dir:
            raise SystemExit("--summarize needs --dir")
        {"trace": _summarize_trace, "traffic": _summarize_traffic, "mfma": _summarize_mfma,
         "prefill": _summarize_prefill, "advantage": _summarize_advantage}[args.summarize](args.config, args.dir)
        return
    _ensure_built()
    if args.advantage:
        _advantage(args)
    elif args.prefill:
        _prefill(args)
    elif args.overlap:
        _overlap()
    elif args.segment_loop:
        _segment_loop(args)
    elif args.profile_pass:
        _profile_pass(args.config, args)
    else:
        _decode_line(args)


if __name__ == "__main__":
    main()
