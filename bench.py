#!/usr/bin/env python3
"""Benchmark: hyperbatch data preparation on one MI355X.

A step is one hyperbatch: L hops of block-bucketed sampling for H minibatches
plus the block-bucketed feature gather, on a fresh hyperbatch of targets (step
s uses targets s and mb_base = s * H).  All inputs (graph, features, every
step's targets) are resident in HBM before timing.  Steps are pipelined with
the two-phase API: the sampling of the next --depth hyperbatches runs on
--sample-streams streams (alternating) while one hyperbatch gathers on its own
stream; every step's outputs are complete when the timed region ends.  A
serial reference (prepare after prepare) is reported beside it.

Default workload: R-MAT 2^23 nodes, average degree 30, fp32 features of 256
dims, fanouts [25, 10], 64 minibatches of 1024 targets, 64 KiB blocks.

Printed (one JSON line): value = algorithmic bytes of sampling + gather per
second (GB/s), with sampled edges/s, gathered feature GB/s and the fraction of
the 8 TB/s HBM peak; the roofline of the row-copy kernel (HIP events on the
gather stream, counter-measured HBM traffic from profiles/); the CPU oracle
timed on a bounded sample of the same work.
"""
import argparse
import json
import os
import sys
import time

import numpy as np

HBM_PEAK_GBPS = 8000.0


GATHER_TRAFFIC_FILE = os.path.join("profiles", "k_gather_rows.rmat-2^23.hbm-traffic.md")


def gather_fingerprint(root: str) -> str:
    """sha256 of the row-copy kernels' source, their launch code and the default
    launch shape: the measured HBM traffic stays valid only while these are
    unchanged."""
    import hashlib
    import re
    src = open(os.path.join(root, "paper_2601_01473_amd", "csrc", "pipeline.hip")).read()
    m = re.search(r"template <[^>]*>\n__global__ __launch_bounds__\(kBlock\) void k_gather_rows\(", src)
    if m is None or "// ----------------------------------------------------------------- staged feature tier" not in src[m.start():]:
        return ""
    a = m.start()
    b = src.index("// ----------------------------------------------------------------- staged feature tier", a)
    rt = open(os.path.join(root, "paper_2601_01473_amd", "csrc", "runtime.hpp")).read()
    shape = [ln.strip() for ln in rt.splitlines() if ln.strip().startswith(("int gather_groups", "int gather_unroll",
                                                                             "int gather_nt"))]
    return hashlib.sha256((src[a:b] + "\n".join(shape)).encode()).hexdigest()


def measured_traffic(root: str, workload: str):
    """(GB per launch, algorithmic GB per launch) of the row-copy kernel from the
    committed counter summary, or None when the kernel changed since or the
    summary was taken on another workload."""
    path = os.path.join(root, GATHER_TRAFFIC_FILE)
    if not os.path.exists(path):
        return None
    vals = {}
    for ln in open(path):
        if ln.startswith("- ") and ": " in ln:
            k, v = ln[2:].split(": ", 1)
            vals[k.strip()] = v.strip().strip("`")
    fp = gather_fingerprint(root)
    if not fp or vals.get("kernel_fingerprint") != fp or vals.get("workload") != workload:
        return None
    return float(vals["traffic_GB_per_launch"]), float(vals["algorithmic_GB_per_launch"])


def offset_bytes(w: dict) -> int:
    """Width of the CSR offsets the method needs: 4 bytes for any graph below
    2^31 edges (the library keeps int64 offsets of such graphs as int32 on the
    device), 8 above or when AGNES_WIDE_OFFSETS=1 keeps them 64-bit."""
    if w["offsets"].dtype != np.int64:
        return 4
    wide = os.environ.get("AGNES_WIDE_OFFSETS") == "1"
    return 8 if (wide or len(w["indices"]) >= (1 << 31) - 1) else 4


def algorithmic_bytes(st: dict, offset_bytes: int, row_bytes: int, ids_in_copy: bool = False) -> tuple:
    """Bytes the method must move (exact counts from the batch statistics).

    sampling, per hop: per request the node id, two offsets and the row-pointer
    write; per sampled edge the index read and the column write; per new node
    its id write.  gather: per output row the node-id write and the row write;
    per distinct row one read."""
    bs = 0
    for R, S, U in zip(st["requests"], st["sampled"], st["new_nodes"]):
        bs += R * (4 + 2 * offset_bytes + 4) + 8 * S + 4 * U
    bg = st["rows"] * (4 + row_bytes) + st["distinct_rows"] * row_bytes
    # the row-copy kernel moves the rows; the sampling phase packs the output
    # node ids (k_list_stats), except on the node-range bucket path, where the
    # row copy writes them
    copy = bg if ids_in_copy else bg - st["rows"] * 4
    return bs, bg, copy


def sampling_replayed(mode: int, H: int, B: int, fanouts, num_nodes: int) -> bool:
    """Whether the library replays the sampling kernels from a HIP graph for
    this shape: always (1), never (0), or (2) when its hops can sample at most
    2^20 edges (H x frontier capacity x fanout summed over the hops)."""
    if mode != 2:
        return mode == 1
    cap, edges = B, 0
    for f in fanouts:
        edges += H * cap * f
        cap = min(cap * (1 + f), max(num_nodes, B))
    return edges <= (1 << 20)


def copy_kernel_name(row_bytes: int) -> str:
    """The library's row copy: one wave per row for rows of 1 KiB and more
    (whole 16-byte units), lane groups per row below."""
    if row_bytes % 16 == 0 and row_bytes >= 1024:
        return "k_gather_rows (row copy)"
    return "k_gather (row copy, rows under 1 KiB)"


def block_model_bytes(st: dict, block_bytes: int) -> int:
    """Bytes the paper's I/O model reads: every non-empty topology block row of
    every hop and every non-empty feature block row, one whole block each."""
    return (sum(st["topo_blocks"]) + st["feat_blocks"]) * block_bytes


def ablation(store, cfg, targets_dev, H, reps, ob, rb, torch):
    """The hyperbatch against the same minibatches prepared one at a time (the
    paper's AGNES-No): time, algorithmic bytes and block reads of both modes.
    Minibatch j alone uses mb_base j, so its output equals its part of the
    hyperbatch; block reads of the one-at-a-time mode are summed over j."""
    def run_hb(batch):
        return store.prepare(targets_dev, cfg.fanouts, seed=cfg.seed, mb_base=0, batch=batch)

    def run_no(batches):
        return [store.prepare(targets_dev[j:j + 1], cfg.fanouts, seed=cfg.seed, mb_base=j, batch=batches[j])
                for j in range(H)]

    b = run_hb(None)
    bs = run_no([None] * H)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(reps):
        b = run_hb(b)
    torch.cuda.synchronize()
    t_hb = (time.perf_counter() - t0) / reps
    t0 = time.perf_counter()
    for _ in range(reps):
        bs = run_no(bs)
    torch.cuda.synchronize()
    t_no = (time.perf_counter() - t0) / reps

    def summary(stats, t):
        tot = {"topo_block_reads": 0, "feat_block_reads": 0, "algorithmic_bytes": 0, "rows": 0,
               "distinct_rows": 0, "sampled_edges": 0}
        for st in stats:
            s_, g_, _ = algorithmic_bytes(st, ob, rb)
            tot["topo_block_reads"] += sum(st["topo_blocks"])
            tot["feat_block_reads"] += st["feat_blocks"]
            tot["algorithmic_bytes"] += s_ + g_
            tot["rows"] += st["rows"]
            tot["distinct_rows"] += st["distinct_rows"]
            tot["sampled_edges"] += sum(st["sampled"])
        tot["block_model_bytes"] = (tot["topo_block_reads"] + tot["feat_block_reads"]) * cfg.block_bytes
        tot["ms"] = round(t * 1e3, 4)
        tot["algorithmic_GBps"] = round(tot["algorithmic_bytes"] / t / 1e9, 2)
        return tot

    hb = summary([b.stats()], t_hb)
    no = summary([x.stats() for x in bs], t_no)
    out = {"mode": "ablation: hyperbatch vs one minibatch at a time (synchronous prepare calls)",
           "config": {"workload": cfg.describe(), "hyperbatch": H, "minibatch": cfg.B,
                      "fanouts": list(cfg.fanouts), "block_bytes": cfg.block_bytes},
           "reps": reps, "hyperbatch": hb, "one_at_a_time": no,
           "time_ratio": round(t_no / t_hb, 3),
           "block_read_ratio": round((no["topo_block_reads"] + no["feat_block_reads"]) /
                                     max(1, hb["topo_block_reads"] + hb["feat_block_reads"]), 3),
           "feature_row_read_ratio": round(no["distinct_rows"] / max(1, hb["distinct_rows"]), 3)}
    for x in bs:
        x.close()
    b.close()
    return out


def staged_tier(ag, w, cfg, dev_targets, H, pool_blocks, warmup, steps, ob, rb, torch, cache_rows=None,
                cache_threshold=2):
    """Hyperbatches on a store whose features sit in pinned host memory, with a
    pool of pool_blocks feature blocks in HBM: consecutive fresh hyperbatches
    (synchronous prepare calls), so later ones hit blocks staged earlier."""
    store = ag.Store(w["offsets"], w["indices"], w["features"], cfg.block_bytes, feat_dtype=cfg.feat_dtype,
                     pool_blocks=pool_blocks, cache_rows=cache_rows, cache_threshold=cache_threshold)
    store.set_profiling(True)
    info = store.info()
    b = None
    for s in range(warmup):
        b = store.prepare(dev_targets[s], cfg.fanouts, seed=cfg.seed, mb_base=s * H, batch=b)
    torch.cuda.synchronize()
    acc = dict(ms=0.0, gather_ms=0.0, bytes=0, staged_blocks=0, hit_blocks=0, needed_blocks=0, rounds=0,
               staged_bytes=0, rows_bytes=0, cache_hit_rows=0, admitted_rows=0, distinct_rows=0)
    for s in range(warmup, warmup + steps):
        t0 = time.perf_counter()
        b = store.prepare(dev_targets[s], cfg.fanouts, seed=cfg.seed, mb_base=s * H, batch=b)
        st = b.stats()
        ts = b.tier_stats()
        acc["ms"] += (time.perf_counter() - t0) * 1e3
        bs, bg, _ = algorithmic_bytes(st, ob, rb)
        acc["bytes"] += bs + bg
        acc["gather_ms"] += ts["gather_ms"]
        acc["rows_bytes"] += st["rows"] * rb
        acc["distinct_rows"] += st["distinct_rows"]
        for k in ("staged_blocks", "hit_blocks", "needed_blocks", "rounds", "staged_bytes", "cache_hit_rows",
                  "admitted_rows"):
            acc[k] += ts[k]
        cached = ts["cached_rows"]
    K = steps
    # The same number of further fresh hyperbatches, pipelined: two sample ahead
    # on streams of their own while one stages and gathers on the default stream,
    # so the host's planning and the sampling overlap the previous staging.
    D = 2
    NS = D + 2
    slots = [None] * NS
    slots[0] = b
    s_streams = [torch.cuda.Stream() for _ in range(D)]
    g_stream = torch.cuda.default_stream()
    s0 = warmup + steps
    pipe = dict(bytes=0, staged_bytes=0, hit_blocks=0, needed_blocks=0)

    def begin(s):
        k = s % NS
        slots[k] = store.begin(dev_targets[s], cfg.fanouts, seed=cfg.seed, mb_base=s * H, batch=slots[k],
                               stream=s_streams[s % D])

    def retire(s, record):
        bb = slots[s % NS]
        st = bb.stats()
        ts = bb.tier_stats()
        if not record:
            return
        bs, bg, _ = algorithmic_bytes(st, ob, rb)
        pipe["bytes"] += bs + bg
        for key in ("staged_bytes", "hit_blocks", "needed_blocks"):
            pipe[key] += ts[key]

    def pipeline(first, n, record):
        for s in range(first, first + min(D, n)):
            begin(s)
        for i in range(n):
            s = first + i
            slots[s % NS].finish(stream=g_stream)
            if i >= 2:
                retire(s - 2, record)
            if i + D < n:
                begin(s + D)
        for s in range(first + max(0, n - 2), first + n):
            retire(s, record)

    W2 = NS + 2                      # every slot allocated before timing
    pipeline(s0, W2, False)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    pipeline(s0 + W2, K, True)
    torch.cuda.synchronize()
    pipe_ms = (time.perf_counter() - t0) * 1e3 / K
    out = {"mode": "staged feature tier: features in pinned host memory, HBM pool of feature blocks "
                   "(synchronous prepare calls on fresh hyperbatches; then as many more, pipelined)",
           "config": {"workload": cfg.describe(), "hyperbatch": H, "minibatch": cfg.B,
                      "pool_blocks": pool_blocks, "pool_bytes": pool_blocks * info["rows_per_block"] * rb,
                      "cache_rows": cache_rows or 0, "cache_threshold": cache_threshold if cache_rows else None,
                      "feature_blocks": info["feat_blocks"], "rows_per_block": info["rows_per_block"]},
           "steps": K, "warmup": warmup,
           "ms_per_step": round(acc["ms"] / K, 3),
           "algorithmic_GBps": round(acc["bytes"] / (acc["ms"] * 1e-3) / 1e9, 2),
           "gather_ms": round(acc["gather_ms"] / K, 3),
           "needed_blocks": acc["needed_blocks"] // K, "staged_blocks": acc["staged_blocks"] // K,
           "hit_blocks": acc["hit_blocks"] // K, "rounds": acc["rounds"] / K,
           "hit_rate": round(acc["hit_blocks"] / max(1, acc["needed_blocks"]), 4),
           "staged_GB": round(acc["staged_bytes"] / K / 1e9, 4),
           "staged_GBps_over_gather": round(acc["staged_bytes"] / max(1e-9, acc["gather_ms"] * 1e-3) / 1e9, 2),
           "gathered_rows_GB": round(acc["rows_bytes"] / K / 1e9, 4),
           "distinct_rows": acc["distinct_rows"] // K, "cache_hit_rows": acc["cache_hit_rows"] // K,
           "cache_row_hit_rate": round(acc["cache_hit_rows"] / max(1, acc["distinct_rows"]), 4),
           "admitted_rows": acc["admitted_rows"] // K, "cached_rows_at_end": cached,
           "pipelined": {"ms_per_step": round(pipe_ms, 3),
                         "algorithmic_GBps": round(pipe["bytes"] / K / (pipe_ms * 1e-3) / 1e9, 2),
                         "staged_GB": round(pipe["staged_bytes"] / K / 1e9, 4),
                         "hit_rate": round(pipe["hit_blocks"] / max(1, pipe["needed_blocks"]), 4),
                         "schedule": f"{D} hyperbatches sample ahead on their own streams while one stages "
                                     "and gathers on the default stream"}}
    for bb in slots:
        if bb is not None:
            bb.close()
    store.close()
    return out


def sage_bench(store, cfg, targets_dev, H, steps, torch, hidden):
    """GraphSAGE forward (agnes_sage_forward) over one prepared hyperbatch:
    random bf16 weights, dims [feature dim, hidden, ..., hidden]; the forward is
    timed alone (HIP events on the current stream), its GEMM flops and the
    aggregation's algorithmic bytes are reported."""
    L = len(cfg.fanouts)
    dims = [cfg.dim] + [hidden] * L
    rng = np.random.default_rng(0)
    def bits(x):
        u = np.asarray(x, np.float32).view(np.uint32).astype(np.uint64)
        return ((u + 0x7FFF + ((u >> 16) & 1)) >> 16).astype(np.uint16).view(np.int16)
    Ws = [torch.from_numpy(bits(rng.standard_normal((dims[i + 1], 2 * dims[i])) / np.sqrt(dims[i]))).cuda()
          for i in range(L)]
    bs = [torch.from_numpy((rng.standard_normal(dims[i + 1]) * 0.1).astype(np.float32)).cuda() for i in range(L)]
    b = store.prepare(targets_dev, cfg.fanouts, seed=cfg.seed, mb_base=0)
    out = b.sage_forward(Ws, bs)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(steps):
        b.sage_forward(Ws, bs, out=out)
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / steps
    st = b.stats()
    v = b.view()
    lsz = np.ctypeslib.as_array(v.layer_sizes, shape=(H * (L + 1),)).reshape(H, L + 1)
    esz0 = 4 if cfg.feat_dtype == "float32" else 2
    flops = agg_bytes = 0
    layers = []
    for i in range(L):
        l = L - 1 - i
        M = int(lsz[:, l].sum())
        din, dout = dims[i], dims[i + 1]
        esz = esz0 if i == 0 else 2
        f = 2 * M * 2 * din * dout
        a = (st["sampled"][l] + M) * din * esz + M * 2 * din * 2
        flops += f
        agg_bytes += a
        layers.append({"hop": l, "rows": M, "edges": st["sampled"][l], "gemm_flop": f, "aggregation_bytes": a})
    res = {"mode": "GraphSAGE forward over one prepared hyperbatch (bf16 MFMA GEMMs, float32 mean aggregation)",
           "config": {"workload": cfg.describe(), "hyperbatch": H, "dims": dims},
           "steps": steps, "forward_ms": round(ms, 4), "gemm_GFLOP": round(flops / 1e9, 3),
           "TFLOPs_over_forward": round(flops / (ms * 1e-3) / 1e12, 2),
           "aggregation_algorithmic_GB": round(agg_bytes / 1e9, 4),
           "aggregation_GBps_over_forward": round(agg_bytes / (ms * 1e-3) / 1e9, 1), "layers": layers}
    b.close()
    return res


def host_identity() -> dict:
    """nproc (online CPUs), the CPUs this process may run on, and the CPU model
    name (/proc/cpuinfo, as lscpu reports it)."""
    model = None
    try:
        with open("/proc/cpuinfo") as fh:
            for ln in fh:
                if ln.startswith("model name"):
                    model = ln.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    try:
        affinity = len(os.sched_getaffinity(0))
    except AttributeError:
        affinity = os.cpu_count()
    return {"nproc": os.cpu_count(), "affinity_cpus": affinity, "cpu_model": model}


def _minibatch_bytes(layer_sizes, edge_counts, L, ob, rb):
    """Algorithmic bytes of one minibatch except the distinct-row reads."""
    t = 0
    for l in range(L):
        R = int(layer_sizes[l])
        S = int(edge_counts[l])
        U = int(layer_sizes[l + 1] - layer_sizes[l])
        t += R * (4 + 2 * ob + 4) + 8 * S + 4 * U
    return t + int(layer_sizes[L]) * (4 + rb)


def cpu_baseline(w, cfg, steps_targets, budget_s=20.0):
    """The oracle on the host, on the benchmark's own hyperbatches in order:
    (i) the plain single-threaded oracle, whole minibatches (sampling + gather)
    until about budget_s / 2 seconds of work; (ii) the same oracle on every
    core, whole hyperbatches with their minibatches spread over the threads
    (OMP_NUM_THREADS, else the CPUs this process may use), until about
    budget_s / 2 seconds.  Same metric as the GPU line: algorithmic bytes of
    sampling + gather per second."""
    import oracle
    o = oracle.Oracle(w["offsets64"], w["indices"])
    fb = np.ascontiguousarray(w["features"]).view(np.uint8).reshape(w["num_nodes"], -1)
    ob = offset_bytes(w)
    rb = cfg.row_bytes
    L = len(cfg.fanouts)
    H = w["H"]
    half = budget_s / 2
    # (i) single thread
    done = 0
    total_bytes = 0
    edges = 0
    t0 = time.perf_counter()
    for s, tg in enumerate(steps_targets):
        seen_rows = set()                       # distinct rows are counted per hyperbatch
        for j in range(H):
            mb = o.minibatch(tg[j], cfg.fanouts, cfg.seed, s * H + j)
            feats = oracle.gather(fb, mb.nodes)
            del feats
            total_bytes += _minibatch_bytes(mb.layer_sizes, [len(c) for c in mb.col], L, ob, rb)
            edges += sum(len(c) for c in mb.col)
            new_distinct = [int(v) for v in mb.nodes if int(v) not in seen_rows]
            seen_rows.update(new_distinct)
            total_bytes += len(new_distinct) * rb
            done += 1
            if time.perf_counter() - t0 > half:
                break
        if time.perf_counter() - t0 > half:
            break
    dt1 = time.perf_counter() - t0
    one = dict(value=total_bytes / dt1 / 1e9, unit="GB/s", cores=1, sampled_edges_per_s=edges / dt1,
               sample=f"{done} minibatches ({H} per hyperbatch), sampling + gather, {dt1:.1f} s")
    # (ii) all cores: whole hyperbatches
    threads = int(os.environ.get("OMP_NUM_THREADS", "0") or 0) or host_identity()["affinity_cpus"]
    run = oracle.ThreadedRunner(w["offsets64"], w["indices"], w["features"])
    hb = 0
    total_bytes = 0
    edges = 0
    used = threads
    t0 = time.perf_counter()
    for s, tg in enumerate(steps_targets):
        r = run.run(tg, cfg.fanouts, cfg.seed, s * H, threads=threads)
        used = r["threads"]
        for j in range(H):
            total_bytes += _minibatch_bytes(r["layer_sizes"][j], r["edge_counts"][j], L, ob, rb)
        total_bytes += r["distinct"] * rb
        edges += int(r["edge_counts"].sum())
        hb += 1
        if time.perf_counter() - t0 > half:
            break
    dt2 = time.perf_counter() - t0
    out = dict(value=total_bytes / dt2 / 1e9, unit="GB/s", cores=used, kind="oracle",
               sample=f"{hb} whole hyperbatches of {H} minibatches on {used} threads, sampling + gather, "
                      f"{dt2:.1f} s",
               sampled_edges_per_s=edges / dt2, single_thread=one)
    out.update(host_identity())
    return out


def copy_calibration(torch, nbytes=4 << 30, reps=5):
    """A plain copy of known size: reads nbytes and writes nbytes per launch."""
    x = torch.empty(nbytes // 4, dtype=torch.int32, device="cuda").fill_(1)
    y = torch.empty_like(x)
    y.copy_(x)
    torch.cuda.synchronize()
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record()
    for _ in range(reps):
        y.copy_(x)
    b.record()
    torch.cuda.synchronize()
    ms = a.elapsed_time(b) / reps
    print(json.dumps({"copy_bytes_read": nbytes, "copy_bytes_written": nbytes, "ms": round(ms, 4),
                      "GBps_read_plus_write": round(2 * nbytes / (ms * 1e-3) / 1e9, 1)}), flush=True)


class Pipeline:
    """The schedule the benchmark times.  Step s is the hyperbatch of
    targets[s] with mb_base s * H; the sampling of steps s+1 .. s+depth runs
    on `sample_streams` streams (alternating, default priority) while step s
    gathers on the default stream (or a stream of its own).  Each step's batch
    lives in one of NSLOT slots and is reused depth + lag steps later; when a
    step is retired (its outputs complete), on_retire(s, batch, record) is
    called before its slot is reused.
    ahead: gather s is queued (behind gather s-1) as soon as step s's sizes
      are known; only then is step s-2 retired and step s+depth begun in its
      slot, so the gather stream never drains while the host enqueues sampling.
    sample-first: step s-1 is retired, step s+depth begun, then gather s queued.
    gather-first: gather s queued, step s-1 retired, step s+depth begun."""

    def __init__(self, store, cfg, H, targets, depth=3, sample_streams=3, gather_stream="default",
                 schedule="ahead", on_retire=None):
        import torch
        self.store, self.cfg, self.H, self.targets = store, cfg, H, targets
        self.D = max(1, depth)
        self.schedule = schedule
        # "ahead" keeps two finished steps unread, so it holds two more slots
        # than the hyperbatches in flight
        self.lag = 2 if schedule == "ahead" else 1
        self.NSLOT = self.D + self.lag
        self.slots = [None] * self.NSLOT
        self.s_streams = [torch.cuda.Stream() for _ in range(max(1, sample_streams))]
        self.g_stream = torch.cuda.default_stream() if gather_stream == "default" else torch.cuda.Stream()
        self.on_retire = on_retire or (lambda s, b, record: b.wait())

    def begin(self, s):
        k = s % self.NSLOT
        self.slots[k] = self.store.begin(self.targets[s], self.cfg.fanouts, seed=self.cfg.seed, mb_base=s * self.H,
                                         batch=self.slots[k], stream=self.s_streams[s % len(self.s_streams)])

    def retire(self, s, record):
        self.on_retire(s, self.slots[s % self.NSLOT], record)

    def run(self, first, n, record):
        """Steps first .. first+n-1 with the sampling of steps s+1 .. s+depth in
        flight while step s gathers; every step is retired before returning."""
        D, lag = self.D, self.lag
        for s in range(first, first + min(D, n)):
            self.begin(s)
        for i in range(n):
            s = first + i
            if self.schedule != "sample-first":
                self.slots[s % self.NSLOT].finish(stream=self.g_stream)   # waits for step s's sizes only
            if i >= lag:
                self.retire(s - lag, record)                              # its slot is free for step s+D
            if i + D < n:
                self.begin(s + D)
            if self.schedule == "sample-first":
                self.slots[s % self.NSLOT].finish(stream=self.g_stream)
        for s in range(first + max(0, n - lag), first + n):
            self.retire(s, record)

    def close(self):
        for b in self.slots:
            if b is not None:
                b.close()


def gather_calibration(ag, w, cfg, torch, reps=5):
    """The row-copy kernel on a list whose rows are all distinct: one
    hyperbatch of 2^21 distinct targets and no sampling (fanout 0), so every
    launch reads and writes exactly rows x row_bytes (plus a 12-byte list
    entry read per row; the output node ids are packed by the sampling
    phase)."""
    n = min(cfg.num_nodes, 1 << 21)
    import synth
    tg = synth.targets(cfg.num_nodes, n, cfg.data_seed + 11).reshape(1, n)
    store = ag.Store(w["offsets"], w["indices"], w["features"], cfg.block_bytes, feat_dtype=cfg.feat_dtype)
    store.set_profiling(True)
    b = None
    ms = []
    for _ in range(reps):
        b = store.prepare(tg, [0], seed=cfg.seed, batch=b)
        st = b.stats()
        ms.append(st["copy_ms"])
    assert st["rows"] == n and st["distinct_rows"] == n
    print(json.dumps({"mode": "row copy over all-distinct rows (fanout 0)", "rows": n, "row_bytes": cfg.row_bytes,
                      "bytes_read": n * cfg.row_bytes, "bytes_written": n * cfg.row_bytes,
                      "copy_ms": [round(x, 4) for x in ms]}), flush=True)
    b.close()
    store.close()


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100,
                    help="timed steps; the pipeline fills and drains inside the timed region (about 0.6 ms at "
                         "the 2^23-node workload), so more steps come closer to a long run's steady state")
    ap.add_argument("--warmup", type=int, default=5,
                    help="untimed steps before the timed ones; raised to depth + 2 so that every batch slot "
                         "is allocated before timing (the JSON line reports the number run)")
    ap.add_argument("--config", default="c3")
    ap.add_argument("--H", type=int, default=None, help="minibatches per hyperbatch (default: the config's)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-budget", type=float, default=20.0)
    ap.add_argument("--depth", type=int, default=3, help="hyperbatches sampled ahead of the one gathering")
    ap.add_argument("--sample-streams", type=int, default=3,
                    help="streams the sampling of consecutive hyperbatches alternates between")
    ap.add_argument("--gather-stream", choices=["default", "own"], default="default",
                    help="gather on the default stream (default: the process's other hardware queues, "
                         "4 per process on this platform, then serve the sampling streams) or on its own")
    ap.add_argument("--schedule", choices=["ahead", "sample-first", "gather-first"], default="ahead",
                    help="ahead: each gather is queued behind the running one and a step's statistics are "
                         "read two steps later, so the host never waits for a gather before queuing work; "
                         "sample-first: the next sampling is enqueued before each gather; gather-first: each "
                         "gather is queued before the previous one is waited for")
    ap.add_argument("--gather-groups", type=int, default=None, help="row-copy kernel workgroups")
    ap.add_argument("--gather-unroll", type=int, default=None,
                    help="rows in flight per lane group, 4, 8 or 16 (default: 16 for rows of 1-2 KiB, else 4)")
    ap.add_argument("--gather-nt", type=int, default=None, help="1 = non-temporal row stores, 0 = ordinary")
    ap.add_argument("--gather-chunks", type=int, default=None, help="launches the row copy is split into")
    ap.add_argument("--sampling-groups", type=int, default=None,
                    help="most workgroups of each sampling-phase kernel that loops over its work")
    ap.add_argument("--join-path", type=int, choices=[0, 1], default=None,
                    help="0: radix sort and merge-path join (default); 1: node-range buckets")
    ap.add_argument("--sampling-graph", type=int, choices=[0, 1, 2], default=2,
                    help="1: replay the sampling kernels from a captured HIP graph; 0: launch them one by one; "
                         "2: replay for shapes of at most 2^20 sampled edges (the library's default)")
    ap.add_argument("--ablation", action="store_true",
                    help="instead of the benchmark line, compare the hyperbatch with its minibatches "
                         "prepared one at a time (time, bytes, block reads)")
    ap.add_argument("--staged", type=int, default=None, metavar="POOL_BLOCKS",
                    help="instead of the benchmark line, run the staged feature tier (features in pinned "
                         "host memory) with a pool of POOL_BLOCKS feature blocks in HBM")
    ap.add_argument("--sage", type=int, default=None, metavar="HIDDEN",
                    help="instead of the benchmark line, time the GraphSAGE forward over one prepared "
                         "hyperbatch with hidden width HIDDEN")
    ap.add_argument("--cache-rows", type=int, default=None,
                    help="with --staged: a feature cache of this many rows in HBM")
    ap.add_argument("--cache-threshold", type=int, default=2,
                    help="with --cache-rows: access count at which a row enters the cache")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="time a plain 4 GiB device-to-device copy (reference for the HBM counters)")
    ap.add_argument("--hbm-ceiling", action="store_true",
                    help="run the HBM ceiling probe (plain streaming read, write and copy kernels) and exit")
    ap.add_argument("--gather-calibration", action="store_true",
                    help="run the row-copy kernel over 2^21 all-distinct rows (reference for its HBM counters)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only; --gpus {args.gpus} is not supported "
              f"(the path shards by minibatch with no communication; see the design notes)",
              file=sys.stderr)
        sys.exit(2)

    root = os.path.dirname(os.path.abspath(__file__))
    sys.path.insert(0, root)
    if args.hbm_ceiling:
        # a child process, started before this one touches the GPU
        import subprocess
        probe = os.path.join(root, "paper_2601_01473_amd", "hbm_ceiling")
        if not os.path.exists(probe):
            sys.exit("the HBM ceiling probe is not built (python -c 'import __graft_entry__ as g; g.build()')")
        sys.exit(subprocess.call([probe]))
    import torch
    if args.copy_calibration:
        copy_calibration(torch)
        return
    import synth
    import paper_2601_01473_amd as ag

    cfg = synth.CONFIGS[args.config]
    t0 = time.time()
    w = synth.workload(cfg, H=args.H)
    H, B = w["H"], w["B"]
    print(f"# inputs ready in {time.time() - t0:.1f}s (E={len(w['indices'])})", file=sys.stderr, flush=True)
    args.warmup = max(args.depth + 2, args.warmup)   # every batch slot is allocated before timing
    # the staged tier's bench runs its steps twice (synchronous, then pipelined
    # after a warm-up of its own)
    nsteps = args.warmup + args.steps * (2 if args.staged is not None else 1) + (8 if args.staged is not None else 0)
    # distinct targets per step: consecutive slices of one permutation of the nodes
    perm = synth.targets(cfg.num_nodes, min(cfg.num_nodes, nsteps * H * B), cfg.data_seed + 7)
    step_targets = []
    for s in range(nsteps):
        a = (s * H * B) % (len(perm) - H * B + 1)
        step_targets.append(perm[a:a + H * B].reshape(H, B))
    dev_targets = [torch.from_numpy(np.ascontiguousarray(t)).cuda() for t in step_targets]

    if args.staged is not None:
        print(json.dumps(staged_tier(ag, w, cfg, dev_targets, H, args.staged, args.warmup, args.steps,
                                     8 if w["offsets"].dtype == np.int64 else 4, cfg.row_bytes, torch,
                                     args.cache_rows, args.cache_threshold)), flush=True)
        return
    if args.gather_calibration:
        gather_calibration(ag, w, cfg, torch)
        return
    store = ag.Store(w["offsets"], w["indices"], w["features"], cfg.block_bytes, feat_dtype=cfg.feat_dtype)
    if args.sage is not None:
        print(json.dumps(sage_bench(store, cfg, dev_targets[0], H, max(1, args.steps), torch, args.sage)), flush=True)
        store.close()
        return
    if args.ablation:
        tg = torch.from_numpy(np.ascontiguousarray(step_targets[0])).cuda()
        ob_ = offset_bytes(w)
        print(json.dumps(ablation(store, cfg, tg, H, max(1, min(args.steps, 5)), ob_, cfg.row_bytes, torch)),
              flush=True)
        store.close()
        return
    store.set_profiling(True)
    store.set_gather_shape(args.gather_groups, args.gather_unroll,
                           None if args.gather_nt is None else bool(args.gather_nt), args.gather_chunks)
    store.set_sampling_graph({0: False, 1: True, 2: "auto"}[args.sampling_graph])
    if args.sampling_groups is not None:
        store.set_sampling_groups(args.sampling_groups)
    if args.join_path is not None:
        store.set_join_path(bool(args.join_path))
    stream = torch.cuda.current_stream()
    ob = offset_bytes(w)
    rb = cfg.row_bytes

    acc = dict(bytes=0, sample=0, gather=0, copy_bytes=0, edges=0, rows=0, distinct=0, block_model=0, sample_ms=0.0, gather_ms=0.0,
               copy_ms=0.0, steps=0)

    def account(batch):
        st = batch.stats()                      # waits for the batch
        bs, bg, bc = algorithmic_bytes(st, ob, rb, ids_in_copy=args.join_path == 1)
        acc["sample"] += bs
        acc["gather"] += bg
        acc["copy_bytes"] += bc
        acc["bytes"] += bs + bg
        acc["edges"] += sum(st["sampled"])
        acc["rows"] += st["rows"]
        acc["distinct"] += st["distinct_rows"]
        acc["block_model"] += block_model_bytes(st, cfg.block_bytes)
        acc["sample_ms"] += st["sample_ms"]
        acc["gather_ms"] += st["gather_ms"]
        acc["copy_ms"] += st["copy_ms"]
        acc["steps"] += 1

    pipe = Pipeline(store, cfg, H, dev_targets, depth=args.depth, sample_streams=args.sample_streams,
                    gather_stream=args.gather_stream, schedule=args.schedule,
                    on_retire=lambda s, b, record: account(b) if record else b.wait())
    D, NSLOT, slots = pipe.D, pipe.NSLOT, pipe.slots
    s_streams = pipe.s_streams

    def pipeline(first, n, record):
        pipe.run(first, n, record)

    # warm-up: every slot allocated at the largest shape seen so far
    pipeline(0, args.warmup, record=False)
    torch.cuda.synchronize()
    print("# warm-up done", file=sys.stderr, flush=True)

    K = args.steps
    s0 = args.warmup
    torch.cuda.synchronize()
    t_start = time.perf_counter()
    pipeline(s0, K, record=True)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t_start
    assert acc["steps"] == K

    # the same steps with the targets handed over in host memory: each begin
    # copies them to pinned memory and uploads them on its sampling stream
    # (reported beside the value, which is measured with inputs in HBM)
    saved = dict(acc)
    for key in acc:
        acc[key] = 0 if isinstance(acc[key], int) else 0.0
    pipe.targets = step_targets
    torch.cuda.synchronize()
    t_h = time.perf_counter()
    pipeline(s0, K, record=True)
    torch.cuda.synchronize()
    host_elapsed = time.perf_counter() - t_h
    host_bytes = acc["bytes"]
    acc.update(saved)
    pipe.targets = dev_targets

    # reference: the same work one hyperbatch at a time (synchronous prepare)
    nser = min(K, 5)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    for k in range(nser):
        s = s0 + k
        slots[0] = store.prepare(dev_targets[s], cfg.fanouts, seed=cfg.seed, mb_base=s * H, batch=slots[0],
                                 stream=s_streams[0])
    torch.cuda.synchronize()
    serial_ms = (time.perf_counter() - t1) / nser * 1e3

    traffic = measured_traffic(root, f"{cfg.describe()}|H={H}")
    tot_bytes, tot_sample, tot_gather = acc["bytes"], acc["sample"], acc["gather"]
    tot_copy_bytes, edges, rows = acc["copy_bytes"], acc["edges"], acc["rows"]
    sample_ms, gather_ms, copy_ms = acc["sample_ms"], acc["gather_ms"], acc["copy_ms"]
    value = tot_bytes / elapsed / 1e9
    copy_avg_ms = copy_ms / K
    replayed = sampling_replayed(args.sampling_graph, H, B, cfg.fanouts, cfg.num_nodes)
    graph_mode = "replayed from a HIP graph" if replayed else "launched one by one"
    achieved = (tot_copy_bytes / K) / (copy_avg_ms * 1e-3) / 1e9
    result = {
        "metric": "sampled edges/s + gathered feature GB/s per hyperbatch (% of HBM peak)",
        "value": round(value, 2),
        "unit": "GB/s (algorithmic bytes of sampling + gather)",
        "n_gpus": 1,
        "steps": K,
        "warmup": args.warmup,
        "ms_per_step": round(elapsed / K * 1e3, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "int32",
        "data": "synthetic (seeded R-MAT graph, N(0,1) features, uniform distinct targets)",
        "config": {"workload": cfg.describe(), "nodes": cfg.num_nodes, "edges": int(len(w["indices"])),
                   "hyperbatch": H, "minibatch": B, "fanouts": list(cfg.fanouts),
                   "block_bytes": cfg.block_bytes, "feature_dtype": cfg.feat_dtype, "dim": cfg.dim,
                   "parallelism": "single GPU"},
        "hbm_frac": round(value / HBM_PEAK_GBPS, 4),
        "sampled_edges_per_s": round(edges / elapsed, 1),
        "gathered_feature_GBps": round(rows * rb / elapsed / 1e9, 2),
        "gather_phase_GBps": round(rows * rb / (gather_ms * 1e-3) / 1e9, 2) if gather_ms > 0 else None,
        "phase_ms": {"sample": round(sample_ms / K, 4), "gather": round(gather_ms / K, 4),
                     "copy_kernel": round(copy_avg_ms, 4)},
        "mode": f"pipelined ({args.schedule}): {NSLOT} batch slots; "
                f"hyperbatches t+1..t+{D} sample while t gathers"
                f"; {len(s_streams)} sampling stream(s); gather on the {args.gather_stream} stream"
                f"; sampling kernels {graph_mode}",
        "serial_ms_per_step": round(serial_ms, 4),
        "host_targets": {"ms_per_step": round(host_elapsed / K * 1e3, 4),
                         "GBps": round(host_bytes / host_elapsed / 1e9, 2),
                         "note": "the same steps with targets in host memory, uploaded by every begin "
                                 "(H*B*4 bytes over PCIe inside the step)"},
        "per_step": {"algorithmic_bytes": tot_bytes // K, "sample_bytes": tot_sample // K,
                     "gather_bytes": tot_gather // K, "rows": rows // K,
                     "distinct_rows": acc["distinct"] // K, "sampled_edges": edges // K,
                     "block_model_bytes": acc["block_model"] // K},
        "roofline": {"kernel": copy_kernel_name(cfg.row_bytes), "bound": "hbm", "achieved": round(achieved, 1),
                     "peak": HBM_PEAK_GBPS, "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBPS, 4),
                     "traffic": traffic[0] if traffic else None,
                     "traffic_unit": "GB per launch, HBM (FETCH_SIZE x2.0 + WRITE_SIZE x1.0, copy-calibrated)",
                     "traffic_algorithmic": traffic[1] if traffic else None},
    }
    if not args.no_cpu_baseline:
        result["cpu_baseline"] = cpu_baseline(w, cfg, step_targets[args.warmup:], args.cpu_budget)
    print(json.dumps(result), flush=True)
    for b in slots:
        b.close()
    store.close()


if __name__ == "__main__":
    main()
