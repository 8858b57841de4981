#!/usr/bin/env python3
"""Throughput of batched dynamic updates and search of a GrAND index on one
MI355X.

Workload (default): 1,000,000 x 128 uint8 vectors from a 256-component
Gaussian mixture (centres U[0,255], sigma 20, rounded and clipped), L2,
Vamana R=64, L=128, alpha=1.2.  The base index is built by 100 batched
inserts of 10,000, then refreshed once: each base batch is deleted and
re-inserted with the same ids and vectors, so every list is rebuilt against
the complete base set (the batched counterpart of a static build's second
pass; untimed).  A step is one round of the streaming workload: +10,000
inserts (smallest free ids), -10,000 uniformly random deletes, 10,000
queries (k=10, beam 64).  Inputs of every round are staged in device memory
before timing.  One JSON line is printed:
  value       = updates/s (inserts + deletes over the time of the insert
                and delete calls), with search QPS and recall@10 alongside;
  roofline    = achieved algorithmic bandwidth of the dominant kernel (the
                one with the largest share of GPU time: k_search, whose
                insert, delete and query launches are summed), from HIP
                events on the library's stream around each phase.  A search
                is charged for the distinct ids whose distance it needs,
                counted exactly by an untimed rerun of the same rounds on the
                same state with an exact visited set; the fraction over every
                evaluation the timed kernel made is given beside it.  The
                other phases' figures are listed in roofline_other_phases;
  cpu_baseline= the CPU oracle on the host cores allotted to the job, on the
                state the timed rounds start from, for the first three timed
                rounds.
Other workloads (--workload) are the fp32 sliding window, the CAGRA
inner-product set, the 960-d set and the tiny set; their lines carry their
own metric and data labels.
"""
import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HEADLINE_METRIC = "updates/sec and search QPS at recall@10≥0.95, 1M×128, 1 MI355X"
HBM_PEAK_GBS = 8000.0

# what each synthetic workload stands in for (no dataset is available here)
DATA_LABEL = {
    "sift1m_u8": "synthetic (seeded 256-component uint8 mixture; stands in for the paper's SIFT-like 128-d set)",
    "deep1m_window": "synthetic (seeded 512-component mixture, L2-normalised, drifting weights; stands in for the "
                     "paper's 96-d Euclidean set under the sliding-window pattern)",
    "glove1m_cagra": "synthetic (seeded 1,000-component Student-t(3) mixture, unit-normalised; stands in for the "
                     "paper's 100-d angular set)",
    "gist500k": "synthetic (seeded 128-component mixture, per-dimension scales, clipped at 0; a 960-d stress case)",
    "tiny": "synthetic (seeded N(0,1), 10,000 x 32)",
    "ip768_mips": "synthetic (seeded 128-component mixture with varying norms, clipped at 40; stands in for the "
                  "paper's 768-d inner-product text-embedding sets)",
}
SHAPE = {"sift1m_u8": "1M×128 uint8", "deep1m_window": "1M×96 fp32 sliding window",
         "glove1m_cagra": "1M×100 fp32 IP, CAGRA degree 64", "gist500k": "500K×960 fp32", "tiny": "10K×32 fp32",
         "ip768_mips": "500K×768 fp32 inner product via L2 augmentation"}


def metric_of(workload, recall_min):
    if workload == "sift1m_u8":
        return HEADLINE_METRIC
    r = "n/a" if recall_min is None else f"{recall_min:.3f}"
    return f"updates/sec and search QPS at recall@10 (min {r}), {SHAPE.get(workload, workload)}, 1 MI355X"


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def parse():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--workload", default="sift1m_u8")
    ap.add_argument("--base", type=int, default=0, help="override the base size (quick runs)")
    ap.add_argument("--build-batch", type=int, default=0, help="override the batch size of the untimed base build")
    ap.add_argument("--build-frac", type=float, default=-1.0, help="override the growth fraction of the base build")
    ap.add_argument("--build-min", type=int, default=0, help="override the smallest base build batch")
    ap.add_argument("--refresh-passes", type=int, default=-1,
                    help="after the base build, delete and re-insert every base batch this many times (untimed; "
                         "default: the workload's, 1 for most, 3 for the 960-d and 768-d sets, 0 for CAGRA, whose "
                         "delete repair the refresh would only degrade)")
    ap.add_argument("--cagra-seed", choices=["construct", "bootstrap", "full"], default="construct",
                    help="CAGRA base build: the first base batch by the CAGRA graph construction (construct) or by "
                         "the empty-index bootstrap of a batch insert (bootstrap), then batched inserts; or the "
                         "whole base by one construction (full)")
    ap.add_argument("--cagra-knn", type=int, default=128, help="construction: k-NN degree")
    ap.add_argument("--cagra-rounds", type=int, default=8, help="construction: NN-Descent rounds")
    ap.add_argument("--cagra-sample", type=int, default=16, help="construction: NN-Descent sample size")
    ap.add_argument("--prune-rule", choices=["alpha_on_sq", "alpha_on_l2"], default=None,
                    help="override the alpha test of GrANDRobustPrune")
    ap.add_argument("--rev-mode", choices=["full", "batch"], default="batch")
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-recall", action="store_true")
    ap.add_argument("--no-concurrent", action="store_true",
                    help="skip the replay of the timed rounds with each round's queries on a second stream, "
                         "overlapping its updates (overall throughput)")
    ap.add_argument("--pattern", default=None,
                    help="run one streaming pattern of the workload generator (sliding_window, interleaved, "
                         "expiration, clustered, insert_heavy) over base_n points of the workload's "
                         "distribution instead of the rounds, and print its line")
    ap.add_argument("--reverse-microbench", action="store_true",
                    help="after the base build, time in-neighbour detection for one delete batch by a per-id "
                         "linear scan, the batch-rows reverse build and the full reverse graph, and print that")
    ap.add_argument("--copy-probe", action="store_true",
                    help="only run a 1 GiB device-to-device copy 5 times (calibrates HBM byte counters)")
    return ap.parse_args()


def copy_probe():
    """A plain copy of known size: 1 GiB read + 1 GiB written per launch."""
    import torch
    n = 1 << 30
    x = torch.ones(n, dtype=torch.uint8, device="cuda:0")
    y = torch.empty_like(x)
    for _ in range(5):
        torch.mul(x, 1, out=y)  # an elementwise shader kernel (a D2D memcpy may run on a DMA engine)
    torch.cuda.synchronize()
    print(json.dumps({"copy_probe_bytes_read": n, "copy_probe_bytes_written": n, "launches": 5}), flush=True)


# ------------------------------------------------------------------ ground truth
class Mirror:
    """Device copy of the pool and active map that follows the operation
    stream, for exact ground truth (measurement only; not the index)."""

    def __init__(self, torch, cfg, dev):
        self.t = torch
        dt = torch.uint8 if cfg.dtype == "u8" else torch.float32
        self.pool = torch.zeros((cfg.capacity, cfg.dim), dtype=dt, device=dev)
        self.active = torch.zeros(cfg.capacity, dtype=torch.bool, device=dev)
        self.metric = cfg.metric
        self.u8 = cfg.dtype == "u8"

    def insert(self, ids, vecs):
        self.pool[ids.long()] = vecs
        self.active[ids.long()] = True

    def delete(self, ids):
        self.active[ids.long()] = False

    def knn(self, q, k, chunk=1024):
        t = self.t
        act = t.nonzero(self.active).squeeze(1)
        # uint8 L2 in fp32 is exact (integer partial sums < 2^24); fp32
        # data in fp64
        ct = t.float32 if self.u8 else t.float64
        X = self.pool[act].to(ct)
        xn = (X * X).sum(1)
        out = []
        for s in range(0, q.shape[0], chunk):
            Q = q[s:s + chunk].to(ct)
            if self.metric == "l2":
                d = (Q * Q).sum(1, keepdim=True) + xn[None, :] - 2.0 * (Q @ X.T)
            else:
                d = -(Q @ X.T)
            idx = t.topk(d, k, dim=1, largest=False).indices
            out.append(act[idx])
        return t.cat(out).to(t.int64)


# ------------------------------------------------------------------ algorithmic bytes
def algorithmic_bytes(st, phase, cfg, stride, distinct=None):
    """Bytes each phase must move over the timed region, from the kernels'
    own work counters (a vector row is `stride` bytes, an adjacency row 4R):
      search : per query one query row; per expanded node one adjacency row;
               per distance the search needs one vector row (the distinct
               ids of a counting rerun when given, else every evaluation the
               kernel made); outputs;
      prune_fwd: per new point its row and its |V_i| candidate rows, V_i
               (8 B an entry), its list (4R) and its records (12 B);
      group  : every record read (12 B) and written grouped (8 B); per
               dirty node its offset and its dirty-list entry;
      reverse: one read of every adjacency row and of the active map, one
               write of the offsets and of the sources (per launch:
               capacity x (4R + 1) + 4 (capacity + 1) + 4 nnz);
      rebuild: per dirty node its degree, adjacency row read and written,
               8 B per scratch record; per pruning rebuild the |C| candidate
               rows and u's row (pairwise distances reuse those rows);
      repair : per deleted node its C_i rows and one row per repaired
               neighbour; 12 B per record written."""
    R = cfg.R
    if phase.startswith("search_"):
        w = phase.split("_")[1]
        hops = st[f"hops_{w}"]
        evals = st[f"evals_{w}"] if distinct is None else distinct[w]
        n = {"insert": st["inserted"], "delete": st["deleted"], "query": st["queried"]}[w]
        outb = {"insert": 8 * hops, "delete": 4 * n * cfg.k_repair, "query": 8 * n * 10}[w]
        return n * stride + hops * 4 * R + evals * stride + outb
    if phase == "prune_fwd":
        n = st["inserted"]
        fwd_records = st["records"] - st["repair_records"]
        return (st["hops_insert"] + n) * stride + 8 * st["hops_insert"] + n * 4 * R + 12 * fwd_records
    if phase == "group":
        return 20 * st["records"] + 8 * st["dirty"]
    if phase == "reverse":
        launches = st["phase_calls"]["reverse"]
        return launches * (cfg.capacity * (4 * R + 1) + 4 * (cfg.capacity + 1)) + 4 * st["rev_edges"]
    if phase == "rebuild":
        return st["dirty"] * (8 * R + 4) + 8 * st["rebuild_records"] + st["rebuild_rows"] * stride
    if phase == "repair":
        return st["repair_rows"] * stride + 12 * st["repair_records"]
    return None


def profiled_traffic(phase):
    """HBM bytes per launch of `phase` (read + write), from the rocprofv3
    counter summary in profiles/, or None when the kernel sources changed
    since the counters were taken (the summary records their hash)."""
    import hashlib
    import glob
    path = os.path.join(ROOT, "profiles", "traffic_sift1m_u8.md")
    if not os.path.exists(path):
        return None
    h = hashlib.sha256()
    for f in sorted(glob.glob(os.path.join(ROOT, "paper_2608_21163_amd", "csrc", "*"))) + \
            [os.path.join(ROOT, "include", "grand.h")]:
        h.update(os.path.basename(f).encode())
        with open(f, "rb") as fh:
            h.update(fh.read())
    want, val = None, None
    with open(path) as fh:
        for line in fh:
            t = line.split()
            if len(t) == 2 and t[0] == "sources-sha256":
                want = t[1]
            elif len(t) == 3 and t[0] == "traffic" and t[1] == phase:
                val = float(t[2])
    if want != h.hexdigest()[:16]:
        return None
    return val


# ------------------------------------------------------------------ cpu baseline
def host_cpu():
    """CPU model and core counts of this host (lscpu-style, from /proc)."""
    model = None
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    return {"model": model, "host_cores": os.cpu_count(), "affinity_cores": len(os.sched_getaffinity(0))}


def oracle_threads():
    """Threads for the oracle: the CPU share the job is given (the
    OMP_NUM_THREADS the environment sets for one GPU's job), else every core
    this process may run on."""
    share = os.environ.get("OMP_NUM_THREADS")
    aff = len(os.sched_getaffinity(0))
    return min(int(share), aff) if share and share.isdigit() and int(share) > 0 else aff


# timed rounds the CPU baseline replays (about 10-30 s of oracle work at 1M points)
CPU_ROUNDS = 3


def cpu_baseline(cfg, spec, snap, host_round, n_rounds, threads, max_seconds=60.0):
    """The oracle (plain C, OpenMP over batch items) on the state the timed
    rounds start from (imported), timed on the first timed rounds' own
    batches: the same workload at the same scale, on `threads` host cores."""
    from oracle.oracle import Oracle
    o = Oracle(cfg, threads=threads)
    t0 = time.perf_counter()
    o.import_graph(snap["vecs"], snap["adj"], snap["deg"], snap["active"], snap["medoid"])
    log(f"cpu baseline: state imported in {time.perf_counter() - t0:.1f} s; oracle on {threads} threads ...")
    t_upd = t_q = 0.0
    n_upd = n_q = 0
    done = {"inserts": 0, "deletes": 0, "searches": 0}
    for kind, ids, vecs in host_round:
        t0 = time.perf_counter()
        if kind == "insert":
            o.insert(ids, vecs)
            t_upd += time.perf_counter() - t0
            n_upd += len(ids)
        elif kind == "delete":
            o.delete(ids)
            t_upd += time.perf_counter() - t0
            n_upd += len(ids)
        else:
            o.search(vecs, spec.k, spec.beam)
            t_q += time.perf_counter() - t0
            n_q += len(vecs)
        plural = {"insert": "inserts", "delete": "deletes", "search": "searches"}[kind]
        done[plural] += len(ids) if ids is not None else len(vecs)
        log(f"cpu baseline: {kind} done, {time.perf_counter() - t0:.1f} s")
    out = {"value": round(n_upd / t_upd, 1) if t_upd > 0 else None, "unit": "updates/s", "cores": threads,
           "kind": "oracle", "search_qps": round(n_q / t_q, 1) if t_q > 0 else None,
           "sample": (f"oracle on the {int(snap['active'].sum()):,}-point index the timed rounds start from "
                      f"(imported from the GPU), timed on the first {n_rounds} timed round"
                      f"{'s' if n_rounds != 1 else ''}: " + ", ".join(f"{v:,} {k}" for k, v in done.items() if v)),
           "cpu": host_cpu()}
    return out


# ------------------------------------------------------------------ streaming patterns
def run_pattern(args):
    """One streaming pattern (Section 5.2) over `base_n` points of the
    workload's distribution, in batches of 1% of them: the starting index is
    built untimed (batched inserts, then one refresh pass as for the
    rounds), every batch of the stream is staged on the device with exact
    ground truth, and the whole stream is timed call by call."""
    import numpy as np
    import torch

    from paper_2608_21163_amd import GrandIndex
    from workloads import PatternStream, make_workload
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    stream = torch.cuda.current_stream()
    st_over = {"base_n": args.base} if args.base else None
    w = make_workload(args.workload, seed=args.seed, stream=st_over)
    cfg, spec = w.cfg, w.spec
    ps = PatternStream(w, args.pattern, spec.base_n, n_query=spec.n_query, seed=args.seed, batch_frac=0.01,
                       build_batch=spec.build_batch)
    g = GrandIndex.from_config(cfg, max_batch=max(spec.build_batch, ps.batch), stream=stream.cuda_stream)
    mirror = Mirror(torch, cfg, dev)
    t0 = time.perf_counter()
    base = []
    for op in ps.base_ops():
        ids = torch.from_numpy(op.ids.astype(np.int32)).to(dev)
        vecs = torch.from_numpy(op.vecs).to(dev)
        g.insert(ids, vecs)
        mirror.insert(ids, vecs)
        base.append((ids, vecs))
    for ids, vecs in base:
        g.delete(ids)
        g.insert(ids, vecs)
    del base
    torch.cuda.synchronize()
    build_s = time.perf_counter() - t0
    log(f"pattern {args.pattern}: base of {int(mirror.active.sum())} points built in {build_s:.1f} s")
    staged = []
    for op in ps.ops():
        if op.kind == "insert":
            ids, vecs = torch.from_numpy(op.ids.astype(np.int32)).to(dev), torch.from_numpy(op.vecs).to(dev)
            mirror.insert(ids, vecs)
            staged.append(("insert", ids, vecs, None))
        elif op.kind == "delete":
            ids = torch.from_numpy(op.ids.astype(np.int32)).to(dev)
            mirror.delete(ids)
            staged.append(("delete", ids, None, None))
        else:
            q = torch.from_numpy(op.vecs).to(dev)
            gt = mirror.knn(q, spec.k)
            outs = (torch.empty((q.shape[0], spec.k), dtype=torch.int32, device=dev),
                    torch.empty((q.shape[0], spec.k), dtype=torch.float32, device=dev))
            staged.append(("search", q, outs, gt))
    torch.cuda.synchronize()
    log(f"pattern {args.pattern}: {len(staged)} operations staged")
    ev = []
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for kind, a, b, _ in staged:
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        if kind == "insert":
            g.insert(a, b)
        elif kind == "delete":
            g.delete(a)
        else:
            g.search(a, spec.k, spec.beam, out_ids=b[0], out_dists=b[1])
        e1.record(stream)
        ev.append((kind, int(a.shape[0]), e0, e1))
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    upd_ms = sum(e0.elapsed_time(e1) for k, n, e0, e1 in ev if k != "search")
    upd_n = sum(n for k, n, e0, e1 in ev if k != "search")
    q_ms = sum(e0.elapsed_time(e1) for k, n, e0, e1 in ev if k == "search")
    q_n = sum(n for k, n, e0, e1 in ev if k == "search")
    recalls = []
    for kind, q, outs, gt in staged:
        if kind == "search":
            hit = (outs[0].to(torch.int64)[:, :, None] == gt[:, None, :]).any(2).sum(1).float()
            recalls.append(float(hit.mean() / spec.k))
    counts = {k: sum(1 for x in staged if x[0] == k) for k in ("insert", "delete", "search")}
    rmin = round(min(recalls), 4) if recalls else None
    res = {"metric": f"updates/sec and search QPS, {args.pattern} pattern, {SHAPE.get(args.workload, args.workload)}, "
                     f"1 MI355X",
           "value": round(upd_n / (upd_ms / 1e3), 1) if upd_ms > 0 else None, "unit": "updates/s", "n_gpus": 1,
           "higher_is_better": True, "dtype": "u8" if cfg.dtype == "u8" else "f32",
           "data": DATA_LABEL.get(args.workload, "synthetic"),
           "config": {"workload": w.wdef.description, "pattern": args.pattern, "points": spec.base_n,
                      "batch": ps.batch, "queries_per_search": spec.n_query, "k": spec.k, "beam": spec.beam,
                      "operations": counts},
           "search_qps": round(q_n / (q_ms / 1e3), 1) if q_ms > 0 else None,
           "overall_ops_per_s": round((upd_n + q_n) / wall, 1),
           "recall_at_10_min": rmin, "recall_at_10_mean": round(float(np.mean(recalls)), 4) if recalls else None,
           "wall_s": round(wall, 3), "build_s": round(build_s, 2)}
    print(json.dumps(res), flush=True)


# ------------------------------------------------------------------ concurrent rounds
def run_concurrent(g, snap, rounds, spec, torch, ops_total, seq_wall):
    """Replays `rounds` from `snap` with each round's searches on a reader
    (grand_reader_*: its own HIP stream, on a second host thread) overlapping
    that round's insert and delete batches; the round ends when both have
    finished.  Overall throughput = (inserts + deletes + queries) / time, the
    paper's overall measure (Section 6.1), against the same rounds run one
    call after another (the timed region)."""
    import threading

    from paper_2608_21163_amd import Reader
    g.import_graph(snap["vecs"], snap["adj"], snap["deg"], snap["active"], snap["medoid"])
    torch.cuda.synchronize()
    reader = Reader(g)
    start, done = threading.Barrier(2), threading.Barrier(2)
    job = {}
    errors = []

    def reader_loop():
        while True:
            start.wait()
            q = job.get("q")
            if q is None:
                return
            try:
                reader.search(q[0], spec.k, spec.beam, out_ids=q[1][0], out_dists=q[1][1])
            except Exception as e:  # reported after the run
                errors.append(e)
            done.wait()

    t = threading.Thread(target=reader_loop, daemon=True)
    t.start()
    recalls = []
    t0 = time.perf_counter()
    for ops in rounds:
        q = next((o for o in ops if o[0] == "search"), None)
        job["q"] = (q[1], q[2]) if q else None
        start.wait()
        for kind, a, b, _ in ops:
            if kind == "insert":
                g.insert(a, b)
            elif kind == "delete":
                g.delete(a)
        done.wait()
    wall = time.perf_counter() - t0
    job["q"] = None
    start.wait()
    t.join()
    reader.close()
    if errors:
        raise errors[0]
    for ops in rounds:
        for kind, q, outs, gt in ops:
            if kind == "search" and gt is not None:
                got = outs[0].to(torch.int64)
                hit = (got[:, :, None] == gt[:, None, :]).any(2).sum(1).float()
                recalls.append(float(hit.mean() / spec.k))
    return {"overall_ops_per_s": round(ops_total / wall, 1), "ms_per_round": round(wall * 1e3 / len(rounds), 3),
            "sequential_overall_ops_per_s": round(ops_total / seq_wall, 1),
            "sequential_ms_per_round": round(seq_wall * 1e3 / len(rounds), 3),
            "recall_at_10_min": round(min(recalls), 4) if recalls else None,
            "recall_note": "queries overlap their round's updates; ground truth is the state after the round",
            "mode": "each round's queries on a reader (own stream, second host thread) while its insert and "
                    "delete run"}


# ------------------------------------------------------------------ reverse-graph microbenchmark
def reverse_microbench(g, w, spec, reps=5):
    """In-neighbour detection for the first round's delete batch (Section 4.2
    compares building the reverse graph with a linear scan of the graph for
    each deleted point).  The reverse builds run on the whole batch; the
    per-id scan costs n passes over the adjacency, so it is timed on subsets
    and its time per id is scaled to the batch.  All methods must agree."""
    import numpy as np
    from paper_2608_21163_amd.grand import INDEG_REV_BATCH, INDEG_REV_FULL, INDEG_SCAN
    ops = {op.kind: op for op in w.round_ops(0)}
    dele = ops["delete"].ids
    # the delete batch of round 0 follows its insert batch; the ids it deletes
    # are all active in the built index except those inserted in round 0
    ids = dele[np.isin(dele, ops["insert"].ids, invert=True)] if "insert" in ops else dele
    res = {"batch": int(len(ids))}
    ref = None
    for name, m in (("reverse_batch_rows", INDEG_REV_BATCH), ("reverse_full", INDEG_REV_FULL)):
        times = []
        for _ in range(reps):
            cnt, ms = g.count_in_edges(ids, m)
            times.append(ms)
        if ref is None:
            ref = cnt
        assert np.array_equal(cnt, ref), name
        res[name + "_ms"] = round(float(np.median(times)), 4)
        log(f"reverse microbench: {name} {res[name + '_ms']} ms")
    per_id = []
    for n in (16, 64, 256):
        times = []
        for _ in range(3):
            cnt, ms = g.count_in_edges(ids[:n], INDEG_SCAN)
            times.append(ms)
        assert np.array_equal(cnt, ref[:n]), n
        t = float(np.median(times))
        per_id.append(t / n)
        res[f"scan_{n}_ids_ms"] = round(t, 4)
        log(f"reverse microbench: scan of {n} ids {t:.3f} ms")
    res["scan_ms_per_id"] = round(per_id[-1], 5)
    res["scan_batch_ms_scaled"] = round(per_id[-1] * len(ids), 2)
    res["speedup_batch_rows_vs_scan"] = round(res["scan_batch_ms_scaled"] / res["reverse_batch_rows_ms"], 1)
    res["speedup_full_vs_scan"] = round(res["scan_batch_ms_scaled"] / res["reverse_full_ms"], 1)
    res["in_edges_found"] = int(ref.sum())
    print(json.dumps({"reverse_microbench": res, "config": w.wdef.description}), flush=True)


# ------------------------------------------------------------------ main
def main():
    args = parse()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py: the update path runs on one GPU; a multi-GPU run "
              "(sharding by id, one index per GPU) is not implemented", file=sys.stderr)
        sys.exit(2)
    if args.copy_probe:
        copy_probe()
        return
    if args.pattern:
        run_pattern(args)
        return
    import numpy as np
    import torch

    from paper_2608_21163_amd import GrandIndex
    from paper_2608_21163_amd.grand import REV_BATCH, REV_FULL
    from workloads import make_workload
    from workloads.generators import Op, cagra_init_lists

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    torch.backends.cuda.matmul.allow_tf32 = False
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    stream = torch.cuda.current_stream()
    W, K = args.warmup, args.steps
    st_over = dict(n_rounds=W + K)
    if args.base:
        st_over["base_n"] = args.base
    if args.build_batch:
        st_over["build_batch"] = args.build_batch
    if args.build_frac >= 0.0:
        st_over["build_frac"] = args.build_frac
    if args.build_min:
        st_over["build_min"] = args.build_min
    idx_over = {"prune_rule": args.prune_rule} if args.prune_rule else None
    w = make_workload(args.workload, seed=args.seed, index=idx_over, stream=st_over)
    cfg, spec = w.cfg, w.spec
    sdim = cfg.dim + (1 if cfg.metric == "mips" else 0)   # stored row (the MIPS augmentation adds one)
    stride = ((sdim * (1 if cfg.dtype == "u8" else 4)) + 15) // 16 * 16
    g = GrandIndex.from_config(cfg, max_batch=max(spec.build_batch, spec.n_insert, spec.n_delete),
                               stream=stream.cuda_stream,
                               rev_mode=REV_BATCH if args.rev_mode == "batch" else REV_FULL)
    mirror = Mirror(torch, cfg, dev)

    def dev_ids(a):
        return torch.from_numpy(a.astype(np.int32)).to(dev)

    def dev_vecs(a):
        return torch.from_numpy(a).to(dev)

    # ---- build (untimed)
    cagra = cfg.algo == "cagra"
    refresh = args.refresh_passes if args.refresh_passes >= 0 else spec.refresh
    t0 = time.perf_counter()
    nb = npts = 0
    base_ops = []
    construct_s = None
    batches = list(w.base_batches())
    if cagra and args.cagra_seed == "full":  # the whole base in one construction
        batches = [Op("insert", np.concatenate([b.ids for b in batches]), np.concatenate([b.vecs for b in batches]))]
    for op in batches:
        ids, vecs = dev_ids(op.ids), dev_vecs(op.vecs)
        if cagra and nb == 0 and args.cagra_seed != "bootstrap":
            # the seed graph by the CAGRA graph construction (random initial
            # lists drawn here, as the library takes them as input)
            init = torch.from_numpy(cagra_init_lists(len(op.ids), args.cagra_knn, args.seed).view(np.int32)).to(dev)
            torch.cuda.synchronize()
            tc = time.perf_counter()
            g.build_cagra(ids, vecs, init, args.cagra_knn, args.cagra_rounds, args.cagra_sample)
            torch.cuda.synchronize()
            construct_s = time.perf_counter() - tc
            log(f"build: seed graph of {len(op.ids):,} points constructed in {construct_s:.2f} s")
            del init
        else:
            g.insert(ids, vecs)
        mirror.insert(ids, vecs)
        base_ops.append((ids, vecs))
        nb += 1
        npts += len(op.ids)
        if nb % 50 == 0:
            log(f"build: {npts:,} points, {time.perf_counter() - t0:.1f} s")
    # refresh passes: the same points leave and re-enter batch by batch, so
    # every list is rebuilt against the complete base set
    for _ in range(refresh):
        for ids, vecs in base_ops:
            g.delete(ids)
            g.insert(ids, vecs)
    del base_ops
    torch.cuda.synchronize()
    build_s = time.perf_counter() - t0
    log(f"build done: {spec.base_n:,} points in {build_s:.1f} s")
    if cagra and args.cagra_seed != "bootstrap":
        how = ("the whole base by one CAGRA graph construction" if args.cagra_seed == "full" else
               f"the first {len(batches[0].ids):,} points by the CAGRA graph construction, then "
               f"{len(batches) - 1} insert batches")
        base_build_label = (f"{how} (NN-Descent k-NN degree {args.cagra_knn}, {args.cagra_rounds} rounds, sample "
                            f"{args.cagra_sample}; rank-based pruning; reverse edges), {refresh} refresh pass(es) "
                            f"(untimed)")
    else:
        base_build_label = (f"{len(spec.build_sizes())} insert batches, then {refresh} refresh pass(es) deleting "
                            f"and re-inserting each base batch (untimed)")

    if args.reverse_microbench:
        reverse_microbench(g, w, spec)
        return

    # ---- stage every round's inputs on the device, with exact ground truth;
    # the pool as the timed rounds find it is kept for the counting rerun and
    # the CPU baseline, and the first CPU_ROUNDS timed rounds' batches on the
    # host
    rounds = []
    snap_vecs = None
    host_round = []
    for r in range(W + K):
        if r == W:
            snap_vecs = mirror.pool.clone()
        ops = []
        for op in w.round_ops(r):
            if W <= r < W + CPU_ROUNDS:
                host_round.append((op.kind, op.ids, op.vecs))
            if op.kind == "insert":
                ids, vecs = dev_ids(op.ids), dev_vecs(op.vecs)
                mirror.insert(ids, vecs)
                ops.append(("insert", ids, vecs, None))
            elif op.kind == "delete":
                ids = dev_ids(op.ids)
                mirror.delete(ids)
                ops.append(("delete", ids, None, None))
            else:
                q = dev_vecs(op.vecs)
                gt = None if args.no_recall else mirror.knn(q, spec.k)
                out_i = torch.empty((q.shape[0], spec.k), dtype=torch.int32, device=dev)
                out_d = torch.empty((q.shape[0], spec.k), dtype=torch.float32, device=dev)
                ops.append(("search", q, (out_i, out_d), gt))
        rounds.append(ops)
    torch.cuda.synchronize()
    log(f"staged {W + K} rounds")

    def run_round(ops, events):
        for kind, a, b, _ in ops:
            e0 = torch.cuda.Event(enable_timing=True)
            e1 = torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            if kind == "insert":
                g.insert(a, b)
            elif kind == "delete":
                g.delete(a)
            else:
                g.search(a, spec.k, spec.beam, out_ids=b[0], out_dists=b[1])
            e1.record(stream)
            events.append((kind, int(a.shape[0]), e0, e1))

    for r in range(W):
        run_round(rounds[r], [])
    snap = g.export()     # the state the timed rounds start from
    snap["vecs"] = snap_vecs
    g.reset_stats()
    g.set_timing(True)
    events = []
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for r in range(W, W + K):
        run_round(rounds[r], events)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    st = g.stats()
    g.set_timing(False)

    upd_ms = sum(e0.elapsed_time(e1) for k, n, e0, e1 in events if k != "search")
    upd_n = sum(n for k, n, e0, e1 in events if k != "search")
    q_ms = sum(e0.elapsed_time(e1) for k, n, e0, e1 in events if k == "search")
    q_n = sum(n for k, n, e0, e1 in events if k == "search")
    ins_ms = sum(e0.elapsed_time(e1) for k, n, e0, e1 in events if k == "insert")
    del_ms = sum(e0.elapsed_time(e1) for k, n, e0, e1 in events if k == "delete")

    recalls = []
    if not args.no_recall:
        for r in range(W + K):
            for kind, q, outs, gt in rounds[r]:
                if kind != "search":
                    continue
                got = outs[0].to(torch.int64)
                hit = (got[:, :, None] == gt[:, None, :]).any(2).sum(1).float()
                recalls.append(float(hit.mean() / spec.k))

    # ---- counting rerun (untimed): the same rounds from the same state, with
    # an exact visited set in every search, give the distinct ids whose
    # distance each search needs.  The path is deterministic, so the rerun
    # performs the same searches as the timed rounds.
    distinct = None
    t0 = time.perf_counter()
    g.import_graph(snap["vecs"], snap["adj"], snap["deg"], snap["active"], snap["medoid"])
    g.reset_stats()
    g.set_counting(True)
    for r in range(W, W + K):
        run_round(rounds[r], [])
    torch.cuda.synchronize()
    cst = g.stats()
    g.set_counting(False)
    same = all(cst[f"hops_{x}"] == 0 for x in ("insert", "delete", "query"))
    distinct = {x: cst[f"distinct_{x}"] for x in ("insert", "delete", "query")}
    log(f"counting rerun: {time.perf_counter() - t0:.1f} s; distinct {distinct} (counters of the timed kernels "
        f"untouched: {same})")

    # ---- overall throughput (untimed for the headline value): the same rounds
    # from the same state, each round's queries on a reader (its own stream and
    # host thread) while the round's insert and delete run.
    concurrent = None
    if not args.no_concurrent:
        concurrent = run_concurrent(g, snap, rounds[W:W + K], spec, torch, upd_n + q_n, wall)
        log(f"concurrent rounds: overall {concurrent['overall_ops_per_s']:.0f} ops/s "
            f"(sequential {concurrent['sequential_overall_ops_per_s']:.0f})")

    # ---- roofline of the dominant kernel (largest share of the timed region).
    # Phase times come from HIP events on the library stream around each
    # phase.  The three search phases are launches of one kernel (k_search);
    # every other phase with a byte count is reported on its own.
    phases = {}
    for ph, ms in st["phase_ms"].items():
        calls = st["phase_calls"][ph]
        if calls == 0:
            continue
        b = algorithmic_bytes(st, ph, cfg, stride, distinct)
        phases[ph] = {"ms_total": round(ms, 3), "launches": int(calls), "ms_per_launch": round(ms / calls, 4)}
        if b is not None:
            phases[ph]["alg_bytes"] = b
            phases[ph]["alg_GB_per_launch"] = round(b / calls / 1e9, 5)
            phases[ph]["achieved_GBps"] = round(b / (ms / 1e3) / 1e9, 1)
            if ph.startswith("search_"):
                be = algorithmic_bytes(st, ph, cfg, stride, None)
                phases[ph]["alg_bytes_all_evals"] = be
    groups = {}
    for ph, v in phases.items():
        if "alg_bytes" not in v:
            continue
        kern = "k_search" if ph.startswith("search_") else ph
        g_ = groups.setdefault(kern, {"ms": 0.0, "launches": 0, "bytes": 0.0, "bytes_all": 0.0, "phases": []})
        g_["ms"] += v["ms_total"]
        g_["launches"] += v["launches"]
        g_["bytes"] += v["alg_bytes"]
        g_["bytes_all"] += v.get("alg_bytes_all_evals", v["alg_bytes"])
        g_["phases"].append(ph)
    profiled_ok = args.workload == "sift1m_u8" and not args.base and not args.build_batch

    def roof(kern):
        g_ = groups[kern]
        ach = g_["bytes"] / (g_["ms"] / 1e3) / 1e9
        tb = None
        if profiled_ok:
            per = [profiled_traffic(ph) for ph in g_["phases"]]
            if all(x is not None for x in per):
                # per-launch traffic of each phase, weighted by its launches
                tb = sum(x * phases[ph]["launches"] for x, ph in zip(per, g_["phases"])) / g_["launches"]
        out = {"bound": "hbm", "kernel": kern, "phases": g_["phases"], "achieved": round(ach, 1),
               "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": round(ach / HBM_PEAK_GBS, 4),
               "traffic": None if tb is None else round(tb / 1e9, 5),
               "traffic_unit": "GB per launch, HBM read + write (rocprofv3 FETCH_SIZE and WRITE_SIZE, "
                               "calibrated on a 1 GiB copy; profiles/traffic_sift1m_u8.md)",
               "ms_per_launch": round(g_["ms"] / g_["launches"], 4),
               "alg_GB_per_launch": round(g_["bytes"] / g_["launches"] / 1e9, 5),
               "ms_total": round(g_["ms"], 3)}
        if kern == "k_search":
            ach_all = g_["bytes_all"] / (g_["ms"] / 1e3) / 1e9
            out["bytes_basis"] = "distinct distance evaluations (counting rerun)"
            out["frac_all_evaluations"] = round(ach_all / HBM_PEAK_GBS, 4)
            out["alg_GB_per_launch_all_evaluations"] = round(g_["bytes_all"] / g_["launches"] / 1e9, 5)
        return out

    dom = max(groups, key=lambda k: groups[k]["ms"]) if groups else None
    roofline = roof(dom) if dom else None
    others = {k: roof(k) for k in groups if k != dom}
    for v in phases.values():
        v.pop("alg_bytes", None)
        v.pop("alg_bytes_all_evals", None)

    searches = {"insert": st["inserted"], "delete": st["deleted"], "query": st["queried"]}
    search_stats = {x: {"searches": int(searches[x]), "hops": int(st[f"hops_{x}"]),
                        "evaluations": int(st[f"evals_{x}"]), "distinct": int(distinct[x]),
                        "repeat_frac": round(1.0 - distinct[x] / max(st[f"evals_{x}"], 1), 4),
                        "max_iters_hits": int(st[f"capped_{x}"]),
                        "max_iters_hit_rate": round(st[f"capped_{x}"] / max(searches[x], 1), 5)}
                    for x in ("insert", "delete", "query") if searches[x]}

    cpu = None
    if not args.no_cpu_baseline:
        snap_host = dict(snap)
        snap_host["vecs"] = snap["vecs"].cpu().numpy()
        n_cpu = min(CPU_ROUNDS, K)
        cpu = cpu_baseline(cfg, spec, snap_host, host_round, n_cpu, oracle_threads())
        if args.workload == "tiny":
            cpu["one_core"] = cpu_baseline(cfg, spec, snap_host, host_round, n_cpu, 1)

    value = upd_n / (upd_ms / 1e3)
    rmin = round(min(recalls), 4) if recalls else None
    res = {
        "metric": metric_of(args.workload, rmin), "value": round(value, 1), "unit": "updates/s", "n_gpus": 1,
        "steps": K, "warmup": W, "ms_per_step": round(wall * 1e3 / K, 3), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "u8" if cfg.dtype == "u8" else "f32",
        "data": DATA_LABEL.get(args.workload, "synthetic"),
        "config": {"workload": w.wdef.description, "base_points": spec.base_n, "insert_batch": spec.n_insert,
                   "delete_batch": spec.n_delete, "queries": spec.n_query, "k": spec.k, "beam": spec.beam,
                   "R": cfg.R, "L": cfg.L_build, "alpha": cfg.alpha, "P": cfg.P, "c": cfg.c,
                   "k_repair": cfg.k_repair, "reverse_graph": args.rev_mode, "parallelism": "single GPU",
                   "base_build": base_build_label},
        "search_qps": round(q_n / (q_ms / 1e3), 1),
        "insert_per_s": round(spec.n_insert * K / (ins_ms / 1e3), 1),
        "delete_per_s": round(spec.n_delete * K / (del_ms / 1e3), 1),
        "recall_at_10_min": rmin,
        "recall_at_10_mean": round(float(np.mean(recalls)), 4) if recalls else None,
        "recall_at_10_per_round": [round(x, 4) for x in recalls],
        "build_s": round(build_s, 2),
        "construct_s": round(construct_s, 3) if construct_s is not None else None,
        "roofline": roofline,
        "roofline_other_phases": others,
        "cpu_baseline": cpu,
        "concurrent": concurrent,
        "searches": search_stats,
        "phases": phases,
        "counters": {k: v for k, v in st.items() if isinstance(v, int)},
    }
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
