"""Throughput of the RheoSampling hot path on one MI355X.

A *step* is one full draft+verify pass of the tree machinery for a batch of
B sequences: depth x rheo_expand_level, rheo_prune, rheo_verify (every row of
the hot path) on synthetic logits that are already resident in HBM.

Protocol
  1. discovery: run_step() generates each level's draft rows from the
     frontier the library picks and the target rows of the pruned tree, and
     records them (several distinct steps, so the timed loop does not re-read
     one step's rows from cache).
  2. timed replay: W warm-up steps, then K steps of the library calls only,
     cycling over the recorded steps, bracketed by torch.cuda.synchronize();
     every replay must reproduce the discovery outputs bit for bit.
  3. HIP events around each rheo_expand_level call (on the stream it launches
     on) give the duration of an expand level (its selection and pool kernels, the
     dominant work); its algorithmic bytes are the draft rows it must read
     (rows x V x 2 bytes): one event pair around each step's depth
     consecutive expand calls gives the average launch duration (events
     around every level, in a pass of their own, give the per-level
     breakdown).  Both passes start behind a spin kernel that holds the
     stream while the host queues the steps, so the launches run back to
     back and the events time the kernels rather than the Python loop's
     launch latency.  Then the same steps are captured as HIP graphs
     (one per recorded step) and replayed; `value` is the faster of the
     eager launch loop and the graph replay (`mode` says which; both are
     reported), the eager loop alone with --graph 0.
  4. cpu_baseline: the CPU oracle timed on a bounded sample of the same
     workload (one step of a few sequences, rows pre-generated).
Prints one JSON line on stdout.
"""

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "tree draft+verify steps/sec at V=128k batch 64; achieved HBM GB/s vs peak"
PEAK_HBM_GBPS = 8000.0


def log(*a):
    print(*a, file=sys.stderr, flush=True)


KERNEL_SRCS = ["expand.hip", "dense.hip", "pool_common.h", "rheo_device.h", "rheo_state.h"]
EXPAND_KERNELS = r"k_select|k_pool|k_dweights|k_dpool|k_expand_row"


def kernel_src_hash():
    import hashlib
    h = hashlib.sha256()
    for f in KERNEL_SRCS:
        with open(os.path.join(ROOT, "paper_2609_21827_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def _counter_rows(path, regex, counter):
    """Per-dispatch values (KiB) of one counter for kernels matching regex."""
    import csv
    import re
    vals = {}
    with open(path) as f:
        for row in csv.DictReader(f):
            if row["Counter_Name"] == counter and re.search(regex, row["Kernel_Name"]):
                key = row.get("Dispatch_Id") or row.get("Correlation_Id")
                vals[key] = vals.get(key, 0.0) + float(row["Counter_Value"])
    return list(vals.values())


_SPIN = {}


def hold_stream(ms):
    """Keeps the current stream busy for about `ms` milliseconds with torch's
    spin kernel, so that the launches the host queues behind it start back
    to back once it ends."""
    import torch
    if "per_ms" not in _SPIN:
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda._sleep(1000)
        e0.record()
        torch.cuda._sleep(1 << 20)
        e1.record()
        torch.cuda.synchronize()
        _SPIN["per_ms"] = (1 << 20) / max(e0.elapsed_time(e1), 1e-3)
    torch.cuda._sleep(max(1, int(ms * _SPIN["per_ms"])))


def expand_kernel_name(w):
    return ("expand level (k_expand_row)" if w.support > 0
            else "expand level (k_select + k_dweights + k_dpool)")


def write_traffic(paths, out, w, copy_bytes):
    """Scales the expand kernel's FETCH_SIZE / WRITE_SIZE by what the same
    counters read for a plain device copy of known size."""
    exp_f, exp_w, cp_f, cp_w = paths
    # one expand level = one k_expand_row dispatch, or one k_select dispatch
    # and the pool kernel(s) after it
    nf = len(_counter_rows(exp_f, r"k_select|k_expand_row", "FETCH_SIZE"))
    nw = len(_counter_rows(exp_w, r"k_select|k_expand_row", "WRITE_SIZE"))
    ef = [sum(_counter_rows(exp_f, EXPAND_KERNELS, "FETCH_SIZE")) / nf]
    ew = [sum(_counter_rows(exp_w, EXPAND_KERNELS, "WRITE_SIZE")) / nw]
    cf = _counter_rows(cp_f, r"copy|Copy", "FETCH_SIZE")
    cw = _counter_rows(cp_w, r"copy|Copy", "WRITE_SIZE")
    # every copy dispatch moves copy_bytes in and copy_bytes out
    k_f = copy_bytes / (sum(cf) / len(cf) * 1024)
    k_w = copy_bytes / (sum(cw) / len(cw) * 1024)
    fetch = sum(ef) / len(ef) * 1024 * k_f
    write = sum(ew) / len(ew) * 1024 * k_w
    res = {"workload": w.name, "kernel": expand_kernel_name(w),
           "kernel_src_sha256": kernel_src_hash(),
           "levels": nf, "copy_dispatches": len(cf),
           "copy_bytes": copy_bytes,
           "copy_fetch_kib": sum(cf) / len(cf), "copy_write_kib": sum(cw) / len(cw),
           "scale_fetch": k_f, "scale_write": k_w,
           "fetch_kib_per_launch": sum(ef) / len(ef),
           "write_kib_per_launch": sum(ew) / len(ew),
           "bytes_per_launch": int(fetch + write),
           "fetch_bytes_per_launch": int(fetch), "write_bytes_per_launch": int(write)}
    with open(out, "w") as f:
        json.dump(res, f, indent=1)
        f.write("\n")
    print(json.dumps(res))


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default="headline")
    ap.add_argument("--distinct", type=int, default=4, help="recorded steps cycled over")
    ap.add_argument("--cpu-seconds", type=float, default=15.0)
    ap.add_argument("--no-cpu", action="store_true")
    ap.add_argument("--graph", type=int, default=1,
                    help="1: the timed loop replays each step as a captured HIP graph")
    ap.add_argument("--traffic", default=None,
                    help="traffic file (default profiles/expand_level_<workload>_traffic.json)")
    ap.add_argument("--copy-probe", type=int, default=0, metavar="MIB",
                    help="only run a plain device copy of MIB MiB five times "
                         "(counter calibration under rocprofv3 --pmc)")
    ap.add_argument("--sweep", choices=["table4", "methods", "rheostat", "support"],
                    default=None,
                    help="instead of the throughput line, print one JSON line per "
                         "configuration of a sweep (see run_sweep)")
    ap.add_argument("--traffic-from", nargs=4, default=None,
                    metavar=("EXP_FETCH", "EXP_WRITE", "COPY_FETCH", "COPY_WRITE"),
                    help="write the traffic file from four rocprofv3 --pmc "
                         "counter_collection.csv files, then exit")
    args = ap.parse_args()
    if args.traffic is None:
        args.traffic = os.path.join(ROOT, "profiles",
                                    f"expand_level_{args.workload}_traffic.json")

    if args.traffic_from:
        import synth
        assert args.copy_probe, "--traffic-from needs the --copy-probe size that was profiled"
        write_traffic(args.traffic_from, args.traffic, synth.WORKLOADS[args.workload],
                      args.copy_probe << 20)
        return

    if args.gpus != 1:
        print(f"bench.py measures one GPU only (asked for {args.gpus}); "
              "the hot path's multi-GPU sharding is a design, not a build", file=sys.stderr)
        sys.exit(2)

    import torch
    assert torch.cuda.is_available(), "bench.py needs a GPU"
    if args.copy_probe:
        n = args.copy_probe << 20
        src = torch.randint(0, 255, (n,), dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(5):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_bytes": n, "copies": 5}), flush=True)
        return

    if args.sweep:
        run_sweep(args)
        return

    import synth
    from paper_2609_21827_amd.driver import make_tree, run_step

    dev = "cuda"
    w = synth.WORKLOADS[args.workload]
    esz = w.elem_bytes
    tree = make_tree(w, device=dev)

    # ---- 1. discovery ------------------------------------------------------
    recs, outs = [], []
    for s in range(args.distinct):
        rec = {}
        acc, alen, fin = run_step(tree, w, s, device=dev, record=rec)
        recs.append(rec)
        outs.append((acc, alen, fin))
        log(f"discovery step {s}: mean accepted {alen.float().mean().item():.3f}")
    torch.cuda.synchronize()
    assert tree.device_error() == 0

    stream = torch.cuda.current_stream()
    out_bufs = [tuple(torch.empty_like(x, device=dev) for x in o) for o in outs]
    pv_buf = tuple(torch.empty((w.B, w.R + 1), dtype=torch.int32, device=dev) for _ in range(2))

    # the frontier each level chooses (which rows the draft model computes
    # next) is read in place through these views: no call, no copy
    fr_view = tree.frontier_view()

    def replay(i, events=None, stream_override=None, bracket=None):
        # the calls a serving loop makes: expand (x depth), prune, pruned
        # view (which rows the target model computes), verify
        stream = stream_override or torch.cuda.current_stream()
        rec = recs[i % len(recs)]
        ob = out_bufs[i % len(recs)]
        tree.begin_step()
        if bracket is not None:
            bracket[0].record(stream)
        for d, rows in enumerate(rec["draft"]):
            if events is not None:
                events[d][0].record(stream)
            tree.expand_level(rows, rec["T"], rec["rng_key"], stream=stream)
            if events is not None:
                events[d][1].record(stream)
        if bracket is not None:
            bracket[1].record(stream)
        tree.prune(w.R, stream=stream)
        tree.pruned_view(out=pv_buf, stream=stream)
        tree.verify(rec["target"], rec["T"], rec["rng_key"], out=ob, stream=stream)

    # ---- 2. timed replay ---------------------------------------------------
    def check_one(i):
        for a, b in zip(out_bufs[i], outs[i]):
            assert torch.equal(a.cpu(), b.cpu()), "replay differs from discovery"

    def check(n_replayed):
        for i in range(min(n_replayed, len(recs))):
            check_one(i)

    for i in range(args.warmup):
        replay(i)
    torch.cuda.synchronize()
    check(args.warmup)
    t0 = time.perf_counter()
    for i in range(args.steps):
        replay(i)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    check(args.steps)
    assert tree.device_error() == 0
    eager_ms = (t1 - t0) * 1e3 / args.steps
    ms, steps_per_s, mode = eager_ms, args.steps / (t1 - t0), "eager"

    # the event pass: the same steps with events around every expand level,
    # queued behind a spin that outlasts the host's enqueueing of them
    ev = [[[torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)]
           for _ in range(w.depth)] for _ in range(args.steps)]
    torch.cuda.synchronize()
    hold_stream(1.5 * eager_ms * args.steps + 5.0)
    for i in range(args.steps):
        replay(i, ev[i])
    torch.cuda.synchronize()
    check(args.steps)
    assert tree.device_error() == 0
    event_pass_ms = ev[0][0][0].elapsed_time(ev[-1][-1][1]) / args.steps
    # the roofline figure: one event pair around each step's depth
    # consecutive expand launches (no event packets between the levels)
    br = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(args.steps)]
    torch.cuda.synchronize()
    hold_stream(1.5 * eager_ms * args.steps + 5.0)
    for i in range(args.steps):
        replay(i, bracket=br[i])
    torch.cuda.synchronize()
    check(args.steps)
    assert tree.device_error() == 0
    bracket_ms = sum(a.elapsed_time(b) for a, b in br)

    # ---- 3. the same steps replayed as HIP graphs (one per recorded step):
    #      the launch sequence of a step is captured once and replayed; every
    #      replay must still reproduce the discovery outputs -------------------
    graph_ms = None
    graph_error = None
    if args.graph:
        try:
            cap = torch.cuda.Stream()
            graphs = []
            for i in range(len(recs)):
                g = torch.cuda.CUDAGraph()
                with torch.cuda.graph(g, stream=cap):
                    replay(i, stream_override=cap)
                graphs.append(g)
            torch.cuda.synchronize()
            for i in range(max(args.warmup, len(recs))):
                for o in out_bufs[i % len(recs)]:
                    o.fill_(-7)
                graphs[i % len(recs)].replay()
                torch.cuda.synchronize()
                check_one(i % len(recs))
            torch.cuda.synchronize()
            g0 = time.perf_counter()
            for i in range(args.steps):
                graphs[i % len(recs)].replay()
            torch.cuda.synchronize()
            g1 = time.perf_counter()
            check(args.steps)
            assert tree.device_error() == 0
            graph_ms = (g1 - g0) * 1e3 / args.steps
            if graph_ms < eager_ms:
                ms, steps_per_s, mode = graph_ms, args.steps / (g1 - g0), "hip-graph"
        except (RuntimeError, AssertionError) as e:
            graph_error = str(e)
            log(f"graph replay unavailable ({e}); reporting the eager launch loop")

    # algorithmic bytes: every draft row once, the target rows on each walk
    rows_per_level = [w.B] + [w.B * w.n_expand] * (w.depth - 1)
    draft_bytes = sum(rows_per_level) * w.V * esz
    walk_rows = [int((o[1] + 1).sum()) for o in outs]
    target_bytes = [r * w.V * esz for r in walk_rows]
    step_bytes = [draft_bytes + tb for tb in target_bytes]
    mean_step_bytes = sum(step_bytes[i % len(recs)] for i in range(args.steps)) / args.steps
    tokens_per_step = sum(walk_rows) / len(walk_rows)

    exp_ms = [[e[0].elapsed_time(e[1]) for e in ev[i]] for i in range(args.steps)]
    n_launch = args.steps * w.depth
    avg_launch_us = bracket_ms * 1e3 / n_launch
    bytes_per_launch = draft_bytes / w.depth
    achieved = bytes_per_launch / (avg_launch_us * 1e-6) / 1e9
    lvl_us = [sum(exp_ms[i][d] for i in range(args.steps)) * 1e3 / args.steps
              for d in range(w.depth)]

    # HBM bytes per launch from the committed counter runs, only while the
    # kernel sources still hash to what was profiled
    traffic = None
    if os.path.exists(args.traffic):
        with open(args.traffic) as f:
            tr = json.load(f)
        if tr.get("workload") == w.name and tr.get("kernel_src_sha256") == kernel_src_hash():
            traffic = tr.get("bytes_per_launch")

    # ---- 4. CPU oracle baseline, and the streaming-read ceiling -----------
    cpu = None if args.no_cpu else cpu_baseline(w, args.cpu_seconds)
    ceiling = stream_ceiling()

    res = {
        "metric": METRIC,
        "value": round(steps_per_s, 3),
        "unit": "steps/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": w.dtype,
        "data": "synthetic",
        "config": {"workload": f"{w.name}: B={w.B} V={w.V} K={w.K} m={w.m} depth={w.depth} "
                               f"budget={w.R} T={w.T} "
                               + (f"sparse top-{w.support}" if w.support > 0 else "dense")
                               + f" {w.dtype}",
                   "batch": w.B, "vocab": w.V, "K": w.K, "m": w.m, "depth": w.depth,
                   "budget": w.R, "T": w.T, "support": w.support},
        "mode": mode,
        "eager_ms_per_step": round(eager_ms, 4),
        "graph_ms_per_step": None if graph_ms is None else round(graph_ms, 4),
        "graph_error": graph_error,
        "event_pass_ms_per_step": round(event_pass_ms, 4),
        "roofline": {"bound": "hbm", "kernel": expand_kernel_name(w),
                     "achieved": round(achieved, 1), "peak": PEAK_HBM_GBPS,
                     "unit": "GB/s", "frac": round(achieved / PEAK_HBM_GBPS, 4),
                     "traffic": traffic,
                     "stream_read_ceiling_GBps": ceiling,
                     "avg_launch_us": round(avg_launch_us, 2),
                     "avg_launch_us_per_level_events": round(
                         sum(sum(x) for x in exp_ms) * 1e3 / n_launch, 2),
                     "bytes_per_launch": int(bytes_per_launch)},
        "cpu_baseline": cpu,
        "step_hbm_GBps": round(mean_step_bytes / (ms * 1e-3) / 1e9, 1),
        "step_hbm_frac": round(mean_step_bytes / (ms * 1e-3) / 1e9 / PEAK_HBM_GBPS, 4),
        "tokens_per_s": round(steps_per_s * tokens_per_step, 1),
        "mean_accept_len": round(tokens_per_step / w.B - 1, 4),
        "expand_level_us": [round(x, 2) for x in lvl_us],
    }
    print(json.dumps(res), flush=True)
    tree.close()


def cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def host_cores():
    """Cores this process may use (the box's share: at most 16)."""
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:
        n = os.cpu_count() or 1
    return max(1, min(16, n))


def _cpu_worker(w, seqs, barrier, q):
    """One worker of the CPU baseline: generates the rows of its sequences,
    waits for every worker, then times the oracle on them (method only)."""
    import torch
    torch.set_num_threads(1)
    from oracle.harness import oracle_step
    cache = {}
    for b in seqs:
        oracle_step(w, b, 0, row_cache=cache)
    barrier.wait()
    t0 = time.perf_counter()
    for b in seqs:
        oracle_step(w, b, 0, row_cache=cache)
    q.put((t0, time.perf_counter(), len(seqs)))


def _cpu_run(w, nworkers, seqs_per_worker):
    import multiprocessing as mp
    ctx = mp.get_context("spawn")
    barrier, q = ctx.Barrier(nworkers), ctx.Queue()
    procs = []
    for k in range(nworkers):
        seqs = [(k * seqs_per_worker + i) % w.B for i in range(seqs_per_worker)]
        p = ctx.Process(target=_cpu_worker, args=(w, seqs, barrier, q))
        p.start()
        procs.append(p)
    res = [q.get() for _ in procs]
    for p in procs:
        p.join()
    t0 = min(r[0] for r in res)
    t1 = max(r[1] for r in res)
    n = sum(r[2] for r in res)
    return n, t1 - t0


def cpu_baseline(w, seconds):
    """The CPU oracle on the host's cores (one process per core, rows
    pre-generated, each worker timing its share of one step's sequences),
    and on one core; steps/s of the whole batch."""
    cores = host_cores()
    # one sequence on one core sizes the sample to about `seconds`
    n1, t1 = _cpu_run(w, 1, 1)
    per_seq = t1 / n1
    per_worker = max(1, min(w.B, int(seconds / 2 / per_seq)))
    n_all, t_all = _cpu_run(w, cores, max(1, min(per_worker, -(-w.B // cores))))
    n_one, t_one = _cpu_run(w, 1, max(1, min(w.B, int(seconds / 2 / per_seq))))
    return {"value": round(n_all / t_all / w.B, 5), "unit": "steps/s", "cores": cores,
            "kind": "oracle", "cpu_model": cpu_model(),
            "single_core_value": round(n_one / t_one / w.B, 5),
            "sample": f"{n_all} sequences of one {w.name} step on {cores} processes "
                      f"({t_all:.1f} s wall), {n_one} on one ({t_one:.1f} s); rows "
                      f"pre-generated, the method timed; steps/s = sequences/s / B"}


def stream_ceiling(gib=2, reps=5):
    """GB/s of a plain streaming read (16-byte non-temporal loads, 512-thread
    blocks reading 256 KiB chunks) of a buffer larger than the Infinity
    Cache: the best of a few grid sizes."""
    import ctypes
    import torch
    lib = ctypes.CDLL(os.path.join(ROOT, "paper_2609_21827_amd", "libstreamprobe.so"))
    lib.stream_read_probe.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_int64,
                                      ctypes.c_int, ctypes.c_void_p, ctypes.c_void_p]
    n = gib << 30
    buf = torch.empty(n, dtype=torch.uint8, device="cuda")
    buf.fill_(1)
    out = torch.zeros(1, dtype=torch.int32, device="cuda")
    st = torch.cuda.current_stream()
    best = 0.0
    for blocks in (512, 1024, 2048, 4096):
        for r in range(reps + 1):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            rc = lib.stream_read_probe(buf.data_ptr(), n, 262144, blocks, out.data_ptr(),
                                       st.cuda_stream)
            e1.record()
            torch.cuda.synchronize()
            assert rc == 0, rc
            if r:
                best = max(best, n / (e0.elapsed_time(e1) * 1e-3) / 1e9)
    del buf
    return round(best, 1)


def run_sweep(args):
    """Sweeps on the batched shape (B = 64, V = 128256 bf16, synthetic rows),
    one JSON line per configuration:
      table4    single-layer acceptance (depth 1, K = 3: top-1, the sampled
                token, the best remaining token) of the three methods
                (App. A, Table 4: Top-K <= RRSw <= Rheo);
      methods   tau = mean tokens emitted per sequence and step, full tree,
                per method (App. A, Table 3);
      rheostat  tau over the leads m and the temperature T (Sec. 5.4);
      support   sparse support S (and the dense tree): top-S coverage of the
                untempered draft distribution, expand-level time, tau
                (Sec. 5.5, Table 5); also two supports with the construction
                over the whole vocabulary (the tail still sparse).
    Acceptance and tau come from the GPU path itself on seeded steps."""
    import torch
    import synth
    from paper_2609_21827_amd.driver import make_tree, run_step, replay_step

    dev = "cuda"
    base = synth.WORKLOADS["headline"]

    def steps_stats(w, nsteps, first=0):
        tree = make_tree(w, device=dev)
        try:
            lens = []
            for s in range(first, first + nsteps):
                _, alen, _ = run_step(tree, w, s, device=dev)
                lens.append(alen)
            assert tree.device_error() == 0
        finally:
            tree.close()
        alen = torch.cat(lens).double()
        return {"tau": round(float((alen + 1).mean()), 4),
                "accept_rate": round(float((alen >= 1).double().mean()), 4),
                "samples": int(alen.numel())}

    def emit(name, cfg, res):
        print(json.dumps({"sweep": name, "config": cfg, **res}), flush=True)

    if args.sweep == "table4":
        for method in ("topk", "rrsw", "rheo"):
            w = base.with_(name="table4_" + method, method=method, K=3, m=1, depth=1, R=3,
                            n_expand=1)
            emit("table4", {"method": method, "K": 3, "m": 1, "depth": 1},
                 steps_stats(w, 60))
    elif args.sweep == "methods":
        for method in ("topk", "rrsw", "rheo"):
            w = base.with_(name="methods_" + method, method=method)
            emit("methods", {"method": method, "K": w.K, "m": w.m, "depth": w.depth,
                             "budget": w.R}, steps_stats(w, 12))
    elif args.sweep == "rheostat":
        for m in (0, 1, 2, 3):
            for T in (0.2, 0.6, 1.0, 1.5):
                w = base.with_(name="rheostat", m=m, T=T)
                emit("rheostat", {"m": m, "T": T, "K": w.K, "depth": w.depth},
                     steps_stats(w, 4))
    else:
        for S, full in ((128, False), (256, False), (512, False), (1024, False), (0, False),
                        (128, True), (1024, True)):
            w = base.with_(name="support", support=S, construct_full=full)
            res = steps_stats(w, 6)
            # coverage of the top-S entries under the untempered draft
            # softmax, over the root rows and one level of frontier rows
            tree = make_tree(w, device=dev)
            rec = {}
            run_step(tree, w, 100, device=dev, record=rec)
            rows = torch.cat([r.reshape(-1, r.shape[-1])[:, :w.V] for r in rec["draft"][:2]]).float()
            lse = torch.logsumexp(rows, dim=1)
            if S > 0:
                top = torch.topk(rows, S, dim=1).values
                cov = torch.exp(torch.logsumexp(top, dim=1) - lse).mean().item()
            else:
                cov = 1.0
            # expand-level time, replayed with the rows resident in HBM
            for _ in range(3):
                replay_step(tree, rec, w.R)
            torch.cuda.synchronize()
            ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
                  for _ in range(10 * w.depth)]
            hold_stream(30.0)
            for it in range(10):
                tree.begin_step()
                for d, r in enumerate(rec["draft"]):
                    ev[it * w.depth + d][0].record()
                    tree.expand_level(r, rec["T"], rec["rng_key"])
                    ev[it * w.depth + d][1].record()
                tree.prune(w.R)
                tree.verify(rec["target"], rec["T"], rec["rng_key"])
            torch.cuda.synchronize()
            lvl = sum(a.elapsed_time(b) for a, b in ev) * 1e3 / len(ev)
            assert tree.device_error() == 0
            tree.close()
            emit("support", {"support": S if S > 0 else "full", "construct_full": full,
                             "K": w.K, "depth": w.depth},
                 {**res, "coverage": round(cov, 4), "expand_level_us": round(lvl, 2)})


if __name__ == "__main__":
    main()
