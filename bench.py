"""Benchmark of the in-place KV-cache splice on one MI355X.

One step = one splice call on the workload's synthetic cache, already resident in HBM: delete
the span, write the replacement, compact every downstream row and re-anchor its rotary band, in
all layers.  Prints one JSON line.

    python bench.py [--steps K] [--warmup W] [--workload NAME] [--gpus 1] [--no-cpu-baseline]
    python bench.py --summarize TRACE_DIR FETCH_DIR WRITE_DIR   # rocprofv3 output -> profiles/

Default workload: MLA DeepSeek-V3 shape (61 layers, c_kv 512 + k_pe 64, bf16), one 32768-token
sequence, a 4096-token span at a seeded start replaced by a 32-token stub, contiguous in place.
"""

import argparse
import csv
import glob
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "re-anchored KV tokens/sec and achieved HBM GB/s (% of peak) per splice"
PEAK_HBM_GBPS = 8000.0
# the sources of the device code and of the planning that shapes its launches
KERNEL_SOURCES = [os.path.join(ROOT, "paper_2606_01065_amd", "csrc", f)
                  for f in ("kernels.hip", "kparams.hpp", "plan.hpp", "plan.cpp")]
PROFILES = os.path.join(ROOT, "profiles")
CONTIG_KERNEL = "contig_move_kernel"
CONTIG_TILE_KERNEL = "contig_tile_kernel"
PAGED_KERNEL = "paged_data_kernel"
ROTATE_KERNEL = "rotate_rows_kernel"
ROTATE_REPLICAS = 4     # rotate-only: cache copies used round-robin (bands of two copies fit the last-level cache)
PAGED_REPLICAS = 4      # paged: at most this many pool copies used round-robin
COPY_KERNEL_HINT = "elementwise"        # torch's device copy kernel used for counter calibration


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default="mla_dsv3_32k")
    ap.add_argument("--replicas", type=int, default=2,
                    help="independent cache copies used round-robin (contiguous workloads), so "
                         "consecutive steps do not find each other's rows in the last-level cache")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=12.0)
    ap.add_argument("--summarize", nargs=3, metavar=("TRACE_DIR", "FETCH_DIR", "WRITE_DIR"))
    ap.add_argument("--counters", nargs="+", metavar="PMC_DIR",
                    help="rocprofv3 --pmc runs of the same bench command -> per-dispatch counter "
                         "table of the dominant kernel in profiles/counters_<kernel>_<workload>.md")
    ap.add_argument("--command", default="", help="command line recorded in --summarize output")
    ap.add_argument("--also", default="gqa_llama3_8b_16k,mla_dsv3_paged_131k,mla_dsv3_paged_b64,mla_dsv3_32k:exact,"
                                      "gqa_llama3_8b_16k:exact",
                    help="further workloads timed in the same run and reported under \"also\" "
                         "(comma-separated; NAME:exact runs libleyline_exact.so; empty: none)")
    ap.add_argument("--graph", action="store_true",
                    help="contiguous and rotate-only workloads: capture GRAPH_SPLICES consecutive splices "
                         "(cache copies in turn) into one HIP graph and time its replays")
    ap.add_argument("--exact", action="store_true",
                    help="run the workload on libleyline_exact.so (fp64 pair arithmetic) instead of libleyline.so")
    ap.add_argument("--cpu-procs", type=int, default=0,
                    help="processes of the all-cores oracle leg (0: every CPU this process may use, at most 16)")
    ap.add_argument("--cpu-leg", nargs=4, metavar=("DATA", "SECONDS", "PROCS", "OUT"),
                    help=argparse.SUPPRESS)
    return ap.parse_args()


def kernel_sha():
    """Identity of the code that the counter runs measured: sha256 of the kernel and planning
    sources with comments and blank lines removed, so that comment edits keep them valid (the
    sources use line comments only and no "//" inside string literals)."""
    h = hashlib.sha256()
    for path in KERNEL_SOURCES:
        with open(path, encoding="utf-8") as f:
            for line in f:
                code = line.split("//", 1)[0].strip()
                if code:
                    h.update(code.encode() + b"\n")
    return h.hexdigest()[:16]


def profile_key(workload, exact=False):
    """Name under which a workload's profiles are kept (the exact library's get a suffix)."""
    return workload + ("_exact" if exact else "")


def measured_traffic(workload, exact=False):
    """HBM bytes per splice from committed rocprofv3 counter runs, if they were taken on the
    current kernel source (else None)."""
    path = os.path.join(PROFILES, f"traffic_{profile_key(workload, exact)}.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        t = json.load(f)
    if t.get("kernel_sha") != kernel_sha():
        return None
    return t


def row_bytes(wl):
    esz = 2 if wl.dtype == "bf16" else 4
    return sum(p.row_elems for p in wl.planes) * esz


def contig_bytes(wl):
    """Algorithmic bytes of one contiguous splice: every moved row read and written once, every
    replacement row read once and written once (deleted rows cost nothing)."""
    n = wl.seq_lens[0]
    rb = row_bytes(wl)
    shift, moved, stub = 0, 0, 0
    for j, d in enumerate(wl.dirs):
        shift += d.stub_len - (d.span_end - d.span_start)
        seg_end = wl.dirs[j + 1].span_start if j + 1 < len(wl.dirs) else n
        if shift != 0:
            moved += seg_end - d.span_end
        stub += d.stub_len
    return 2 * (moved + stub) * rb * wl.n_layers, moved


def rotate_bytes(wl):
    """Algorithmic bytes of one in-place re-anchoring: every rotary band of the listed rows read
    and written once."""
    esz = 2 if wl.dtype == "bf16" else 4
    _, _, n = wl.rotate
    band = sum(p.rot_dim * p.n_heads for p in wl.planes) * esz
    return 2 * n * band * wl.n_layers, n


def paged_bytes(wl, kinds, new_lens, bt_stride, L):
    """Algorithmic bytes of one paged splice from the library's page plan (kinds per page of each
    sequence): every row gathered into a fresh page read and written once (downstream rows,
    replacement rows and the prefix rows that share a page with them), and the rotary bands of
    remapped pages read and written once."""
    rb = row_bytes(wl)
    esz = 2 if wl.dtype == "bf16" else 4
    rot_b = sum(p.rot_dim * p.n_heads for p in wl.planes) * esz
    asm_rows = remap_rows = moved = 0
    P = wl.page_size
    for b, n_new in enumerate(new_lens):
        for k in range(bt_stride):
            kind = kinds[b * bt_stride + k]
            rows = max(0, min(P, n_new - k * P))
            if kind == L.PAGE_ASSEMBLE:
                asm_rows += rows
            elif kind == L.PAGE_REMAP:
                remap_rows += rows
    for b, n in enumerate(wl.seq_lens):
        shift = 0
        mine = [d for d in wl.dirs if d.seq == b]
        for j, d in enumerate(mine):
            shift += d.stub_len - (d.span_end - d.span_start)
            seg_end = mine[j + 1].span_start if j + 1 < len(mine) else n
            if shift != 0:
                moved += seg_end - d.span_end
    return 2 * wl.n_layers * (asm_rows * rb + remap_rows * rot_b), moved, PAGED_KERNEL


COPY_CAP = 1 << 31          # bytes per side of the reference / calibration copy


def copy_half(nbytes):
    return min(nbytes // 2, COPY_CAP)


def copy_ceiling(nbytes, dev, stream):
    """Device-to-device copy of min(nbytes/2, 2 GiB) bytes with torch, once untimed and ten times
    timed: a reference rate, and the calibration kernel for the rocprofv3 byte counters."""
    import torch
    half = copy_half(nbytes)
    a = torch.empty(half, dtype=torch.uint8, device=dev)
    b = torch.empty(half, dtype=torch.uint8, device=dev)
    b.copy_(a)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(10):
        b.copy_(a)
    e1.record(stream)
    torch.cuda.synchronize()
    return 2 * half * 10 / (e0.elapsed_time(e1) * 1e-3) / 1e9, half


def setup_workload(wl, dev, L, W, args, stream):
    """(step, kernel, algorithmic bytes, moved tokens, dominant-kernel launches, keep, layout)."""
    specs = lambda planes: [L.PlaneSpec(t, p.n_heads, p.head_stride or p.row_elems, p.rot_offset,
                                        p.rot_dim, p.style, p.base) for p, t in zip(wl.planes, planes)]
    if wl.rotate:
        step, kernel, alg_bytes, moved, launches, keep = setup_rotate(wl, dev, L, W, specs, stream)
        layout = (("token slots listed by physical slot" if wl.page_size else "contiguous")
                  + f", rotary bands re-anchored in place (no movement), {ROTATE_REPLICAS} cache copies round-robin")
    elif wl.page_size:
        step, kernel, alg_bytes, moved, launches, keep = setup_paged(wl, dev, L, W, specs, stream)
        layout = (f"paged, {wl.page_size}-token pages, {len(wl.seq_lens)} sequences"
                  + (", copy-on-write" if wl.paged_flags else "")
                  + (f", {keep['replicas']} pool copies round-robin" if keep["replicas"] > 1 else ""))
    else:
        step, kernel, alg_bytes, moved, launches, keep = setup_contig(wl, dev, L, W, specs, stream, args)
        layout = "contiguous in place"
    return step, kernel, alg_bytes, moved, launches, keep, layout


GRAPH_SPLICES = 4     # splices per captured graph (cycling the cache copies)


def graph_step(step):
    """A step function that replays a HIP graph holding GRAPH_SPLICES consecutive splices, one
    splice per call: replay k runs on call k * GRAPH_SPLICES (the others enqueue nothing)."""
    import torch
    g = torch.cuda.CUDAGraph()
    for i in range(GRAPH_SPLICES):      # eager warm-up: workspaces and plans allocated outside the capture
        step(i)
    torch.cuda.synchronize()
    with torch.cuda.graph(g, stream=torch.cuda.Stream()):
        for i in range(GRAPH_SPLICES):
            step(i)
    torch.cuda.synchronize()

    def replayed(i):
        if i % GRAPH_SPLICES == 0:
            g.replay()
    replayed.graph = g
    return replayed


def timed(step, steps, warmup, stream):
    """Milliseconds per step: `warmup` untimed steps, then `steps` steps back to back on the
    stream the kernels run on, bracketed by two HIP events and nothing in between (an event
    between splices adds its own packet)."""
    import torch
    for i in range(warmup):
        step(i)
    torch.cuda.synchronize()
    t_begin = torch.cuda.Event(enable_timing=True)
    t_end = torch.cuda.Event(enable_timing=True)
    t_begin.record(stream)
    for i in range(steps):
        step(i)
    t_end.record(stream)
    torch.cuda.synchronize()
    return t_begin.elapsed_time(t_end) / steps


def roofline_of(wl, kernel, alg_bytes, launches, splice_ms, exact=False):
    """The dominant kernel against the HBM peak: algorithmic bytes per launch over the average
    launch duration (the event-timed splice divided by its launches of that kernel), with the
    committed counter traffic when it was taken on the current kernel sources."""
    achieved = alg_bytes / (splice_ms * 1e-3) / 1e9
    rec = measured_traffic(wl.name, exact)
    traffic = rec["dispatch_bytes"] if rec and rec.get("kernel") == kernel else None
    return achieved, traffic, rec


def measure_also(spec, args, dev, L, W, stream):
    """A further configuration timed in the same run (same protocol as the headline), reported as
    a compact record.  spec: a workload name, with ":exact" for libleyline_exact.so (fp64 pair
    arithmetic, results bit-identical to the oracle) instead of libleyline.so."""
    import torch
    name, _, variant = spec.partition(":")
    exact = variant == "exact"
    wl = W.WORKLOADS[name]()
    L.use_library(exact)
    try:
        step, kernel, alg_bytes, moved, launches, keep, layout = setup_workload(wl, dev, L, W, args, stream)
        ms = timed(step, args.steps, args.warmup, stream)
        pair_bits = L.leyline_pair_bits()
        del step, keep
        torch.cuda.synchronize()
    finally:
        L.use_library(False)
    torch.cuda.empty_cache()
    achieved, traffic, _ = roofline_of(wl, kernel, alg_bytes, launches, ms, exact)
    return {
        "workload": wl.name,
        "pair_bits": pair_bits,
        "layout": layout,
        "ms_per_step": ms,
        "value": moved / (ms * 1e-3),
        "unit": "tokens/s",
        "kernel": kernel,
        "launches_per_splice": launches,
        "avg_launch_ms": ms / max(1, launches),
        "achieved_GBps": achieved,
        "frac": achieved / PEAK_HBM_GBPS,
        "traffic": traffic,
        "algorithmic_bytes_per_splice": alg_bytes,
        "steps": args.steps,
        "warmup": args.warmup,
    }


def main():
    args = parse()
    if args.summarize:
        summarize(args)
        return
    if args.counters:
        summarize_counters(args)
        return
    if args.cpu_leg:
        cpu_leg(*args.cpu_leg)
        return
    if args.gpus != 1:
        print(json.dumps({"error": "this benchmark runs on one GPU only: a splice of one sequence "
                                   "or one batch is a single-GPU operation", "n_gpus": args.gpus}))
        sys.exit(2)

    import torch
    import workloads as W
    from paper_2606_01065_amd import leyline as L

    wl = W.WORKLOADS[args.workload]()
    dev = "cuda:0"
    torch.cuda.set_device(0)
    stream = torch.cuda.current_stream()
    L.use_library(args.exact)
    if args.graph and wl.page_size and not wl.rotate:
        raise SystemExit("--graph: paged splices with uploaded plans cannot be captured")
    # graph mode: the calls take the stream that is current when they run (the capture stream)
    step, kernel, alg_bytes, moved, launches, keep, layout = setup_workload(
        wl, dev, L, W, args, None if args.graph else stream)
    if args.graph:
        step = graph_step(step)
        layout += f", {GRAPH_SPLICES} splices captured in one HIP graph, replayed"

    ms_per_step = timed(step, args.steps, args.warmup, stream)
    splice_ms = ms_per_step
    achieved, traffic, rec = roofline_of(wl, kernel, alg_bytes, launches, splice_ms, args.exact)
    # Spread of single splices, from a separate untimed pass with an event pair around each.
    n_spread = min(args.steps, 20)
    starts = [torch.cuda.Event(enable_timing=True) for _ in range(n_spread)]
    ends = [torch.cuda.Event(enable_timing=True) for _ in range(n_spread)]
    for i in range(n_spread):
        starts[i].record(stream)
        if args.graph:
            step.graph.replay()                 # GRAPH_SPLICES splices
        else:
            step(args.steps + i)
        ends[i].record(stream)
    torch.cuda.synchronize()
    per_splice = np.array([s.elapsed_time(e) for s, e in zip(starts, ends)]) / (GRAPH_SPLICES if args.graph else 1)
    copy_gbps, _ = copy_ceiling(alg_bytes, dev, stream)
    out = {
        "metric": METRIC,
        "value": moved / (ms_per_step * 1e-3),
        "unit": "tokens/s",
        "token_layer_rows_per_s": moved * wl.n_layers / (ms_per_step * 1e-3),
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": wl.dtype,
        "data": "synthetic (seeded N(0,1) cache and replacement rows)",
        "config": {
            "workload": wl.name,
            "layers": wl.n_layers,
            "seq_lens": wl.seq_lens if len(wl.seq_lens) <= 4 else f"{len(wl.seq_lens)} sequences, "
                        f"{sum(wl.seq_lens)} tokens",
            "directives": [[d.seq, d.span_start, d.span_end, d.stub_len] for d in wl.dirs][:8],
            "moved_tokens": moved,
            "layout": layout,
            "pair_bits": L.leyline_pair_bits(),
            "graph": bool(args.graph),
            **({"rotate_delta_row0_rows": list(wl.rotate)} if wl.rotate else {}),
        },
        "roofline": {
            "bound": "hbm",
            "kernel": kernel,
            "achieved": achieved,
            "peak": PEAK_HBM_GBPS,
            "unit": "GB/s",
            "frac": achieved / PEAK_HBM_GBPS,
            "traffic": traffic,
            "traffic_unit": "HBM bytes per launch (rocprofv3 FETCH_SIZE + WRITE_SIZE, calibrated)",
            "algorithmic_bytes_per_launch": alg_bytes / max(1, launches),
            "algorithmic_bytes_per_splice": alg_bytes,
            "traffic_per_splice": None if rec is None else {k: rec[k] for k in ("fetch_bytes", "write_bytes", "total_bytes")},
            "splice_ms": splice_ms,
            "splice_ms_p10_p50_p90": [float(x) for x in np.percentile(per_splice, [10, 50, 90])],
            "splice_spread_sample": (f"{n_spread} graph replays of {GRAPH_SPLICES} splices after the timed region, "
                                     "an event pair around each, per splice" if args.graph else
                                     f"{n_spread} splices after the timed region, an event pair around each"),
            "launches_per_splice": launches,
            "avg_launch_ms": splice_ms / max(1, launches),
            "d2d_copy_GBps": copy_gbps,
            "kernel_sha": kernel_sha(),
        },
    }
    del step
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    L.use_library(False)
    this = profile_key(wl.name, args.exact).replace("_exact", ":exact")
    also = [a for a in args.also.split(",") if a and a != this]
    if also:
        out["also"] = [measure_also(a, args, dev, L, W, stream) for a in also]
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(wl, keep, args.cpu_seconds, moved, args.cpu_procs)
    print(json.dumps(out), flush=True)


def setup_contig(wl, dev, L, W, specs, stream, args):
    import torch
    base_planes, stubs = W.alloc_contig(wl, dev)
    replicas = [base_planes] + [[t.clone() for t in base_planes] for _ in range(1, args.replicas)]
    caches = [L.make_cache(specs(r)) for r in replicas]
    dirs = L.make_directives([dict(span_start=d.span_start, span_end=d.span_end, stub=stubs[j],
                                   stub_len=d.stub_len) for j, d in enumerate(wl.dirs)])
    n, nd = wl.seq_lens[0], len(wl.dirs)
    q = L.leyline_contig_query(caches[0], n, dirs, nd)
    ws = torch.empty(q.workspace_bytes, dtype=torch.uint8, device=dev) if q.workspace_bytes else None
    alg_bytes, moved = contig_bytes(wl)
    # the kernel that carries most of the bytes: ordered tiles when the plan has them
    kernel, launches = (CONTIG_TILE_KERNEL, q.tile_launches) if q.tile_launches else (CONTIG_KERNEL, q.launches)

    def step(i):
        L.leyline_splice_contig(caches[i % len(caches)], n, dirs, nd, stream, workspace=ws)

    # pristine host copy of the first layers for the CPU baseline (before any step runs)
    keep = dict(planes=[t[:8].cpu() for t in base_planes], stubs=[[s[:8].cpu() for s in per] for per in stubs])
    torch.cuda.synchronize()
    return step, kernel, alg_bytes, moved, launches, keep


def setup_rotate(wl, dev, L, W, specs, stream):
    import torch
    delta, row0, n = wl.rotate
    if wl.page_size:
        # a token-slot (paged) cache: the rows are the physical slots of logical rows
        # [row0, row0 + n) of the sequence, listed
        pools, bt, _, _ = W.alloc_paged(wl, dev)
        replicas = [pools] + [[t.clone() for t in pools] for _ in range(1, ROTATE_REPLICAS)]
        caches = [L.make_cache(specs(r), paged=True) for r in replicas]
        idx = torch.arange(row0, row0 + n, device=dev)
        rows = (bt[0].long()[idx // wl.page_size] * wl.page_size + idx % wl.page_size).contiguous()
    else:
        base_planes, _ = W.alloc_contig(wl, dev)
        replicas = [base_planes] + [[t.clone() for t in base_planes] for _ in range(1, ROTATE_REPLICAS)]
        caches = [L.make_cache(specs(r)) for r in replicas]
        rows = None
    alg_bytes, moved = rotate_bytes(wl)
    launches = 1                                  # every rotary plane in one launch

    def step(i):
        if rows is None:
            L.leyline_rotate_delta(caches[i % len(caches)], delta, row0=row0, n_rows=n, stream=stream)
        else:
            L.leyline_rotate_delta(caches[i % len(caches)], delta, rows=rows, stream=stream)

    torch.cuda.synchronize()
    return step, ROTATE_KERNEL, alg_bytes, moved, launches, dict(rotate=True)


def setup_paged(wl, dev, L, W, specs, stream):
    import torch
    pools, bt, free, stubs = W.alloc_paged(wl, dev)
    # Copies of the pool used in turn (same tables), so that a splice whose data would fit the
    # last-level cache does not find the previous step's rows there; as many as fit in 40 GB.
    pool_bytes = sum(p.numel() * p.element_size() for p in pools)
    n_rep = max(1, min(PAGED_REPLICAS, int(40e9 // pool_bytes)))
    copies = [pools] + [[p.clone() for p in pools] for _ in range(1, n_rep)]
    caches = [L.make_cache(specs(c), paged=True) for c in copies]
    cache = caches[0]
    dirs = L.make_directives([dict(span_start=d.span_start, span_end=d.span_end, stub=stubs[j],
                                   seq=d.seq, stub_len=d.stub_len) for j, d in enumerate(wl.dirs)])
    nd = len(wl.dirs)
    bt_stride = bt.shape[1]
    fl = wl.paged_flags
    new_lens, fresh, n_freed, ws_bytes = L.leyline_paged_query(cache, wl.seq_lens, bt_stride, dirs, nd, fl)
    bt_out = torch.empty_like(bt)
    freed = torch.empty(max(1, n_freed), dtype=torch.int32, device=dev)
    ws = torch.empty(max(256, ws_bytes), dtype=torch.uint8, device=dev)
    kinds, _, _, _ = L.leyline_paged_plan(wl.page_size, wl.seq_lens, dirs, nd, bt_stride, max(1, n_freed), fl)
    alg_bytes, moved, kernel = paged_bytes(wl, kinds, new_lens, bt_stride, L)

    # The paged splice reads old pages and writes fresh ones; re-running it on the same inputs
    # repeats the same work (remapped pages are rotated again, which does not change the bytes).
    def step(i):
        L.leyline_splice_paged(caches[i % n_rep], wl.seq_lens, bt, bt_out, dirs, nd, free, freed, ws,
                               stream=stream, flags=fl)

    keep = dict(paged=True, replicas=n_rep)
    torch.cuda.synchronize()
    # one data launch per splice (gather of assembled pages and in-place rotation of remapped
    # ones) carries the bytes; the order and resolve launches of large gathers are inside the
    # timed splice
    return step, kernel, alg_bytes, moved, 1, keep


def _cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return None


def _oracle_inputs(meta):
    from oracle import splice_oracle as O
    dirs = [O.Directive(*d) for d in meta["dirs"]]
    planes = [O.Plane(**p) for p in meta["planes"]]
    return O, dirs, planes


def _leg_work(arg):
    """One worker of the all-cores leg: splices the sample's layers (worker i takes layers i,
    i + procs, ... cyclically) with the oracle until `seconds` have passed; returns the count."""
    data, i, procs, seconds = arg
    with open(os.path.join(data, "meta.json")) as f:
        meta = json.load(f)
    O, dirs, planes = _oracle_inputs(meta)
    rows = [np.load(os.path.join(data, f"plane_{pi}.npy"), mmap_mode="r") for pi in range(len(planes))]
    stubs = [[np.load(os.path.join(data, f"stub_{j}_{pi}.npy"), mmap_mode="r") for pi in range(len(planes))]
             for j in range(len(dirs))]
    n_keep, done = rows[0].shape[0], 0
    t0 = time.perf_counter()
    while time.perf_counter() - t0 < seconds:
        l = (i + done * procs) % n_keep
        for pi, plane in enumerate(planes):
            O.splice_rows(np.asarray(rows[pi][l]), meta["n"], dirs, [np.asarray(st[pi][l]) for st in stubs],
                          plane, meta["dtype"])
        done += 1
    return done


def cpu_leg(data, seconds, procs, out):
    """The all-cores leg, in a child process that touches no GPU: `procs` forked workers run
    _leg_work at once; writes the layer-splices done and the wall time."""
    import multiprocessing as mp
    procs = int(procs)
    with mp.get_context("fork").Pool(procs) as pool:
        t0 = time.perf_counter()
        done = pool.map(_leg_work, [(data, i, procs, float(seconds)) for i in range(procs)])
        wall = time.perf_counter() - t0
    with open(out, "w") as f:
        json.dump({"layer_splices": int(sum(done)), "wall_s": wall, "procs": procs}, f)


def _host_cpus():
    """CPUs this process may run on (its CPU affinity set)."""
    try:
        return len(os.sched_getaffinity(0))
    except AttributeError:
        return os.cpu_count() or 1


def cpu_baseline(wl, keep, budget_s, moved, procs=0):
    """The oracle, as it stands, on a bounded sample of the same splice: whole layers of the
    headline cache (host copies taken before the first step), scaled to all layers.  Two legs:
    one thread (numpy, single-threaded here), cycling over the sample's layers for about
    budget_s seconds; and all host cores, `procs` processes (default: every CPU this process may
    use, at most 16) splicing different layers at once for about the same time, in a child
    process started for it."""
    import shutil
    import subprocess
    import tempfile

    import torch
    from oracle import splice_oracle as O
    if keep.get("paged") or keep.get("rotate"):
        return None

    def host(t):
        return t.view(torch.int16).numpy().view(np.uint16) if t.dtype == torch.bfloat16 else t.numpy()

    n = wl.seq_lens[0]
    meta = {"n": n, "dtype": wl.dtype, "n_layers": wl.n_layers,
            "dirs": [[d.span_start, d.span_end, d.stub_len] for d in wl.dirs],
            "planes": [dict(row_elems=p.row_elems, n_heads=p.n_heads, head_stride=p.head_stride or p.row_elems,
                            rot_offset=p.rot_offset, rot_dim=p.rot_dim, style=p.style, base=p.base)
                       for p in wl.planes]}
    _, dirs, planes = _oracle_inputs(meta)
    n_keep = keep["planes"][0].shape[0]
    rows = [[host(t[l]).reshape(t.shape[1], -1) for t in keep["planes"]] for l in range(n_keep)]
    stubs = [[[host(s[l]).reshape(s.shape[1], -1) for s in per] for per in keep["stubs"]] for l in range(n_keep)]
    done, spent = 0, 0.0
    while spent < budget_s:
        l = done % n_keep
        t0 = time.perf_counter()
        for pi, plane in enumerate(planes):
            O.splice_rows(rows[l][pi], n, dirs, [s[pi] for s in stubs[l]], plane, wl.dtype)
        spent += time.perf_counter() - t0
        done += 1
    per_layer = spent / done
    full_s = per_layer * wl.n_layers
    out = {
        "value": moved / full_s,
        "unit": "tokens/s",
        "cores": 1,
        "host_cpus": _host_cpus(),
        "host_cpu_model": _cpu_model(),
        "kind": "oracle",
        "sample": f"{done} layer-splices of this workload (numpy fp64, one thread, layers cycled "
                  f"over {n_keep} host-resident layers), {spent:.1f} s; scaled to {wl.n_layers} "
                  f"layers: {full_s:.3f} s per splice",
    }
    # all host cores: the same oracle in `procs` processes at once, each on its own layers
    procs = procs or min(16, _host_cpus())
    tmp = tempfile.mkdtemp(prefix="leyline_cpu_leg_")
    try:
        for pi in range(len(planes)):
            np.save(os.path.join(tmp, f"plane_{pi}.npy"), np.stack([rows[l][pi] for l in range(n_keep)]))
            for j in range(len(dirs)):
                np.save(os.path.join(tmp, f"stub_{j}_{pi}.npy"), np.stack([stubs[l][j][pi] for l in range(n_keep)]))
        with open(os.path.join(tmp, "meta.json"), "w") as f:
            json.dump(meta, f)
        res = os.path.join(tmp, "leg.json")
        env = dict(os.environ, OMP_NUM_THREADS="1", OPENBLAS_NUM_THREADS="1", MKL_NUM_THREADS="1")
        subprocess.run([sys.executable, os.path.abspath(__file__), "--cpu-leg", tmp, str(budget_s), str(procs), res],
                       check=True, env=env, timeout=budget_s * 4 + 120)
        with open(res) as f:
            leg = json.load(f)
    finally:
        shutil.rmtree(tmp, ignore_errors=True)
    splices = leg["layer_splices"] / wl.n_layers
    out["all_cores"] = {
        "value": moved * splices / leg["wall_s"],
        "unit": "tokens/s",
        "cores": leg["procs"],
        "sample": f"{leg['layer_splices']} layer-splices in {leg['procs']} processes at once (one numpy "
                  f"thread each, every process cycling over its share of the same {n_keep} layers) in "
                  f"{leg['wall_s']:.1f} s of wall time; {wl.n_layers} layer-splices make one splice",
    }
    return out


# ---------------------------------------------------------------------- profile summaries ---

def _read_csv(d, name):
    hits = glob.glob(os.path.join(d, "**", f"*{name}*.csv"), recursive=True)
    if not hits:
        raise SystemExit(f"no *{name}*.csv under {d}")
    with open(hits[0]) as f:
        return list(csv.DictReader(f))


def _counter_per_dispatch(rows, counter, match, after=-1):
    """Counter value per dispatch of the kernels `match` accepts, for dispatch ids > after."""
    vals = {}
    for r in rows:
        did = int(r.get("Dispatch_Id") or r.get("Correlation_Id"))
        if did > after and match(r.get("Kernel_Name", "")) and r.get("Counter_Name") == counter:
            vals[did] = vals.get(did, 0.0) + float(r["Counter_Value"])
    return [vals[k] for k in sorted(vals)]


def _last_dispatch(rows, match):
    ids = [int(r.get("Dispatch_Id") or r.get("Correlation_Id")) for r in rows if match(r.get("Kernel_Name", ""))]
    return max(ids) if ids else -1


def _profiled_sha(trace_dir):
    """kernel_sha printed by the profiled bench run (its output sits in <trace_dir>.log)."""
    log = trace_dir.rstrip("/") + ".log"
    if os.path.exists(log):
        for line in open(log):
            if line.startswith("{") and '"kernel_sha"' in line:
                return json.loads(line)["roofline"]["kernel_sha"]
    raise SystemExit(f"no bench JSON line with kernel_sha in {log}")


def _flag(cmd, name, default):
    parts = cmd.split()
    return int(parts[parts.index(name) + 1]) if name in parts else default


def summarize(args):
    """Turn rocprofv3 output (a --kernel-trace --stats run and two --pmc runs, FETCH_SIZE and
    WRITE_SIZE, of the same bench command, recorded in --command) into
    profiles/<kernel>_<workload>.md and the traffic record bench.py reports."""
    trace_dir, fetch_dir, write_dir = args.summarize
    import workloads as W
    wl = W.WORKLOADS[args.workload]()
    if wl.rotate:
        alg, _ = rotate_bytes(wl)
        kernel = ROTATE_KERNEL
    elif wl.page_size:
        from paper_2606_01065_amd import leyline as L
        bt_stride = W.paged_bt_stride(wl)
        dirs = L.make_directives([dict(span_start=d.span_start, span_end=d.span_end, seq=d.seq,
                                       stub_len=d.stub_len, stub=None) for d in wl.dirs])
        new_lens = W.paged_new_lens(wl)
        kinds, _, _, _ = L.leyline_paged_plan(wl.page_size, wl.seq_lens, dirs, len(wl.dirs), bt_stride,
                                              sum(-(-n // wl.page_size) for n in wl.seq_lens),
                                              wl.paged_flags)
        alg, _, kernel = paged_bytes(wl, kinds, new_lens, bt_stride, L)
    else:
        alg, _ = contig_bytes(wl)
        kernel = CONTIG_KERNEL
    steps = _flag(args.command, "--steps", 100)
    # warmup, timed steps, then the spread pass of up to 20 single splices
    splices = steps + _flag(args.command, "--warmup", 10) + min(steps, 20)
    stats = _read_csv(trace_dir, "kernel_stats")
    trace = _read_csv(trace_dir, "kernel_trace")
    if not wl.page_size and not wl.rotate:
        # the contiguous kernel that took the most time (rounds, or ordered tiles)
        best = max((r for r in stats if CONTIG_KERNEL in r["Name"] or CONTIG_TILE_KERNEL in r["Name"]),
                   key=lambda r: float(r["TotalDurationNs"]), default=None)
        if best is not None and CONTIG_TILE_KERNEL in best["Name"]:
            kernel = CONTIG_TILE_KERNEL
    durs = [(int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3 for r in trace
            if kernel in r["Kernel_Name"]]
    fetch = _read_csv(fetch_dir, "counter_collection")
    write = _read_csv(write_dir, "counter_collection")
    is_k = lambda name: kernel in name
    is_lib = lambda name: "leyline::" in name
    is_copy = lambda name: "leyline" not in name and ("copyBuffer" in name or "copy" in name.lower())
    f_k = _counter_per_dispatch(fetch, "FETCH_SIZE", is_k)
    w_k = _counter_per_dispatch(write, "WRITE_SIZE", is_k)
    f_all = _counter_per_dispatch(fetch, "FETCH_SIZE", is_lib)      # every library kernel of the splice
    w_all = _counter_per_dispatch(write, "WRITE_SIZE", is_lib)
    # calibration copies: the device copies the bench issues after its last splice
    f_c = _counter_per_dispatch(fetch, "FETCH_SIZE", is_copy, _last_dispatch(fetch, is_k))
    w_c = _counter_per_dispatch(write, "WRITE_SIZE", is_copy, _last_dispatch(write, is_k))
    # calibration: the bench's 11 device copies each read and write copy_half(alg) bytes
    half = copy_half(alg)
    cal_f = (11 * half / (sum(f_c) * 1024)) if (half and f_c) else None
    cal_w = (11 * half / (sum(w_c) * 1024)) if (half and w_c) else None
    per_splice = len(durs) / splices if splices else 0
    lines = [f"# {kernel} on {wl.name}", "", f"Command: `{args.command}`", "",
             "## Kernel time (rocprofv3 --kernel-trace --stats)", "",
             "| kernel | calls | avg us | total us |", "|---|---|---|---|"]
    for r in stats:
        nm = r["Name"]
        if "leyline" in nm or is_copy(nm):
            lines.append(f"| {nm[:90]} | {r['Calls']} | {float(r['AverageNs'])/1e3:.1f} | "
                         f"{float(r['TotalDurationNs'])/1e3:.1f} |")
    lines += ["", f"{kernel}: {len(durs)} dispatches for {splices} splices "
              f"({per_splice:.1f} per splice); mean {np.mean(durs):.1f} us per dispatch; "
              f"{np.sum(durs) / splices:.1f} us of kernel time per splice", "",
              "## HBM bytes (rocprofv3 --pmc FETCH_SIZE, then --pmc WRITE_SIZE; KiB per dispatch)", "",
              f"{kernel}: FETCH_SIZE mean {np.mean(f_k):.0f} KiB over {len(f_k)} dispatches; "
              f"WRITE_SIZE mean {np.mean(w_k):.0f} KiB over {len(w_k)} dispatches"]
    rec = None
    if f_c and w_c and half:
        lines.append(f"device copy after the last splice (calibration; 11 copies of {half} B each "
                     f"way, {len(f_c)} / {len(w_c)} dispatches): FETCH_SIZE {sum(f_c):.0f} KiB, "
                     f"WRITE_SIZE {sum(w_c):.0f} KiB in total -> bytes per counted byte "
                     f"{cal_f:.3f} (fetch), {cal_w:.3f} (write)")
        fetch_b = sum(f_all) * 1024 * cal_f / splices
        write_b = sum(w_all) * 1024 * cal_w / splices
        dom_b = (sum(f_k) * cal_f + sum(w_k) * cal_w) * 1024 / splices
        lines.append(f"per splice, all library kernels: fetched {fetch_b/1e9:.4f} GB, written "
                     f"{write_b/1e9:.4f} GB; algorithmic {alg/1e9:.4f} GB; measured/algorithmic "
                     f"{(fetch_b + write_b)/alg:.3f}; {kernel} alone {dom_b/1e9:.4f} GB "
                     f"({100 * dom_b / (fetch_b + write_b):.1f}%)")
        rec = dict(kernel_sha=_profiled_sha(trace_dir), workload=wl.name, kernel=kernel,
                   dispatch_bytes=(np.mean(f_k) * cal_f + np.mean(w_k) * cal_w) * 1024,
                   dispatches_per_splice=per_splice, fetch_bytes=fetch_b, write_bytes=write_b,
                   total_bytes=fetch_b + write_b, calibration=[cal_f, cal_w], per="splice",
                   algorithmic_bytes=alg)
    os.makedirs(PROFILES, exist_ok=True)
    key = profile_key(wl.name, "--exact" in args.command.split())
    with open(os.path.join(PROFILES, f"{kernel}_{key}.md"), "w") as f:
        f.write("\n".join(lines) + "\n")
    if rec:
        with open(os.path.join(PROFILES, f"traffic_{key}.json"), "w") as f:
            json.dump(rec, f, indent=1)
    print("\n".join(lines))


def summarize_counters(args):
    """Mean value per dispatch of every counter in rocprofv3 --pmc runs (one directory per run) for
    the workload's dominant library kernel, and per KiB of the splice's algorithmic bytes moved
    by that kernel per dispatch."""
    import workloads as W
    wl = W.WORKLOADS[args.workload]()
    kernel = ROTATE_KERNEL if wl.rotate else PAGED_KERNEL if wl.page_size else None
    rows = []
    for d in args.counters:
        data = _read_csv(d, "counter_collection")
        names = sorted({r["Counter_Name"] for r in data})
        if kernel is None:     # contiguous: the library kernel with the most dispatches
            counts = {}
            for r in data:
                if "leyline::" in r.get("Kernel_Name", ""):
                    counts[r["Kernel_Name"]] = counts.get(r["Kernel_Name"], 0) + 1
            top = max(counts, key=counts.get)
            kernel = CONTIG_TILE_KERNEL if CONTIG_TILE_KERNEL in top else CONTIG_KERNEL
        for n in names:
            vals = _counter_per_dispatch(data, n, lambda k: kernel in k)
            rows.append((n, len(vals), float(np.mean(vals)) if vals else float("nan")))
    lines = [f"# {kernel} on {wl.name}: counters", "", f"Command: `{args.command}`", "",
             "| counter | dispatches | mean per dispatch |", "|---|---|---|"]
    lines += [f"| {n} | {k} | {v:.4g} |" for n, k, v in rows]
    os.makedirs(PROFILES, exist_ok=True)
    with open(os.path.join(PROFILES, f"counters_{kernel}_{wl.name}.md"), "w") as f:
        f.write("\n".join(lines) + "\n")
    print("\n".join(lines))


if __name__ == "__main__":
    main()
