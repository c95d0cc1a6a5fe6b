"""Benchmark of the in-place KV-cache splice on one MI355X.

One step = one splice call (delete the span, write the replacement, compact every downstream
row and re-anchor its rotary band, all layers) on the workload's synthetic cache, already
resident in HBM.  Prints one JSON line.

    python bench.py [--steps K] [--warmup W] [--workload NAME] [--gpus 1] [--no-cpu-baseline]

Default workload: MLA DeepSeek-V3 shape (61 layers, c_kv 512 + k_pe 64, bf16), one 32768-token
sequence, a 4096-token span at a seeded start replaced by a 32-token stub, contiguous in place.
"""

import argparse
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
KERNEL_SRC = os.path.join(ROOT, "paper_2606_01065_amd", "csrc", "kernels.hip")
TRAFFIC_DIR = os.path.join(ROOT, "profiles")


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default="mla_dsv3_32k")
    ap.add_argument("--replicas", type=int, default=2,
                    help="independent cache copies used round-robin, so consecutive steps do not "
                         "find each other's rows in the last-level cache")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=12.0)
    return ap.parse_args()


def kernel_sha():
    with open(KERNEL_SRC, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()[:16]


def measured_traffic(workload):
    """Per-launch HBM bytes from committed rocprofv3 counter runs, if they were taken on the
    current kernel source (else None)."""
    path = os.path.join(TRAFFIC_DIR, f"traffic_{workload}.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        t = json.load(f)
    if t.get("kernel_sha") != kernel_sha():
        return None
    return t.get("bytes_per_launch")


def contig_bytes(wl):
    """Algorithmic bytes of one contiguous splice: every moved row read and written once, every
    stub row read once and written once (deleted rows cost nothing)."""
    total = 0
    n = wl.seq_lens[0]
    esz = 2 if wl.dtype == "bf16" else 4
    row_bytes = sum(p.row_elems for p in wl.planes) * esz
    shift, moved = 0, 0
    for j, d in enumerate(wl.dirs):
        shift += d.stub_len - (d.span_end - d.span_start)
        seg_end = wl.dirs[j + 1].span_start if j + 1 < len(wl.dirs) else n
        if shift != 0:
            moved += seg_end - d.span_end
        total += 2 * d.stub_len * row_bytes * wl.n_layers
    total += 2 * moved * row_bytes * wl.n_layers
    return total, moved


def main():
    args = parse()
    if args.gpus != 1:
        print(json.dumps({"error": "this benchmark runs on one GPU only; the splice of one "
                                   "sequence (or one batch) is a single-GPU operation",
                          "n_gpus": args.gpus}))
        sys.exit(2)

    import torch
    import workloads as W
    from paper_2606_01065_amd import leyline as L

    wl = W.WORKLOADS[args.workload]()
    if wl.page_size:
        print(json.dumps({"error": "paged workloads are measured with --workload on the paged "
                                   "benchmark path, not implemented in this entry"}))
        sys.exit(2)
    dev = "cuda:0"
    torch.cuda.set_device(0)
    stream = torch.cuda.current_stream()

    replicas = []
    base_planes, stubs = W.alloc_contig(wl, dev)
    replicas.append(base_planes)
    for _ in range(1, args.replicas):
        replicas.append([t.clone() for t in base_planes])
    specs = lambda planes: [L.PlaneSpec(t, p.n_heads, p.head_stride or p.row_elems, p.rot_offset,
                                        p.rot_dim, p.style, p.base) for p, t in zip(wl.planes, planes)]
    caches = [L.make_cache(specs(r)) for r in replicas]
    dirs = L.make_directives([dict(span_start=d.span_start, span_end=d.span_end, stub=stubs[j],
                                   stub_len=d.stub_len) for j, d in enumerate(wl.dirs)])
    n = wl.seq_lens[0]
    nd = len(wl.dirs)

    for i in range(args.warmup):
        L.leyline_splice_contig(caches[i % len(caches)], n, dirs, nd, stream)
    torch.cuda.synchronize()

    starts = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps)]
    ends = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps)]
    t_begin = torch.cuda.Event(enable_timing=True)
    t_end = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t_begin.record(stream)
    for i in range(args.steps):
        starts[i].record(stream)
        L.leyline_splice_contig(caches[i % len(caches)], n, dirs, nd, stream)
        ends[i].record(stream)
    t_end.record(stream)
    torch.cuda.synchronize()
    total_ms = t_begin.elapsed_time(t_end)
    per_launch_ms = [s.elapsed_time(e) for s, e in zip(starts, ends)]
    avg_launch_ms = float(np.mean(per_launch_ms))

    alg_bytes, moved = contig_bytes(wl)
    achieved = alg_bytes / (avg_launch_ms * 1e-3) / 1e9
    ms_per_step = total_ms / args.steps
    value = moved / (ms_per_step * 1e-3)

    # device-to-device copy of the same number of bytes read (= written): the copy ceiling
    half = alg_bytes // 2
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
    copy_gbps = 2 * half * 10 / (e0.elapsed_time(e1) * 1e-3) / 1e9
    del a, b

    traffic = measured_traffic(wl.name)
    out = {
        "metric": METRIC,
        "value": value,
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": wl.dtype,
        "data": "synthetic (seeded N(0,1) cache and stub)",
        "config": {
            "workload": wl.name,
            "layers": wl.n_layers,
            "seq_len": n,
            "directives": [[d.span_start, d.span_end, d.stub_len] for d in wl.dirs],
            "moved_tokens": moved,
            "layout": "contiguous in place",
        },
        "roofline": {
            "bound": "hbm",
            "kernel": "contig_splice_kernel",
            "achieved": achieved,
            "peak": PEAK_HBM_GBPS,
            "unit": "GB/s",
            "frac": achieved / PEAK_HBM_GBPS,
            "traffic": traffic,
            "algorithmic_bytes": alg_bytes,
            "avg_launch_ms": avg_launch_ms,
            "d2d_copy_GBps": copy_gbps,
        },
    }

    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(wl, base_planes, stubs, args.cpu_seconds, moved, ms_per_step)
    print(json.dumps(out), flush=True)


def cpu_baseline(wl, planes_dev, stubs_dev, budget_s, moved, gpu_ms):
    """The oracle, as it stands, on a bounded sample: whole layers of the same splice, run one
    after another until about budget_s seconds have passed; scaled to all layers."""
    import torch
    from oracle import splice_oracle as O

    def host(t):
        t = t.detach().cpu()
        return t.view(torch.int16).numpy().view(np.uint16) if t.dtype == torch.bfloat16 else t.numpy()

    n = wl.seq_lens[0]
    dirs = [O.Directive(d.span_start, d.span_end, d.stub_len) for d in wl.dirs]
    planes = [O.Plane(row_elems=p.row_elems, n_heads=p.n_heads, head_stride=p.head_stride or p.row_elems,
                      rot_offset=p.rot_offset, rot_dim=p.rot_dim, style=p.style, base=p.base)
              for p in wl.planes]
    done, spent = 0, 0.0
    while done < wl.n_layers and spent < budget_s:
        rows = [host(t[done]).reshape(t.shape[1], -1) for t in planes_dev]
        stubs = [[host(s[done]).reshape(s.shape[1], -1) for s in per] for per in stubs_dev]
        t0 = time.perf_counter()
        for pi, plane in enumerate(planes):
            O.splice_rows(rows[pi], n, dirs, [s[pi] for s in stubs], plane, wl.dtype)
        spent += time.perf_counter() - t0
        done += 1
    per_layer = spent / done
    full_s = per_layer * wl.n_layers
    return {
        "value": moved / full_s,
        "unit": "tokens/s",
        "cores": 1,
        "kind": "oracle",
        "sample": f"{done} of {wl.n_layers} layers of the same splice (numpy fp64, one thread), "
                  f"{spent:.1f} s, scaled to all layers: {full_s:.2f} s per splice",
        "gpu_speedup": full_s / (gpu_ms * 1e-3),
    }


if __name__ == "__main__":
    main()
