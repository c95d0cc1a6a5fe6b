"""The benchmark's output contract: one JSON line with the fields the round driver reads, a
roofline object for the dominant kernel and, for the default workload, the oracle's CPU baseline."""

import json
import os
import subprocess
import sys

import pytest

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _bench(*args):
    print(f"[case] bench.py {' '.join(args)}", flush=True)
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), *args], capture_output=True, text=True,
                       timeout=300)
    assert r.returncode == 0, r.stderr[-3000:]
    return json.loads(r.stdout.strip().splitlines()[-1])


def _check_common(d, steps, warmup):
    for key in ("metric", "value", "unit", "n_gpus", "steps", "warmup", "ms_per_step", "higher_is_better",
                "scaling", "vs_baseline", "dtype", "data", "config", "roofline"):
        assert key in d, key
    assert d["n_gpus"] == 1 and d["steps"] == steps and d["warmup"] == warmup
    assert d["unit"] == "tokens/s" and d["higher_is_better"] is True and d["scaling"] == "weak"
    assert d["value"] > 0 and d["ms_per_step"] > 0
    assert abs(d["value"] - d["config"]["moved_tokens"] / (d["ms_per_step"] * 1e-3)) <= 1e-6 * d["value"]
    r = d["roofline"]
    assert r["bound"] == "hbm" and r["unit"] == "GB/s" and r["peak"] == 8000.0
    assert abs(r["frac"] - r["achieved"] / r["peak"]) < 1e-12
    assert abs(r["achieved"] - r["algorithmic_bytes_per_splice"] / (r["splice_ms"] * 1e-3) / 1e9) <= 1e-6 * r["achieved"]
    assert r["traffic"] is None or r["traffic"] > 0
    assert isinstance(d["config"]["workload"], str)


def test_default_run_reports_roofline_and_cpu_baseline():
    d = _bench("--steps", "3", "--warmup", "1", "--cpu-seconds", "1")
    _check_common(d, 3, 1)
    assert d["config"]["workload"] == "mla_dsv3_32k" and d["dtype"] == "bf16"
    c = d["cpu_baseline"]
    assert c["kind"] == "oracle" and c["unit"] == "tokens/s" and c["value"] > 0
    assert isinstance(c["cores"], int) and c["cores"] >= 1 and c["sample"]
    ac = c["all_cores"]        # the same oracle in one process per host core
    assert ac["unit"] == "tokens/s" and ac["value"] > 0 and ac["cores"] >= 1 and ac["sample"]
    # the GQA target configuration, the 8-directive paged splice and the 64-sequence paged batch,
    # timed in the same run
    also = {(a["workload"], a["pair_bits"]): a for a in d["also"]}
    assert set(also) == {("gqa_llama3_8b_16k", 32), ("mla_dsv3_paged_131k", 32), ("mla_dsv3_paged_b64", 32),
                         ("mla_dsv3_32k", 64), ("gqa_llama3_8b_16k", 64)}
    assert d["config"]["pair_bits"] == 32
    for a in also.values():
        assert a["ms_per_step"] > 0 and a["kernel"] and a["steps"] == 3
        assert a["value"] > 0 and a["unit"] == "tokens/s"
        assert abs(a["frac"] - a["achieved_GBps"] / 8000.0) < 1e-12
        assert abs(a["achieved_GBps"] - a["algorithmic_bytes_per_splice"] / (a["ms_per_step"] * 1e-3) / 1e9) \
            <= 1e-6 * a["achieved_GBps"]


def test_graph_replay_keeps_the_contract():
    """--graph: splices captured in a HIP graph and replayed (small-call latency without launch
    overhead), on the one-layer workload and on the 8-edit tile splice."""
    for workload in ("mla_1l_4k_f32", "mla_dsv3_32k_edits8"):
        d = _bench("--workload", workload, "--steps", "8", "--warmup", "4", "--no-cpu-baseline", "--also=", "--graph")
        _check_common(d, 8, 4)
        assert d["config"]["graph"] is True and "HIP graph" in d["config"]["layout"]


@pytest.mark.parametrize("workload", ["mla_dsv3_slots_32k", "gqa_llama3_8b_rotate_16k", "mla_dsv3_32k_edits8"])
def test_other_workloads_keep_the_contract(workload):
    d = _bench("--workload", workload, "--steps", "3", "--warmup", "1", "--no-cpu-baseline", "--also", "")
    _check_common(d, 3, 1)
    assert d["config"]["workload"] == workload and "cpu_baseline" not in d and "also" not in d
