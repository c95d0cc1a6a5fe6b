"""The benchmark's byte accounting and its command-line contract (no GPU).

Algorithmic bytes follow the KV size of a token: (kv_lora_rank + rope_dim) elements per layer for
an MLA cache (the per-token KV formula of the section "Deployment-cell evidence at the policy
layer", paragraph on KV bytes attributable to the splice), K and V heads for GQA; a moved or
assembled row is read once and written once, a re-used page only has its rotary bands rewritten.
The paged accounting is checked against a count over the oracle's own page plan."""

import random
import subprocess
import sys
import json
import os

import pytest

import bench as B
import workloads as W
from oracle import splice_oracle as O
from paper_2606_01065_amd import leyline as L

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_mla_and_gqa_bytes_per_token():
    mla = W.mla_dsv3_32k()
    assert B.row_bytes(mla) == (512 + 64) * 2                    # 1152 B per token and layer
    alg, moved = B.contig_bytes(mla)
    d = mla.dirs[0]
    assert moved == 32768 - d.span_end
    assert alg == 2 * (moved + d.stub_len) * 1152 * 61
    assert 2 * 1152 * 61 == 140544                               # per moved token, all layers
    gqa = W.gqa_llama3_8b_16k()
    assert B.row_bytes(gqa) == 2 * 8 * 128 * 2                   # K and V rows
    alg, moved = B.contig_bytes(gqa)
    assert moved == 16384 - 6144 and alg == 2 * (moved + 24) * 4096 * 32
    assert 2 * 4096 * 32 == 262144


def test_multi_directive_bytes_skip_unshifted_segments():
    base = W.mla_dsv3_32k()
    # the second edit restores the first one's shift: the segment after it does not move
    dirs = [W.Dir(100, 110, 4), W.Dir(500, 504, 10), W.Dir(900, 910, 3)]
    wl = W.Workload("t", base.n_layers, base.dtype, base.planes, dirs, [2000], capacity=2100, seed=1)
    alg, moved = B.contig_bytes(wl)
    assert moved == (500 - 110) + (2000 - 910)                   # [504, 900) has shift 0
    assert alg == 2 * (moved + 4 + 10 + 3) * 1152 * 61


@pytest.mark.parametrize("page,cow", [(1, False), (4, False), (64, False), (4, True)])
def test_paged_bytes_match_a_count_over_the_oracle_plan(page, cow):
    rng = random.Random(page * 7 + cow)
    for _ in range(10):
        lens = [rng.randint(0, 700) for _ in range(rng.randint(1, 4))]
        dirs = []
        for b, n in enumerate(lens):
            cuts = sorted(rng.sample(range(n + 1), min(2 * rng.randint(0, 3), n + 1)))
            for i in range(0, len(cuts) - 1, 2):
                s, e = cuts[i], cuts[i + 1]
                dirs.append(W.Dir(s, e, rng.choice([0, e - s, rng.randint(0, 2 * (e - s) + 3), e - s + page]),
                                  seq=b))
        wl = W.Workload("t", 3, "bf16", [W.mla_plane()], dirs, lens, page_size=page, seed=1,
                        paged_flags=L.PAGED_COPY_ON_WRITE if cow else 0)
        odirs = [O.Directive(d.span_start, d.span_end, d.stub_len, seq=d.seq) for d in dirs]
        plans = O.plan_paged(lens, odirs, page, remap=not cow)
        bt_stride = max(max(O.pages_for(n, page), O.pages_for(p.new_len, page)) for n, p in zip(lens, plans)) + 1
        cdirs = L.make_directives([dict(span_start=d.span_start, span_end=d.span_end, seq=d.seq,
                                        stub_len=d.stub_len, stub=None) for d in dirs])
        kinds, _, _, _ = L.leyline_paged_plan(page, lens, cdirs, len(dirs), bt_stride,
                                              sum(O.pages_for(n, page) for n in lens) + 1, wl.paged_flags)
        alg, _, _ = B.paged_bytes(wl, kinds, [p.new_len for p in plans], bt_stride, L)
        want = 0
        for p in plans:
            for k, kind in enumerate(p.kinds):
                rows = min(page, p.new_len - k * page)
                if kind == O.ASSEMBLE:
                    want += rows * 1152
                elif kind == O.REMAP:
                    want += rows * 64 * 2
        assert alg == 2 * 3 * want


def test_more_than_one_gpu_is_refused_with_a_message():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2
    out = json.loads(r.stdout.strip().splitlines()[-1])
    assert out["n_gpus"] == 2 and "one GPU" in out["error"]
