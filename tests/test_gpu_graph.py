"""The contiguous splice and the in-place rotation enqueue kernels only, so a caller may capture
them into a HIP graph.  Each test runs the call eagerly, captures it, then replays the graph
several times, restoring the input eagerly between replays, and compares every replay with the
eager result bit for bit (same kernels, same inputs)."""

import numpy as np
import pytest
import torch

import workloads as W
from tests.parity_util import host

pytestmark = pytest.mark.gpu

DEV = "cuda:0"


@pytest.fixture(scope="module")
def L():
    from paper_2606_01065_amd import leyline
    return leyline


def _mla_cache(L, n_layers, capacity, seed):
    wl = W.Workload("graph", n_layers, "bf16", [W.mla_plane()], [], [capacity], capacity=capacity, seed=seed)
    planes, _ = W.alloc_contig(wl, DEV)
    t = planes[0]
    return t, L.make_cache([L.PlaneSpec(t, 1, 576, 512, 64, L.ROPE_INTERLEAVED, 10000.0)])


def _replay_and_compare(fn, t, pristine, eager):
    stream = torch.cuda.Stream()
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    t.copy_(pristine)
    torch.cuda.synchronize()
    with torch.cuda.graph(g, stream=stream):
        fn()
    torch.cuda.synchronize()
    for rep in range(3):
        t.copy_(pristine)                      # eager work between replays
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert np.array_equal(host(t), eager), f"replay {rep} differs from the eager call"


@pytest.mark.parametrize("layers,n,edits,tiles", [
    (3, 3000, [(500, 501, 0)], 1),                        # shift -1: prep + one tile launch
    (20, 12000, [(1000, 5000, 16)], 0),                   # shift -3984, 92 MB rounds + stub copy
    (3, 3000, [(100, 104, 1), (700, 700, 2), (1500, 1530, 25), (2900, 2950, 0)], 1),  # edits in one tile launch
])
def test_contig_splice_in_a_graph(L, layers, n, edits, tiles):
    cap = n + 8
    t, cache = _mla_cache(L, layers, cap, seed=31)
    pristine = t.clone()
    stubs = [torch.randn((layers, r, 576), device=DEV).to(torch.bfloat16) if r else None for _, _, r in edits]
    dirs = L.make_directives([dict(span_start=s, span_end=e, stub=[stubs[j]] if stubs[j] is not None else None,
                                   stub_len=r) for j, (s, e, r) in enumerate(edits)])
    k = len(edits)
    q = L.leyline_contig_query(cache, n, dirs, k)
    assert q.tile_launches == tiles
    ws = torch.empty(max(256, q.workspace_bytes), dtype=torch.uint8, device=DEV)
    print(f"[case] graph contig edits={edits} launches={q.launches} tiles={q.tile_launches}", flush=True)
    L.leyline_splice_contig(cache, n, dirs, k, workspace=ws)
    torch.cuda.synchronize()
    eager = host(t)
    assert not np.array_equal(eager, host(pristine))
    _replay_and_compare(lambda: L.leyline_splice_contig(cache, n, dirs, k, workspace=ws), t, pristine, eager)


def test_rotate_delta_in_a_graph(L):
    t, cache = _mla_cache(L, 2, 2048, seed=32)
    pristine = t.clone()
    print("[case] graph rotate", flush=True)
    L.leyline_rotate_delta(cache, -4064, row0=100, n_rows=1500)
    torch.cuda.synchronize()
    eager = host(t)
    _replay_and_compare(lambda: L.leyline_rotate_delta(cache, -4064, row0=100, n_rows=1500), t, pristine, eager)


@pytest.mark.parametrize("page,span,stub,n", [
    (1, (300, 420), 24, 1500),      # token slots: REMAP rotation in place plus the stub rows
    (16, (100, 137), 3, 600),       # 16-token pages: a gather of about 500 rows into fresh pages
])
def test_paged_small_splice_in_a_graph(L, page, span, stub, n):
    """A paged splice whose plan fits the kernel arguments (one sequence, one directive) and whose
    gather is small enqueues one kernel; the block table and freed list are outputs of the same
    launch."""
    wl = W.Workload("graph_paged", 2, "bf16", [W.mla_plane()], [W.Dir(span[0], span[1], stub)], [n],
                    page_size=page, seed=33)
    pools, bt, free, stubs = W.alloc_paged(wl, DEV)
    t = pools[0]
    pristine = t.clone()
    cache = L.make_cache([L.PlaneSpec(t, 1, 576, 512, 64, L.ROPE_INTERLEAVED, 10000.0)], paged=True)
    d = wl.dirs[0]
    dirs = L.make_directives([dict(span_start=d.span_start, span_end=d.span_end, stub=stubs[0], stub_len=d.stub_len)])
    new_lens, fresh, n_freed, ws_bytes = L.leyline_paged_query(cache, wl.seq_lens, bt.shape[1], dirs, 1)
    bt_out = torch.full_like(bt, -7)
    freed = torch.full((max(1, n_freed),), -7, dtype=torch.int32, device=DEV)
    ws = torch.empty(max(256, ws_bytes), dtype=torch.uint8, device=DEV)
    run = lambda: L.leyline_splice_paged(cache, wl.seq_lens, bt, bt_out, dirs, 1, free, freed, ws)
    print(f"[case] graph paged page={page} ws={ws_bytes} freed={n_freed} fresh={fresh}", flush=True)
    run()
    torch.cuda.synchronize()
    eager, eager_bt, eager_freed = host(t), host(bt_out), host(freed)
    assert not np.array_equal(eager, host(pristine))
    bt_out.fill_(-7)
    freed.fill_(-7)
    _replay_and_compare(run, t, pristine, eager)
    assert np.array_equal(host(bt_out), eager_bt) and np.array_equal(host(freed), eager_freed)
