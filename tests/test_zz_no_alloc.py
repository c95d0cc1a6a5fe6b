"""The splice without device allocation (leyline_splice_contig_noalloc: the workspace is the
library's fixed per-GPU scratch array) against leyline_splice_contig with a caller workspace:
identical lengths and bit-identical caches on two calls in a row, the second on a smaller input
than the first, both through the C ABI.  The shifts are small, so both calls run as ordered tiles
whose counters, flags and cos/sin table live in the scratch array."""

import pytest
import torch

import workloads as W
from oracle import splice_oracle as O
from tests.parity_util import bits

pytestmark = pytest.mark.gpu

DEV = "cuda:0"

# (label, planes, layers, sequence length, directives), largest first
CALLS = [
    ("mla 4 layers, 8192 tokens, 3 small-shift edits", [W.mla_plane()], 4, 8192,
     [W.Dir(100, 101, 0), W.Dir(3000, 3010, 12), W.Dir(5000, 5000, 3)]),
    ("gqa K+V 2 layers, 2048 tokens, 1 edit", W.gqa_planes(), 2, 2048, [W.Dir(500, 502, 1)]),
]


def _specs(L, wl, tensors):
    return [L.PlaneSpec(t, p.n_heads, p.head_stride or p.row_elems, p.rot_offset, p.rot_dim,
                        p.style, p.base) for p, t in zip(wl.planes, tensors)]


def test_noalloc_matches_the_workspace_entry_point_on_two_calls():
    from paper_2606_01065_amd import leyline as L
    torch.cuda.set_device(0)
    for i, (label, planes, n_layers, n, dirs) in enumerate(CALLS):
        print(f"[case] no-alloc call {i}: {label}", flush=True)
        wl = W.Workload(f"noalloc_{i}", n_layers, "bf16", planes, dirs, [n], capacity=n + 64, seed=40 + i)
        tensors, stubs = W.alloc_contig(wl, DEV)
        other = [t.clone() for t in tensors]
        cache_ws = L.make_cache(_specs(L, wl, tensors))
        cache_na = L.make_cache(_specs(L, wl, other))
        dd = L.make_directives([dict(span_start=d.span_start, span_end=d.span_end, stub=stubs[j],
                                     stub_len=d.stub_len) for j, d in enumerate(wl.dirs)])
        q = L.leyline_contig_query(cache_ws, n, dd, len(dirs))
        assert q.tile_launches > 0 and 0 < q.workspace_bytes <= L.SCRATCH_BYTES, q
        ws = torch.empty(q.workspace_bytes, dtype=torch.uint8, device=DEV)
        status = torch.zeros(2, dtype=torch.int32, device=DEV)
        n_ws = L.leyline_splice_contig(cache_ws, n, dd, len(dirs), workspace=ws, device_status=status[0:1])
        n_na = L.leyline_splice_contig_noalloc(cache_na, n, dd, len(dirs), device_status=status[1:2])
        torch.cuda.synchronize()
        want_len = O.new_length(n, [O.Directive(d.span_start, d.span_end, d.stub_len) for d in dirs])
        assert n_ws == n_na == want_len
        assert status.tolist() == [0, 0]
        for a, b in zip(tensors, other):
            assert torch.equal(bits(a[:, :want_len]), bits(b[:, :want_len])), label
        del tensors, other, stubs, ws
