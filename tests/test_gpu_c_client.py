"""The library used from C with no torch in the process: tests/_bin/c_client (built from
tests/c_client.c by __graft_entry__.build()) allocates device memory with hipMalloc, splices a
contiguous cache through the C ABI and writes the cache back; the result must match the oracle."""

import os
import random
import struct
import subprocess

import numpy as np
import pytest

import workloads as W
from oracle import splice_oracle as O
from tests.parity_util import assert_rows_match, host, oracle_plane

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CLIENT = os.path.join(ROOT, "tests", "_bin", "c_client")

CASES = [
    # (label, planes, dtype, layers, seq_len, directives, spare capacity)
    ("mla, one round", [W.mla_plane()], "bf16", 3, 3000, [W.Dir(400, 2000, 8)], 0),
    ("mla tiles, three edits", [W.mla_plane()], "bf16", 2, 2000,
     [W.Dir(10, 13, 0), W.Dir(700, 700, 5), W.Dir(1500, 1540, 44)], 8),
    ("gqa f32, two planes", W.gqa_planes(heads=2, dim=128), "f32", 2, 900, [W.Dir(100, 130, 2)], 0),
]


def _write_input(path, wl, planes_h, stubs_h):
    with open(path, "wb") as f:
        f.write(struct.pack("<6i", 0 if wl.dtype == "bf16" else 1, wl.n_layers, len(wl.planes), wl.capacity,
                            wl.seq_lens[0], len(wl.dirs)))
        for desc in wl.planes:
            pl = oracle_plane(desc)
            f.write(struct.pack("<6id", pl.row_elems, pl.n_heads, pl.head_stride, pl.rot_offset, pl.rot_dim,
                                pl.style, pl.base))
        for d in wl.dirs:
            f.write(struct.pack("<3q", d.span_start, d.span_end, d.stub_len))
        for a in planes_h:
            f.write(np.ascontiguousarray(a).tobytes())
        for per in stubs_h:
            for a in per:
                f.write(np.ascontiguousarray(a).tobytes())


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_c_client_splice_matches_oracle(tmp_path, case):
    label, planes, dtype, layers, n, dirs, extra = case
    assert os.path.exists(CLIENT), "tests/_bin/c_client is not built: run __graft_entry__.build()"
    wl = W.Workload(f"c_client {label}", layers, dtype, planes, dirs, [n], capacity=n + extra, seed=55)
    planes_t, stubs_t = W.alloc_contig(wl, "cpu")
    planes_h = [host(t) for t in planes_t]
    stubs_h = [[host(s) for s in per] for per in stubs_t]
    inp, out = str(tmp_path / "in.bin"), str(tmp_path / "out.bin")
    _write_input(inp, wl, planes_h, stubs_h)
    print(f"[case] c client: {label}", flush=True)
    r = subprocess.run([CLIENT, inp, out], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, r.stdout + r.stderr
    print(r.stdout.strip(), flush=True)
    tiles = int(r.stdout.split("tile_launches")[1].split()[0])
    assert (tiles == 0) == label.startswith("mla, one round"), r.stdout
    with open(out, "rb") as f:
        rc, new_len = struct.unpack("<2q", f.read(16))
        assert rc == 0, r.stdout
        odirs = [O.Directive(d.span_start, d.span_end, d.stub_len) for d in wl.dirs]
        assert new_len == O.new_length(n, odirs)
        for pi, desc in enumerate(wl.planes):
            plane = oracle_plane(desc)
            sdt = O.storage_numpy_dtype(dtype)
            count = layers * wl.capacity * plane.row_elems
            got = np.frombuffer(f.read(count * np.dtype(sdt).itemsize), dtype=sdt).reshape(
                layers, wl.capacity, plane.row_elems)
            src = planes_h[pi].reshape(layers, wl.capacity, plane.row_elems)
            st = [s[pi].reshape(layers, s[pi].shape[1], plane.row_elems) for s in stubs_h]
            want, _ = O.splice_contig(src, n, odirs, st, plane, dtype)
            assert_rows_match(got[:, :new_len], want[:, :new_len], plane, dtype, what=f"{label} plane {pi}")
