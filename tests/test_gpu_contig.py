"""GPU parity of the contiguous in-place splice and of the in-place rotation (through the C ABI)
against the CPU oracle, on the same seeded inputs."""

import random
import zlib

import numpy as np
import pytest
import torch

import workloads as W
from oracle import splice_oracle as O
from tests import parity_util as PU
from tests.parity_util import assert_rows_match, host, oracle_plane

pytestmark = pytest.mark.gpu

DEV = "cuda:0"


@pytest.fixture(scope="module")
def L():
    from paper_2606_01065_amd import leyline
    return leyline


def _specs(L, wl, tensors):
    return [L.PlaneSpec(t, p.n_heads, p.head_stride or p.row_elems, p.rot_offset, p.rot_dim,
                        p.style, p.base) for p, t in zip(wl.planes, tensors)]


def _dir_dicts(wl, stubs):
    return [dict(span_start=d.span_start, span_end=d.span_end, stub=stubs[j], seq=d.seq,
                 stub_len=d.stub_len, mode=d.mode) for j, d in enumerate(wl.dirs)]


def _run_and_check(L, wl, planes_dev, stubs_dev, label, layers=None, stream=None):
    """Snapshot inputs, splice on the GPU, splice in the oracle, compare rows [0, n') (of the
    listed layers only, when given)."""
    print(f"[case] {label}", flush=True)
    if layers is not None:
        sel = torch.tensor(layers, device=DEV)
        before = [host(t.index_select(0, sel)) for t in planes_dev]
        stubs_h = [[host(s.index_select(0, sel)) for s in per] for per in stubs_dev]
        before_dev = [t.clone() for t in planes_dev]      # every layer, for the property check
    else:
        before = [host(t) for t in planes_dev]
    if layers is None:
        stubs_h = [[host(s) for s in per] for per in stubs_dev]
    n_check = wl.n_layers if layers is None else len(layers)
    cache = L.make_cache(_specs(L, wl, planes_dev))
    dirs = L.make_directives(_dir_dicts(wl, stubs_dev))
    n = wl.seq_lens[0]
    new_len = L.leyline_splice_contig(cache, n, dirs, len(wl.dirs), stream=stream)
    torch.cuda.synchronize()
    odirs = [O.Directive(d.span_start, d.span_end, d.stub_len, mode=d.mode) for d in wl.dirs]
    assert new_len == O.new_length(n, odirs)
    for pi, (desc, t) in enumerate(zip(wl.planes, planes_dev)):
        plane = oracle_plane(desc)
        got_t = t if layers is None else t.index_select(0, torch.tensor(layers, device=DEV))
        got = host(got_t).reshape(n_check, wl.capacity, plane.row_elems)
        src = before[pi].reshape(n_check, wl.capacity, plane.row_elems)
        stubs = [s[pi].reshape(n_check, s[pi].shape[1], plane.row_elems) for s in stubs_h]
        want, _ = O.splice_contig(src, n, odirs, stubs, plane, wl.dtype)
        assert_rows_match(got[:, :new_len], want[:, :new_len], plane, wl.dtype,
                          inputs=_inputs_for_new_rows(src, n, odirs, stubs),
                          what=f"{label} plane {pi}")
    if layers is not None:
        _check_every_layer(wl, before_dev, planes_dev, stubs_dev, n, odirs, new_len, label)
    return new_len


def _check_every_layer(wl, before, after, stubs, n, odirs, new_len, label):
    """Rows [0, n') of every layer by properties (the oracle compares whole layers on a subset):
    non-rotary elements and replacement rows bit-exact against their sources, shift-0 rows
    bit-identical, every rotary pair of a moved row turned by its angle (cos and sin from the
    oracle once per distinct shift)."""
    src = O.row_sources(n, odirs)
    assert len(src) == new_len
    kind = np.array([x[0] == "old" for x in src], dtype=bool)
    a = np.array([x[1] for x in src], dtype=np.int64)
    c = np.array([x[2] for x in src], dtype=np.int64)
    q = np.arange(new_len, dtype=np.int64)
    base = np.cumsum([0] + [d.stub_len for d in odirs])
    stub_row = np.array([base[j] for j in a[~kind]], dtype=np.int64) + c[~kind]
    t = lambda x: torch.from_numpy(np.ascontiguousarray(x)).to(DEV)
    q_old, a_old, q_st, st = t(q[kind]), t(a[kind]), t(q[~kind]), t(stub_row)
    shift = c[kind]
    moved = t(shift != 0)
    for pi, desc in enumerate(wl.planes):
        plane = oracle_plane(desc)
        row = plane.row_elems
        rot = t(PU.rotary_mask(plane))
        tables = PU.angle_tables(plane, shift[shift != 0], DEV) if plane.rot_dim else None
        b4 = before[pi].reshape(wl.n_layers, -1, row)
        af = after[pi].reshape(wl.n_layers, -1, row)
        st_all = torch.cat([s[pi].reshape(wl.n_layers, s[pi].shape[1], row) for s in stubs], dim=1) \
            if len(stubs) else None
        for layer in range(wl.n_layers):
            what = f"{label} plane {pi} layer {layer}"
            g, s0 = af[layer, q_old], b4[layer, a_old]
            assert torch.equal(PU.bits(g[:, ~rot]), PU.bits(s0[:, ~rot])), f"{what}: non-rotary"
            if st_all is not None:
                assert torch.equal(PU.bits(af[layer, q_st]), PU.bits(st_all[layer, st])), f"{what}: replacement"
            if plane.rot_dim:
                gr, sr = g[:, rot], s0[:, rot]
                assert torch.equal(PU.bits(gr[~moved]), PU.bits(sr[~moved])), f"{what}: shift-0 rows"
                PU.assert_bands_rotated(sr[moved], gr[moved], tables, wl.dtype, what)
    print(f"[info] {label}: every layer checked by properties ({new_len} rows x {wl.n_layers} layers)",
          flush=True)


def _inputs_for_new_rows(src, n, dirs, stubs):
    """The pre-rotation rows in new-position order (prefix, stub, downstream), per layer."""
    dirs = O.resolve_forget(n, dirs)
    pieces, cursor = [], 0
    for j, d in enumerate(dirs):
        pieces.append(src[:, cursor:d.span_start])
        pieces.append(stubs[j])
        cursor = d.span_end
    pieces.append(src[:, cursor:n])
    return np.concatenate(pieces, axis=1)


def _small_workload(rng, kind, dtype, n_layers, n, dirs, extra=0):
    if kind == "mla":
        planes = [W.mla_plane()]
    elif kind == "gqa":
        planes = W.gqa_planes(heads=2, dim=128)
    elif kind == "mla_neox":
        planes = [W.PlaneDesc((576,), 1, 576, 512, 64, 1, 10000.0)]
    elif kind == "four":      # the most planes a cache may have, both rotary styles and band widths
        planes = FOUR_PLANES
    elif kind == "mla_split":  # K_pe and c_kv in two arrays: a plane that is all rotary band
        planes = W.mla_split_planes()
    else:  # several interleaved heads with a partial rotary band, and a move-only plane
        planes = [W.PlaneDesc((4, 64), 4, 64, 32, 32, 0, 50000.0), W.PlaneDesc((128,))]
    cap = n + max(0, sum(d.stub_len - (d.span_end - d.span_start) for d in dirs)) + extra
    return W.Workload(f"small_{kind}", n_layers, dtype, planes, dirs, [n], capacity=max(cap, n),
                      seed=rng.randint(0, 10 ** 6))


# MLA row (narrow interleaved band), two-head half-split K, V, and a small plane whose interleaved
# band is half its row
FOUR_PLANES = [W.mla_plane(), W.PlaneDesc((2, 128), 2, 128, 0, 128, 1, 500000.0), W.PlaneDesc((256,)),
               W.PlaneDesc((64,), 1, 64, 32, 32, 0, 10000.0)]


def _random_dirs(rng, n, k):
    cuts = sorted(rng.sample(range(n + 1), min(2 * k, n + 1)))
    out = []
    for i in range(0, len(cuts) - 1, 2):
        s, e = cuts[i], cuts[i + 1]
        r = rng.choice([0, 1, rng.randint(0, 2 * (e - s) + 4), e - s, max(0, e - s - 1), e - s + 1])
        out.append(W.Dir(s, e, r))
    return out


def test_mla_1l_4k_f32_exact_recipe(L):
    """Keys built exactly as described: raw N(0,1) K_pe RoPE'd at its position (theta 1e4,
    interleaved); stub K_pe RoPE'd at 1024..1039.  After the splice every moved K_pe must match
    a fresh RoPE of its raw key at the new position, and the whole cache must match the oracle."""
    wl = W.mla_1l_4k_f32()
    gen = torch.Generator().manual_seed(wl.seed)
    cache = torch.randn((1, 4096, 576), generator=gen, dtype=torch.float32)
    raw = torch.randn((4096, 64), generator=gen, dtype=torch.float64).numpy()
    plane = oracle_plane(wl.planes[0])
    f = plane.frequencies()
    cache[0, :, 512:] = torch.from_numpy(O.encode(O.rope(raw, np.arange(4096), f, O.INTERLEAVED), O.F32))
    stub = torch.randn((1, 16, 576), generator=gen, dtype=torch.float32)
    stub_raw = torch.randn((16, 64), generator=gen, dtype=torch.float64).numpy()
    stub[0, :, 512:] = torch.from_numpy(O.encode(O.rope(stub_raw, np.arange(1024, 1040), f, O.INTERLEAVED), O.F32))
    planes_dev = [cache.to(DEV)]
    stubs_dev = [[stub.to(DEV)]]
    n_new = _run_and_check(L, wl, planes_dev, stubs_dev, "mla_1l_4k_f32")
    assert n_new == 4096 - 496
    got = host(planes_dev[0])[0]
    fresh = O.rope(raw[1536:], np.arange(1536, 4096) - 496, f, O.INTERLEAVED)
    err = np.abs(got[1040:n_new, 512:].astype(np.float64) - fresh)
    assert err.max() < 2e-5, err.max()
    assert np.array_equal(got[1024:1040], host(stub)[0])


@pytest.mark.parametrize("kind,dtype", [("mla", "bf16"), ("mla", "f32"), ("gqa", "bf16"),
                                        ("gqa", "f32"), ("mla_neox", "bf16"), ("heads", "bf16"),
                                        ("four", "bf16")])
def test_small_random_splices(L, kind, dtype):
    rng = random.Random(zlib.crc32(f"{kind}/{dtype}".encode()))
    cases = []
    for n in (1, 7, 64, 257, 600):
        for k in (1, 2, 3):
            cases.append((n, _random_dirs(rng, n, k)))
    # edge cases: delete at the very end, insert at 0, |Delta| = 1 both signs, Delta = 0,
    # empty stub, span bigger than the downstream, growth into spare capacity
    cases += [
        (300, [W.Dir(250, 300, 0)]),
        (300, [W.Dir(0, 0, 5)]),
        (300, [W.Dir(10, 11, 0)]),
        (300, [W.Dir(10, 10, 1)]),
        (300, [W.Dir(10, 20, 10)]),
        (300, [W.Dir(0, 280, 3)]),
        (300, [W.Dir(5, 6, 200)]),
        (300, [W.Dir(3, 9, 1), W.Dir(9, 9, 4), W.Dir(100, 180, 120), W.Dir(200, 290, 0)]),
        (0, [W.Dir(0, 0, 3)]),
    ]
    for ci, (n, dirs) in enumerate(cases):
        wl = _small_workload(rng, kind, dtype, 3, n, dirs, extra=rng.randint(0, 9))
        planes_dev, stubs_dev = W.alloc_contig(wl, DEV, seed=1000 + ci)
        _run_and_check(L, wl, planes_dev, stubs_dev, f"{kind}/{dtype} case {ci} n={n} dirs={dirs}")


@pytest.mark.parametrize("name", ["mla_dsv3_32k", "mla_dsv3_32k_split"])
def test_mla_dsv3_32k_full(L, name):
    """The 32K MLA splice, whole cache against the oracle; also on a cache that keeps K_pe and
    c_kv in separate arrays."""
    wl = W.WORKLOADS[name]()
    planes_dev, stubs_dev = W.alloc_contig(wl, DEV)
    n_new = _run_and_check(L, wl, planes_dev, stubs_dev, name)
    assert n_new == 32768 - 4064
    print(f"[info] bf16 rotary elements bit-identical to the oracle: {PU.LAST_BF16_EXACT_FRACTION:.6f}")


def test_gqa_llama3_8b_16k_full(L):
    wl = W.gqa_llama3_8b_16k()
    planes_dev, stubs_dev = W.alloc_contig(wl, DEV)
    n_new = _run_and_check(L, wl, planes_dev, stubs_dev, "gqa_llama3_8b_16k")
    assert n_new == 16384 - 2024
    print(f"[info] bf16 rotary elements bit-identical to the oracle: {PU.LAST_BF16_EXACT_FRACTION:.6f}")


@pytest.mark.parametrize("kind", ["mla", "gqa"])
def test_forget_prefix_trim(L, kind):
    """A trailing FORGET directive cuts the sequence after the earlier edits; rows before the cut
    match the oracle, nothing past it is compared (the caller re-prefills it)."""
    rng = random.Random(71 if kind == "mla" else 72)
    for ci in range(6):
        n = rng.randint(50, 700)
        dirs = _random_dirs(rng, n, rng.randint(0, 2))
        lo = dirs[-1].span_end if dirs else 0
        s = rng.randint(lo, n)
        dirs.append(W.Dir(s, rng.randint(s, n), 0, mode=1))
        grow = sum(max(0, d.stub_len - (d.span_end - d.span_start)) for d in dirs if d.mode == 0)
        wl = _small_workload(rng, kind, "bf16", 3, n, dirs, extra=grow + 4)
        planes_dev, stubs_dev = W.alloc_contig(wl, DEV, seed=500 + ci)
        _run_and_check(L, wl, planes_dev, stubs_dev, f"forget {kind} case {ci} n={n} dirs={dirs}")


@pytest.mark.parametrize("name,dirs,extra", [
    ("mla_dsv3_32k", [W.Dir(2048, 2049, 0)], 0),           # shift -1: ordered tiles, ascending
    ("mla_dsv3_32k", [W.Dir(2048, 2048, 3)], 3),           # insertion, shift +3: descending
    ("gqa_llama3_8b_16k", [W.Dir(4096, 4103, 0)], 0),      # shift -7, K and V planes in one launch
])
def test_small_shift_full_size(L, name, dirs, extra):
    """Shifts far too small for rounds run as ordered tiles; first, middle and last layers are
    compared whole against the oracle."""
    base = W.WORKLOADS[name]()
    wl = W.Workload(name, base.n_layers, base.dtype, base.planes, dirs, base.seq_lens,
                    capacity=base.capacity + extra, seed=base.seed)
    planes_dev, stubs_dev = W.alloc_contig(wl, DEV)
    cache = L.make_cache(_specs(L, wl, planes_dev))
    q = L.leyline_contig_query(cache, wl.seq_lens[0], L.make_directives(_dir_dicts(wl, stubs_dev)), len(dirs))
    assert q.tile_launches == 1 and q.workspace_bytes > 0
    layers = [0, wl.n_layers // 2, wl.n_layers - 1]
    _run_and_check(L, wl, planes_dev, stubs_dev, f"{name} small shift {dirs}", layers=layers)


@pytest.mark.parametrize("kind,k", [("mla", 16), ("mla", 20), ("gqa", 8)])
def test_many_directives_several_tile_launches(L, kind, k):
    """More (job, plane) items than one tile launch holds: the call runs as consecutive tile
    launches in dependency order; whole cache against the oracle."""
    rng = random.Random(900 + k + (kind == "gqa"))
    for ci in range(3):
        n = rng.randint(2500, 4000)
        cuts = sorted(rng.sample(range(n + 1), 2 * k))
        dirs = []
        for i in range(0, 2 * k, 2):
            s = cuts[i]
            e = min(cuts[i + 1], s + rng.randint(0, 40))
            dirs.append(W.Dir(s, e, max(0, (e - s) + rng.choice([-3, -1, 1, 2, 5]))))
        wl = _small_workload(rng, kind, "bf16", 3, n, dirs, extra=rng.randint(0, 5))
        planes_dev, stubs_dev = W.alloc_contig(wl, DEV, seed=2000 + ci)
        cache = L.make_cache(_specs(L, wl, planes_dev))
        q = L.leyline_contig_query(cache, n, L.make_directives(_dir_dicts(wl, stubs_dev)), k)
        assert q.tile_launches >= 2, q
        _run_and_check(L, wl, planes_dev, stubs_dev,
                       f"{kind} {k} directives case {ci} n={n} tile launches={q.tile_launches}")


def test_side_stream_without_caller_workspace(L):
    """Ordered-tile splices enqueued on a side stream with no caller workspace: the binding
    allocates the workspace on that stream; results match the oracle."""
    rng = random.Random(77)
    side = torch.cuda.Stream()
    for ci, kind in enumerate(["mla", "gqa", "mla", "gqa"]):
        n = rng.randint(1500, 3000)
        s = rng.randint(0, n - 10)
        dirs = [W.Dir(s, s + rng.randint(1, 9), rng.randint(0, 12))]
        wl = _small_workload(rng, kind, "bf16", 3, n, dirs, extra=12)
        planes_dev, stubs_dev = W.alloc_contig(wl, DEV, seed=3000 + ci)
        torch.cuda.synchronize()
        _run_and_check(L, wl, planes_dev, stubs_dev, f"side stream {kind} case {ci} n={n} dirs={dirs}",
                       stream=side)


def test_mla_dsv3_32k_edits8(L):
    """Eight edits drawn like the paper's randomized edit suite, both signs, one call."""
    wl = W.mla_dsv3_32k_edits8()
    planes_dev, stubs_dev = W.alloc_contig(wl, DEV)
    layers = [0, 30, 60]
    n_new = _run_and_check(L, wl, planes_dev, stubs_dev, "mla_dsv3_32k_edits8", layers=layers)
    assert n_new == 32768 + sum(d.stub_len - (d.span_end - d.span_start) for d in wl.dirs)


@pytest.mark.parametrize("paged", [False, True])
@pytest.mark.parametrize("kind,dtype", [("mla", "bf16"), ("gqa", "f32"), ("heads", "bf16")])
def test_rotate_delta(L, kind, dtype, paged):
    rng = random.Random(7)
    wl = _small_workload(rng, kind, dtype, 2, 512, [])
    print(f"[case] rotate {kind}/{dtype} paged={paged}", flush=True)
    planes_dev, _ = W.alloc_contig(wl, DEV, seed=3)
    if paged:   # view [L, 512 rows] as [L, 32 pages, 16 rows]
        planes_dev = [t.view((t.shape[0], 32, 16) + t.shape[2:]) for t in planes_dev]
    before = [host(t) for t in planes_dev]
    cache = L.make_cache(_specs(L, wl, planes_dev), paged=paged)
    rows = np.array(sorted(rng.sample(range(512), 77)), dtype=np.int64)
    for delta, use_list in ((-4064, True), (131071, False), (1, True)):
        if use_list:
            L.leyline_rotate_delta(cache, delta, rows=torch.from_numpy(rows).to(DEV))
            sel = rows
        else:
            L.leyline_rotate_delta(cache, delta, row0=100, n_rows=300)
            sel = np.arange(100, 400)
        torch.cuda.synchronize()
        for pi, desc in enumerate(wl.planes):
            plane = oracle_plane(desc)
            b = before[pi].reshape(2, 512, -1)
            g = host(planes_dev[pi]).reshape(2, 512, -1)
            want = b.copy()
            for layer in range(2):
                want[layer, sel] = O.rotate_rows(b[layer, sel], delta, plane, dtype)
            assert_rows_match(g, want, plane, dtype, inputs=b, what=f"rotate {delta}")
            before[pi] = g.reshape(before[pi].shape)


@pytest.mark.parametrize("name", ["mla_dsv3_rotate_32k", "gqa_llama3_8b_rotate_16k", "mla_dsv3_rotate_split_32k"])
def test_rotate_delta_full_size(L, name):
    """Re-anchoring in place at full size (the benchmark's rotate-only workloads): three whole
    layers against the oracle; every layer by properties (each member of the listed rows' pairs
    within 1.5 ulps of the exact rotation of its input, every other element bit-identical)."""
    wl = W.WORKLOADS[name]()
    delta, row0, n = wl.rotate
    planes_dev, _ = W.alloc_contig(wl, DEV)
    before = [t.clone() for t in planes_dev]
    layers = [0, wl.n_layers // 2, wl.n_layers - 1]
    sel = torch.tensor(layers, device=DEV)
    print(f"[case] {name}: rotate rows [{row0}, {row0 + n}) by {delta}", flush=True)
    cache = L.make_cache(_specs(L, wl, planes_dev))
    L.leyline_rotate_delta(cache, delta, row0=row0, n_rows=n)
    torch.cuda.synchronize()
    rows = torch.arange(row0, row0 + n, device=DEV)
    for pi, desc in enumerate(wl.planes):
        plane = oracle_plane(desc)
        row = plane.row_elems
        b = host(before[pi].index_select(0, sel)).reshape(len(layers), wl.capacity, row)
        g = host(planes_dev[pi].index_select(0, sel)).reshape(len(layers), wl.capacity, row)
        want = b.copy()
        for i in range(len(layers)):
            want[i, row0:row0 + n] = O.rotate_rows(b[i, row0:row0 + n], delta, plane, wl.dtype)
        assert_rows_match(g, want, plane, wl.dtype, inputs=b, what=f"{name} plane {pi}")
        rot = torch.from_numpy(PU.rotary_mask(plane)).to(DEV)
        tables = PU.angle_tables(plane, np.full(n, delta), DEV) if plane.rot_dim else None
        b4, af = before[pi].reshape(wl.n_layers, -1, row), planes_dev[pi].reshape(wl.n_layers, -1, row)
        for layer in range(wl.n_layers):
            what = f"{name} plane {pi} layer {layer}"
            gl, bl = af[layer], b4[layer]
            assert torch.equal(PU.bits(gl[:, ~rot]), PU.bits(bl[:, ~rot])), f"{what}: non-rotary"
            assert torch.equal(PU.bits(gl[:row0]), PU.bits(bl[:row0])), f"{what}: rows before"
            assert torch.equal(PU.bits(gl[row0 + n:]), PU.bits(bl[row0 + n:])), f"{what}: rows after"
            if plane.rot_dim:
                PU.assert_bands_rotated(bl[rows][:, rot], gl[rows][:, rot], tables, wl.dtype, what)


def test_rotate_delta_token_slots_full_size(L):
    """Re-anchoring in place on a token-slot cache at full size (the paper's own kernel operation:
    the K_pe bands of the 32K MLA splice's downstream slots, listed by physical slot, rotated
    where they are): three whole layers of the pool against the oracle; every layer by
    properties (each member of the listed slots' pairs within 1.5 ulps of the exact rotation of
    its input, every other element bit-identical)."""
    wl = W.WORKLOADS["mla_dsv3_slots_rotate_32k"]()
    delta, row0, n = wl.rotate
    pools, bt, _, _ = W.alloc_paged(wl, DEV)
    before = [t.clone() for t in pools]
    slots = bt[0, row0:row0 + n].long().contiguous()
    print(f"[case] {wl.name}: rotate {n} listed slots by {delta}", flush=True)
    specs = [L.PlaneSpec(t, p.n_heads, p.head_stride or p.row_elems, p.rot_offset, p.rot_dim, p.style, p.base)
             for p, t in zip(wl.planes, pools)]
    L.leyline_rotate_delta(L.make_cache(specs, paged=True), delta, rows=slots)
    torch.cuda.synchronize()
    plane = oracle_plane(wl.planes[0])
    row = plane.row_elems
    layers = [0, wl.n_layers // 2, wl.n_layers - 1]
    sel = torch.tensor(layers, device=DEV)
    b = host(before[0].index_select(0, sel)).reshape(len(layers), -1, row)
    g = host(pools[0].index_select(0, sel)).reshape(len(layers), -1, row)
    s_h = slots.cpu().numpy()
    want = b.copy()
    for i in range(len(layers)):
        want[i, s_h] = O.rotate_rows(b[i, s_h], delta, plane, wl.dtype)
    assert_rows_match(g, want, plane, wl.dtype, inputs=b, what=wl.name)
    rot = torch.from_numpy(PU.rotary_mask(plane)).to(DEV)
    tables = PU.angle_tables(plane, np.full(n, delta), DEV)
    listed = torch.zeros(pools[0].shape[1], dtype=torch.bool, device=DEV)
    listed[slots] = True
    b4, af = before[0].reshape(wl.n_layers, -1, row), pools[0].reshape(wl.n_layers, -1, row)
    for layer in range(wl.n_layers):
        what = f"{wl.name} layer {layer}"
        gl, bl = af[layer], b4[layer]
        assert torch.equal(PU.bits(gl[:, ~rot]), PU.bits(bl[:, ~rot])), f"{what}: non-rotary"
        assert torch.equal(PU.bits(gl[~listed]), PU.bits(bl[~listed])), f"{what}: slots not listed"
        PU.assert_bands_rotated(bl[slots][:, rot], gl[slots][:, rot], tables, wl.dtype, what)


def test_rotate_delta_flags_bad_rows(L):
    wl = _small_workload(random.Random(1), "mla", "bf16", 1, 64, [])
    planes_dev, _ = W.alloc_contig(wl, DEV, seed=4)
    before = host(planes_dev[0])
    cache = L.make_cache(_specs(L, wl, planes_dev))
    status = torch.zeros(1, dtype=torch.int32, device=DEV)
    rows = torch.tensor([3, 64, -1, 5], dtype=torch.int64, device=DEV)
    L.leyline_rotate_delta(cache, 10, rows=rows, device_status=status)
    torch.cuda.synchronize()
    assert int(status.item()) == L.STATUS_BAD_ROW
    after = host(planes_dev[0])
    plane = oracle_plane(wl.planes[0])
    want = before.copy()
    want[0, [3, 5]] = O.rotate_rows(before[0, [3, 5]], 10, plane, "bf16")
    assert_rows_match(after, want, plane, "bf16")
