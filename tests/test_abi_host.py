"""C-ABI checks that need no GPU: every declared symbol is exported, argument validation returns
the documented codes before anything is enqueued, and the host page planner agrees bit-exactly
with the oracle's page plan."""

import ctypes
import os
import random
import re

import numpy as np
import pytest

from oracle import splice_oracle as O

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

L = pytest.importorskip("paper_2606_01065_amd.leyline",
                        reason="libleyline.so not built (python -m paper_2606_01065_amd.build)")


def _declared_functions():
    text = open(os.path.join(ROOT, "include", "leyline.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(leyline_[a-z_]+)\s*\(", text)))


def test_library_exports_every_declared_symbol():
    declared = _declared_functions()
    assert declared, "no functions found in the header"
    lib = ctypes.CDLL(L.LIB_PATH)
    for name in declared:
        assert hasattr(lib, name), name
    assert sorted(L.SYMBOLS) == declared
    assert L.leyline_abi_version() == 3
    assert "overlap" in L.strerror(L.E_OVERLAP)


class _FakeTensor:
    """Stands in for a device tensor when only pointers and shapes are needed (validation paths
    return before any device access)."""

    def __init__(self, shape, dtype, ptr=0x10000, strides=None):
        import torch
        self.shape = shape
        self.dtype = dtype
        self._ptr = ptr
        if strides is None:
            strides, acc = [], 1
            for d in reversed(shape):
                strides.append(acc)
                acc *= d
            strides = list(reversed(strides))
        self._strides = strides

    def data_ptr(self):
        return self._ptr

    def stride(self, i):
        return self._strides[i]

    def numel(self):
        return int(np.prod(self.shape))

    def element_size(self):
        import torch
        return torch.empty(0, dtype=self.dtype).element_size()


def _mla_cache(n_layers=2, cap=64, ptr=0x10000):
    import torch
    t = _FakeTensor((n_layers, cap, 576), torch.bfloat16, ptr)
    return L.make_cache([L.PlaneSpec(t, 1, 576, 512, 64, L.ROPE_INTERLEAVED, 10000.0)])


def _dirs(spec, stub_ptr=0x20000):
    arr = (L.leyline_directive * max(1, len(spec)))()
    for i, (s, e, r, *rest) in enumerate(spec):
        arr[i].seq = rest[0] if rest else 0
        arr[i].mode = rest[1] if len(rest) > 1 else L.AMORTIZE
        arr[i].span_start, arr[i].span_end, arr[i].stub_len = s, e, r
        arr[i].stub[0] = stub_ptr if r else None
    return arr


def _contig_rc(cache, n, spec):
    new_len = ctypes.c_int64(-1)
    d = _dirs(spec)
    return L._lib.leyline_splice_contig(ctypes.byref(cache), n, d, len(spec), ctypes.byref(new_len), None,
                                        None, 0, None)


def test_descriptors_keep_the_tensors_they_point_to_alive():
    """make_cache and make_directives store raw device pointers; the descriptors must keep the
    plane and replacement tensors alive, or a caller that keeps only the descriptors (a
    benchmark's step closure, a captured graph) would splice freed memory."""
    import gc
    import weakref

    import torch
    plane = torch.zeros((2, 64, 576), dtype=torch.bfloat16)
    stub = torch.zeros((2, 3, 576), dtype=torch.bfloat16)
    wp, ws = weakref.ref(plane), weakref.ref(stub)
    cache = L.make_cache([L.PlaneSpec(plane, 1, 576, 512, 64, L.ROPE_INTERLEAVED, 10000.0)])
    dirs = L.make_directives([dict(span_start=1, span_end=2, stub=[stub])])
    del plane, stub
    gc.collect()
    assert wp() is not None and ws() is not None
    assert cache.planes[0].base == wp().data_ptr() and dirs[0].stub[0] == ws().data_ptr()
    del cache, dirs
    gc.collect()
    assert wp() is None and ws() is None


def test_contig_validation_codes():
    c = _mla_cache()
    assert _contig_rc(c, 65, [(0, 1, 0)]) == L.E_RANGE                    # seq_len > capacity
    assert _contig_rc(c, 60, [(5, 70, 0)]) == L.E_RANGE                   # span past seq_len
    assert _contig_rc(c, 60, [(6, 5, 0)]) == L.E_RANGE                    # start > end
    assert _contig_rc(c, 60, [(10, 20, 1), (5, 8, 1)]) == L.E_ORDER
    assert _contig_rc(c, 60, [(10, 20, 1), (15, 30, 1)]) == L.E_OVERLAP
    assert _contig_rc(c, 60, [(10, 10, 5)]) == L.E_CAPACITY               # 65 > 64 rows
    d = _dirs([(1, 2, 0), (5, 6, 0)])
    d[0].mode = L.FORGET                                                  # FORGET not last
    assert L._lib.leyline_splice_contig(ctypes.byref(c), 10, d, 2, None, None, None, 0, None) == L.E_MODE
    d = _dirs([(1, 2, 3)])
    d[0].mode = L.FORGET                                                  # FORGET with a replacement
    assert L._lib.leyline_splice_contig(ctypes.byref(c), 10, d, 1, None, None, None, 0, None) == L.E_MODE
    d = _dirs([(1, 2, 0)])
    d[0].mode = 7
    assert L._lib.leyline_splice_contig(ctypes.byref(c), 10, d, 1, None, None, None, 0, None) == L.E_INVAL
    d = _dirs([(1, 2, 3)], stub_ptr=0)                                    # stub pointer missing
    assert L._lib.leyline_splice_contig(ctypes.byref(c), 10, d, 1, None, None, None, 0, None) == L.E_INVAL
    d = _dirs([(1, 2, 3)], stub_ptr=0x20008)                              # stub misaligned
    assert L._lib.leyline_splice_contig(ctypes.byref(c), 10, d, 1, None, None, None, 0, None) == L.E_INVAL
    bad = _mla_cache(ptr=0x10008)                                         # cache misaligned
    assert _contig_rc(bad, 10, [(1, 2, 0)]) == L.E_INVAL
    c.planes[0].rot_dim = 63                                              # odd rotary band
    assert _contig_rc(c, 10, [(1, 2, 0)]) == L.E_INVAL
    c = _mla_cache()
    c.planes[0].rot_offset = 520                                          # band overruns the head
    assert _contig_rc(c, 10, [(1, 2, 0)]) == L.E_INVAL
    c = _mla_cache()
    c.page_size = 64                                                      # paged layout refused
    assert _contig_rc(c, 10, [(1, 2, 0)]) == L.E_INVAL


def test_contig_query_reports_rounds_tiles_and_workspace():
    """A left shift by m of D downstream rows can run as ceil(D/m) rounds (one launch each, no
    workspace) when every round moves at least 64 MB; otherwise, and whenever it would take more
    than 16 rounds, the whole call (moves and replacement copies) runs as ordered tiles in one
    launch, after one launch that clears the tiles' counter and flags in the workspace and writes
    the cos/sin table there.  With rounds, a left shift's replacement copy rides in the first
    round's launch with a workgroup range of its own; a right shift's copy overwrites downstream
    rows and waits for the move in a launch of its own."""
    big = _mla_cache(n_layers=61, cap=32768)                                # 1152-byte rows
    q = L.leyline_contig_query(big, 32768, _dirs([(14055, 18151, 32)]), 1)   # m=4064: 513 MB rounds
    assert (q.new_len, q.launches, q.tile_launches, q.workspace_bytes) == (32768 - 4064, 4, 0, 0)
    c = _mla_cache(cap=64)                                                  # 2 layers, 72 chunks/row
    q = L.leyline_contig_query(c, 60, _dirs([(10, 20, 2)]), 1)               # m=8, D=40: small rounds
    assert (q.new_len, q.launches, q.tile_launches) == (52, 1 + 1, 1)        # prep, tiles (+ stub)
    q = L.leyline_contig_query(c, 60, _dirs([(10, 11, 0)]), 1)               # m=1, D=49
    tiles = -(-49 * 72 // 8192)                      # per layer; a tile is 1024 threads x 8 chunks
    assert (q.new_len, q.launches, q.tile_launches) == (59, 1 + 1, 1)
    # one 256-byte counter, a flag per (layer, tile), then 32 cos/sin pairs of 8 bytes
    flags_end = 256 + 4 * 2 * tiles
    assert q.workspace_bytes == -(-(-(-flags_end // 256) * 256 + 32 * 8) // 256) * 256
    q = L.leyline_contig_query(c, 60, _dirs([(10, 12, 4)]), 1)               # m=2 right, D=48
    assert (q.new_len, q.launches, q.tile_launches) == (62, 1 + 1, 1)
    q = L.leyline_contig_query(c, 60, _dirs([(10, 40, 2)]), 1)               # m=28 > D=20: one round
    assert (q.new_len, q.launches, q.tile_launches, q.workspace_bytes) == (32, 1, 0, 0)
    # a right shift's replacement overwrites downstream rows: it waits for the move (two launches)
    q = L.leyline_contig_query(c, 30, _dirs([(10, 10, 20)]), 1)              # m=20 right, D=20
    assert (q.new_len, q.launches, q.tile_launches, q.workspace_bytes) == (50, 2, 0, 0)
    # several directives with small shifts: one prep and one tile launch for all of them
    q = L.leyline_contig_query(c, 60, _dirs([(5, 7, 1), (20, 22, 3), (40, 41, 0)]), 3)
    assert (q.new_len, q.launches, q.tile_launches) == (59, 1 + 1, 1)
    with pytest.raises(L.LeylineError) as e:
        L.leyline_contig_query(c, 60, _dirs([(10, 10, 5)]), 1)
    assert e.value.code == L.E_CAPACITY


def test_contig_many_directives_split_tile_and_prep_launches():
    """A tile launch holds at most 24 (job, plane) items and a prep launch writes at most 320
    cos/sin pairs: 16 small-shift edits on the MLA cache (16 moves, 16 copies, 16 shifts of 32
    pairs) need two of each; the workspace holds both counters, the flags and the table."""
    c = _mla_cache(n_layers=3, cap=4000)
    spec = [(100 + 200 * i, 110 + 200 * i, 10 + (i % 3) + 1) for i in range(16)]
    q = L.leyline_contig_query(c, 3800, _dirs(spec), 16)
    assert (q.tile_launches, q.launches) == (2, 2 + 2)
    assert q.workspace_bytes >= 2 * 256 + 16 * 32 * 8


def test_contig_tiles_need_a_workspace():
    c = _mla_cache(cap=64)
    new_len = ctypes.c_int64(-1)
    d = _dirs([(10, 11, 0)])
    assert L._lib.leyline_splice_contig(ctypes.byref(c), 60, d, 1, ctypes.byref(new_len), None,
                                        None, 0, None) == L.E_WORKSPACE
    assert L._lib.leyline_splice_contig(ctypes.byref(c), 60, d, 1, ctypes.byref(new_len), None,
                                        0x10080, 4096, None) == L.E_WORKSPACE      # misaligned
    assert L._lib.leyline_splice_contig(ctypes.byref(c), 60, d, 1, ctypes.byref(new_len), None,
                                        0x10000, 16, None) == L.E_WORKSPACE        # too small


def test_noalloc_splice_refuses_more_than_its_scratch_before_any_enqueue():
    """leyline_splice_contig_noalloc takes its workspace from a fixed 1 MiB array: a small-shift
    splice whose ordered tiles need more (here 61 layers of a 600K-token MLA cache: one 4-byte
    flag per tile of 8192 chunks and layer) is refused with E_WORKSPACE before any device call;
    a call that moves nothing needs no scratch and no device."""
    big = _mla_cache(n_layers=61, cap=600000)
    d = _dirs([(10, 11, 0)])
    assert L.leyline_contig_query(big, 600000, d, 1).workspace_bytes > L.SCRATCH_BYTES
    new_len = ctypes.c_int64(-1)
    assert L._lib.leyline_splice_contig_noalloc(ctypes.byref(big), 600000, d, 1, ctypes.byref(new_len),
                                                None, None) == L.E_WORKSPACE
    c = _mla_cache()
    assert L._lib.leyline_splice_contig_noalloc(ctypes.byref(c), 40, None, 0, ctypes.byref(new_len),
                                                None, None) == 0
    assert new_len.value == 40
    assert L._lib.leyline_splice_contig_noalloc(ctypes.byref(c), 70, None, 0, ctypes.byref(new_len),
                                                None, None) == L.E_RANGE


def test_exact_library_sizes_its_tables_for_fp64_pairs():
    """libleyline_exact.so keeps 16-byte fp64 cos/sin entries: a one-token shift of the 2-layer
    MLA cache needs the same counter and flags and 32 pairs of 16 bytes; the small-shift edits
    that need two prep launches of 320 fp32 pairs need three of 208 fp64 pairs."""
    L.use_library(True)
    try:
        assert L.leyline_pair_bits() == 64
        c = _mla_cache(cap=64)
        q = L.leyline_contig_query(c, 60, _dirs([(10, 11, 0)]), 1)
        tiles = -(-49 * 72 // 8192)
        flags_end = 256 + 4 * 2 * tiles
        assert q.workspace_bytes == -(-(-(-flags_end // 256) * 256 + 32 * 16) // 256) * 256
        c = _mla_cache(n_layers=3, cap=4000)
        spec = [(100 + 200 * i, 110 + 200 * i, 10 + (i % 3) + 1) for i in range(16)]
        q = L.leyline_contig_query(c, 3800, _dirs(spec), 16)
        assert (q.tile_launches, q.launches) == (2, 3 + 2)
    finally:
        L.use_library(False)
    assert L.leyline_pair_bits() == 32


def test_forget_trims_without_moving_anything():
    """A FORGET directive (last of its sequence, no replacement) cuts the sequence at its span's
    start after the earlier directives; the cut itself moves nothing."""
    c = _mla_cache(cap=64)
    d = _dirs([(30, 45, 0)])
    d[0].mode = L.FORGET
    q = L.leyline_contig_query(c, 60, d, 1)
    assert (q.new_len, q.launches, q.workspace_bytes) == (30, 0, 0)
    new_len = ctypes.c_int64(-1)
    assert L._lib.leyline_splice_contig(ctypes.byref(c), 60, d, 1, ctypes.byref(new_len), None, None, 0, None) == 0
    assert new_len.value == 30
    d = _dirs([(10, 12, 0), (30, 30, 0)])                                # after a 2-row deletion
    d[1].mode = L.FORGET
    assert L.leyline_contig_query(c, 60, d, 2).new_len == 28


def test_contig_noop_calls_do_not_need_a_device():
    """A call with nothing to move (no directives, or Delta = 0 with an empty stub) enqueues
    nothing and reports the unchanged length."""
    c = _mla_cache()
    new_len = ctypes.c_int64(-1)
    assert L._lib.leyline_splice_contig(ctypes.byref(c), 40, None, 0, ctypes.byref(new_len), None, None, 0, None) == 0
    assert new_len.value == 40
    d = _dirs([(10, 10, 0)])
    assert L._lib.leyline_splice_contig(ctypes.byref(c), 40, d, 1, ctypes.byref(new_len), None, None, 0, None) == 0
    assert new_len.value == 40


def _random_paged(rng, n_seqs, page, max_len=400):
    lens = [rng.randint(0, max_len) for _ in range(n_seqs)]
    spec = []
    for b, n in enumerate(lens):
        k = rng.randint(0, 3)
        cuts = sorted(rng.sample(range(n + 1), min(2 * k, n + 1)))
        for i in range(0, len(cuts) - 1, 2):
            s, e = cuts[i], cuts[i + 1]
            r = rng.choice([0, rng.randint(0, 2 * (e - s) + 3), (e - s), max(0, e - s - page)])
            spec.append((s, e, r, b))
    return lens, spec


def test_paged_plan_matches_oracle_bit_exactly():
    rng = random.Random(31)
    for page in (1, 4, 16, 64):
        for _ in range(40):
            lens, spec = _random_paged(rng, rng.randint(1, 5), page)
            dirs = [O.Directive(s, e, r, seq=b) for s, e, r, b in spec]
            plans = O.plan_paged(lens, dirs, page)
            bt_stride = max([1] + [O.pages_for(max(n, p.new_len), page) for n, p in zip(lens, plans)])
            n_freed = sum(len(p.freed) for p in plans)
            kinds, srcs, fs, fp = L.leyline_paged_plan(page, lens, _dirs(spec), len(spec), bt_stride,
                                                       n_freed)
            kinds = np.array(kinds).reshape(len(lens), bt_stride)
            srcs = np.array(srcs).reshape(len(lens), bt_stride)
            for b, p in enumerate(plans):
                k = len(p.kinds)
                assert list(kinds[b, :k]) == p.kinds
                assert list(srcs[b, :k]) == p.sources
                assert np.all(kinds[b, k:] == L.PAGE_NONE)
            assert fs[:n_freed] == [b for b, p in enumerate(plans) for _ in p.freed]
            assert fp[:n_freed] == [x for p in plans for x in p.freed]


def _random_paged_degenerate(rng, n_seqs, page, max_len=300):
    """Directives drawn with replacement: empty spans, empty stubs (together: a directive that
    changes nothing), adjacent spans and equal starts all occur."""
    lens = [rng.randint(0, max_len) for _ in range(n_seqs)]
    spec = []
    for b, n in enumerate(lens):
        k = rng.randint(0, 4)
        cuts = sorted(rng.randint(0, n) for _ in range(2 * k))
        for i in range(0, len(cuts), 2):
            s, e = cuts[i], cuts[i + 1]
            r = rng.choice([0, 0, e - s, rng.randint(0, 2 * (e - s) + 3), (e - s) + page,
                            max(0, e - s - 2 * page)])
            spec.append((s, e, r, b))
        if rng.random() < 0.3:                                           # a trailing FORGET
            lo = spec[-1][1] if spec and spec[-1][3] == b else 0
            s = rng.randint(lo, n)
            spec.append((s, rng.randint(s, n), 0, b, O.FORGET))
    return lens, spec


def test_paged_plan_matches_oracle_on_degenerate_directives():
    """Degenerate directives, trailing FORGET directives, in-place and copy-on-write plans."""
    rng = random.Random(37)
    for page in (1, 2, 16):
        for _ in range(150):
            lens, spec = _random_paged_degenerate(rng, rng.randint(1, 4), page)
            cow = rng.random() < 0.5
            flags = L.PAGED_COPY_ON_WRITE if cow else 0
            dirs = [O.Directive(x[0], x[1], x[2], seq=x[3], mode=x[4] if len(x) > 4 else O.AMORTIZE)
                    for x in spec]
            try:
                plans = O.plan_paged(lens, dirs, page, remap=not cow)
                for b, n in enumerate(lens):
                    O.check_directives(n, O.resolve_forget(n, [d for d in dirs if d.seq == b]))
            except O.DirectiveError:
                with pytest.raises(L.LeylineError):
                    L.leyline_paged_plan(page, lens, _dirs(spec), len(spec), 64, 4096, flags)
                continue
            bt_stride = max([1] + [O.pages_for(max(n, p.new_len), page) for n, p in zip(lens, plans)])
            n_freed = sum(len(p.freed) for p in plans)
            kinds, srcs, fs, fp = L.leyline_paged_plan(page, lens, _dirs(spec), len(spec), bt_stride,
                                                       n_freed, flags)
            kinds = np.array(kinds).reshape(len(lens), bt_stride)
            srcs = np.array(srcs).reshape(len(lens), bt_stride)
            for b, p in enumerate(plans):
                k = len(p.kinds)
                assert list(kinds[b, :k]) == p.kinds, (lens, spec, b)
                assert list(srcs[b, :k]) == p.sources, (lens, spec, b)
                assert np.all(kinds[b, k:] == L.PAGE_NONE)
            assert fs[:n_freed] == [b for b, p in enumerate(plans) for _ in p.freed]
            assert fp[:n_freed] == [x for p in plans for x in p.freed]


def test_paged_query_and_plan_errors():
    import torch
    pool = _FakeTensor((2, 32, 16, 576), torch.bfloat16)
    cache = L.make_cache([L.PlaneSpec(pool, 1, 576, 512, 64)], paged=True)
    lens = [100, 40]
    spec = [(10, 50, 3, 0), (0, 8, 0, 1)]
    new, fresh, freed, ws = L.leyline_paged_query(cache, lens, 8, _dirs(spec), 2)
    dirs = [O.Directive(s, e, r, seq=b) for s, e, r, b in spec]
    plans = O.plan_paged(lens, dirs, 16)
    assert new == [p.new_len for p in plans]
    assert fresh == sum(k == O.ASSEMBLE for p in plans for k in p.kinds)
    assert freed == sum(len(p.freed) for p in plans)
    assert ws > 0 and ws % 256 == 0
    with pytest.raises(L.LeylineError) as e:
        L.leyline_paged_query(cache, lens, 8, _dirs([(10, 50, 3, 1), (0, 8, 0, 0)]), 2)
    assert e.value.code == L.E_ORDER
    with pytest.raises(L.LeylineError) as e:
        L.leyline_paged_query(cache, lens, 8, _dirs([(10, 50, 3, 2)]), 1)
    assert e.value.code == L.E_RANGE
    with pytest.raises(L.LeylineError) as e:
        L.leyline_paged_plan(16, lens, _dirs(spec), 2, 4, 16)               # 100 tokens need 7 pages
    assert e.value.code == L.E_CAPACITY


def test_paged_splice_validates_before_any_enqueue():
    import torch
    pool = _FakeTensor((2, 32, 16, 576), torch.bfloat16)
    cache = L.make_cache([L.PlaneSpec(pool, 1, 576, 512, 64)], paged=True)
    lens = [100]
    d = _dirs([(10, 50, 3, 0)])
    bt_in = _FakeTensor((1, 8), torch.int32, ptr=0x30000)
    bt_out = _FakeTensor((1, 8), torch.int32, ptr=0x40000)
    free = _FakeTensor((2,), torch.int32, ptr=0x50000)                     # too few free pages
    freed = _FakeTensor((8,), torch.int32, ptr=0x60000)
    ws = _FakeTensor((4096,), torch.uint8, ptr=0x70000)
    with pytest.raises(L.LeylineError) as e:
        L.leyline_splice_paged(cache, lens, bt_in, bt_out, d, 1, free, freed, ws, stream=0)
    assert e.value.code == L.E_CAPACITY
    free = _FakeTensor((16,), torch.int32, ptr=0x50000)
    small = _FakeTensor((16,), torch.uint8, ptr=0x70000)
    with pytest.raises(L.LeylineError) as e:
        L.leyline_splice_paged(cache, lens, bt_in, bt_out, d, 1, free, freed, small, stream=0)
    assert e.value.code == L.E_WORKSPACE
    with pytest.raises(L.LeylineError) as e:                                # tables alias
        L.leyline_splice_paged(cache, lens, bt_in, bt_in, d, 1, free, freed, ws, stream=0)
    assert e.value.code == L.E_INVAL
    # buffers that the same launch reads and writes may not share a byte: each overlapping pair
    # is refused before anything is enqueued (a mere neighbour is fine, as above)
    overlapping = [
        dict(bt_out=_FakeTensor((1, 8), torch.int32, ptr=0x30000 + 16)),    # old / new table
        dict(freed=_FakeTensor((8,), torch.int32, ptr=0x50000 + 60)),       # free list / freed list
        dict(freed=_FakeTensor((8,), torch.int32, ptr=0x40000 + 28)),       # new table / freed list
        dict(ws=_FakeTensor((4096,), torch.uint8, ptr=0x50000 - 256)),      # workspace / free list
        dict(status=_FakeTensor((1,), torch.int32, ptr=0x30000 + 4)),       # status / old table
    ]
    for o in overlapping:
        args = dict(bt_out=bt_out, freed=freed, ws=ws, status=None)
        args.update(o)
        with pytest.raises(L.LeylineError) as e:
            L.leyline_splice_paged(cache, lens, bt_in, args["bt_out"], d, 1, free, args["freed"], args["ws"],
                                   device_status=args["status"], stream=0)
        assert e.value.code == L.E_INVAL, o


def test_paged_splice_of_empty_sequences_with_empty_tables():
    """A batch whose sequences are and stay empty needs block tables without columns
    (bt_stride 0); the splice accepts what the query accepts, and with nothing to move, rotate or
    write it returns the (empty) results without enqueueing anything."""
    import torch
    pool = _FakeTensor((2, 32, 48, 576), torch.bfloat16)
    cache = L.make_cache([L.PlaneSpec(pool, 1, 576, 512, 64)], paged=True)
    lens = [0, 0]
    new, fresh, freed, ws_bytes = L.leyline_paged_query(cache, lens, 0, None, 0)
    assert (new, fresh, freed) == ([0, 0], 0, 0)
    bt_in = _FakeTensor((2, 0), torch.int32, ptr=0)                       # no columns, no memory
    bt_out = _FakeTensor((2, 0), torch.int32, ptr=0)
    free = _FakeTensor((4,), torch.int32, ptr=0x50000)
    freed_out = _FakeTensor((1,), torch.int32, ptr=0x60000)
    ws = _FakeTensor((max(256, ws_bytes),), torch.uint8, ptr=0x70000)
    assert L.leyline_splice_paged(cache, lens, bt_in, bt_out, None, 0, free, freed_out, ws,
                                  stream=0) == ([0, 0], 0, 0)
    with pytest.raises(L.LeylineError) as e:                                # a page would be needed
        L.leyline_splice_paged(cache, [1, 0], bt_in, bt_out, None, 0, free, freed_out, ws, stream=0)
    assert e.value.code == L.E_CAPACITY


def test_rotate_delta_validation():
    c = _mla_cache(cap=64)
    with pytest.raises(L.LeylineError) as e:
        L.leyline_rotate_delta(c, 5, row0=60, n_rows=5, stream=0)
    assert e.value.code == L.E_RANGE
    L.leyline_rotate_delta(c, 0, row0=0, n_rows=64, stream=0)             # R(0): nothing enqueued


def test_sizes_beyond_31_bit_indices_are_refused_before_any_enqueue():
    """Kernels index chunks with 31-bit integers; descriptors whose moves or tables would not fit
    are refused on the host (no device access: the pointers here are fake)."""
    huge = _mla_cache(n_layers=2, cap=1 << 31)                # 72 chunks per row
    n = (1 << 31) - 8
    rc = _contig_rc(huge, n, [(10, 12, 0)])                    # ~2^31 rows moved: > 2^31 chunks
    assert rc in (L.E_INVAL, L.E_WORKSPACE)
    with pytest.raises(L.LeylineError) as e:
        L.leyline_contig_query(huge, n, _dirs([(10, 12, 0)]), 1)
    assert e.value.code == L.E_INVAL
    import torch
    pool = _FakeTensor((2, 1 << 26, 64, 576), torch.bfloat16)  # 2^32 rows in the pool
    cache = L.make_cache([L.PlaneSpec(pool, 1, 576, 512, 64)], paged=True)
    with pytest.raises(L.LeylineError) as e:                 # in-place rotation of paged rows
        L.leyline_rotate_delta(cache, 5, row0=0, n_rows=10, stream=0)
    assert e.value.code == L.E_INVAL


@pytest.mark.parametrize("name", ["mla_dsv3_paged_b64", "mla_dsv3_paged_131k", "mla_dsv3_slots_32k",
                                  "gqa_llama3_8b_slots_16k", "mla_dsv3_slots_cow_32k"])
def test_paged_plan_matches_oracle_on_benchmark_workloads(name):
    """The page plans of the benchmarked paged splices (full size, host only) equal the oracle's."""
    import workloads as W
    wl = W.WORKLOADS[name]()
    remap = not (wl.paged_flags & L.PAGED_COPY_ON_WRITE)
    dirs = [O.Directive(d.span_start, d.span_end, d.stub_len, seq=d.seq) for d in wl.dirs]
    plans = O.plan_paged(wl.seq_lens, dirs, wl.page_size, remap=remap)
    bt_stride = W.paged_bt_stride(wl)
    n_freed = sum(len(p.freed) for p in plans)
    spec = [(d.span_start, d.span_end, d.stub_len, d.seq) for d in wl.dirs]
    kinds, srcs, fs, fp = L.leyline_paged_plan(wl.page_size, wl.seq_lens, _dirs(spec), len(spec), bt_stride,
                                               max(1, n_freed), wl.paged_flags)
    kinds = np.array(kinds).reshape(len(wl.seq_lens), bt_stride)
    srcs = np.array(srcs).reshape(len(wl.seq_lens), bt_stride)
    for b, p in enumerate(plans):
        k = len(p.kinds)
        assert list(kinds[b, :k]) == p.kinds
        assert list(srcs[b, :k]) == p.sources
    assert fp[:n_freed] == [x for p in plans for x in p.freed]


def test_contig_planning_scales_to_thousands_of_directives():
    """Ordering the moves of a call is near-linear in its directives (a sweep over the sorted
    source and destination ranges): 4096 small edits of a 400K-row cache plan in well under a
    second."""
    import time
    rng = random.Random(4096)
    n, k = 400000, 4096
    starts = sorted(rng.sample(range(0, n - 20, 20), k))
    spec = [(s, s + rng.randint(0, 10), rng.randint(0, 12)) for s in starts]
    c = _mla_cache(n_layers=2, cap=n + 12 * k)
    t0 = time.perf_counter()
    q = L.leyline_contig_query(c, n, _dirs(spec), k)
    assert time.perf_counter() - t0 < 1.0
    assert q.new_len == n + sum(r - (e - s) for s, e, r in spec)
    assert k // 24 <= q.tile_launches <= (2 * k) // 24 + 1
