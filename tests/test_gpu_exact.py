"""libleyline_exact.so (fp64 cos/sin and fp64 pair products, one rounding to the storage dtype)
against the oracle bit for bit: every element of the compared rows, rotary ones included, equals
the oracle's float64 rotation rounded once (Eq. "rotate"; the rounding of App. "bf16 K-storage
precision floor" taken exactly).  Full-size contiguous splices on three whole layers, the
8-edit ordered-tile splice, one fp32 layer, small random paged pools of every kernel path, the
full-size 131K paged splice (sampled rows, and every row's rotary bands on three layers), and
re-anchoring in place."""

import random

import numpy as np
import pytest
import torch

import workloads as W
from oracle import splice_oracle as O
from tests.parity_util import host, oracle_plane
from tests.test_gpu_paged import _check_sampled, _odirs, _random_workload, _run_gpu

pytestmark = pytest.mark.gpu

DEV = "cuda:0"


@pytest.fixture
def L():
    from paper_2606_01065_amd import leyline
    leyline.use_library(True)
    assert leyline.leyline_pair_bits() == 64
    yield leyline
    leyline.use_library(False)


def _specs(L, wl, tensors):
    return [L.PlaneSpec(t, p.n_heads, p.head_stride or p.row_elems, p.rot_offset, p.rot_dim,
                        p.style, p.base) for p, t in zip(wl.planes, tensors)]


@pytest.mark.parametrize("name", ["mla_dsv3_32k", "gqa_llama3_8b_16k", "mla_dsv3_32k_edits8", "mla_1l_4k_f32"])
def test_contiguous_splice_is_bit_identical_to_the_oracle(L, name):
    wl = W.WORKLOADS[name]()
    layers = sorted({0, wl.n_layers // 2, wl.n_layers - 1})
    print(f"[case] exact {name} layers {layers}", flush=True)
    planes, stubs = W.alloc_contig(wl, DEV)
    sel = torch.tensor(layers, device=DEV)
    before = [host(t.index_select(0, sel)) for t in planes]
    stubs_h = [[host(s.index_select(0, sel)) for s in per] for per in stubs]
    cache = L.make_cache(_specs(L, wl, planes))
    dirs = L.make_directives([dict(span_start=d.span_start, span_end=d.span_end, stub=stubs[j], stub_len=d.stub_len)
                              for j, d in enumerate(wl.dirs)])
    n = wl.seq_lens[0]
    new_len = L.leyline_splice_contig(cache, n, dirs, len(wl.dirs))
    torch.cuda.synchronize()
    odirs = [O.Directive(d.span_start, d.span_end, d.stub_len) for d in wl.dirs]
    for pi, desc in enumerate(wl.planes):
        plane = oracle_plane(desc)
        k = len(layers)
        want, n_want = O.splice_contig(before[pi].reshape(k, wl.capacity, -1), n, odirs,
                                       [s[pi].reshape(k, s[pi].shape[1], -1) for s in stubs_h], plane, wl.dtype)
        assert new_len == n_want
        got = host(planes[pi].index_select(0, sel)).reshape(want.shape)
        g, w = got[:, :new_len], want[:, :new_len]
        if wl.dtype == "f32":
            g, w = g.view(np.uint32), w.view(np.uint32)
        same = g == w
        assert same.all(), f"{name} plane {pi}: {int((~same).sum())} elements differ"


@pytest.mark.parametrize("kind,dtype", [("mla", "bf16"), ("gqa", "bf16"), ("mla", "f32"), ("mla_neox", "bf16"),
                                        ("four", "bf16"), ("gqa8", "bf16")])
def test_small_paged_pools_are_bit_identical_to_the_oracle(L, kind, dtype):
    rng = random.Random({"mla": 801, "gqa": 802, "mla_neox": 803, "four": 804, "gqa8": 805}[kind] + (dtype == "f32"))
    for page in (1, 16, 64):
        for ci in range(4):
            wl = _random_workload(rng, page, kind, dtype, max_len=900 if page == 1 else None)
            print(f"[case] exact paged {kind}/{dtype} page={page} case={ci} lens={wl.seq_lens} dirs={wl.dirs}",
                  flush=True)
            pools, bt, free, stubs = W.alloc_paged(wl, DEV, spare_pages=3)
            before = [host(p) for p in pools]
            bt_h, free_h = host(bt), host(free)
            stubs_h = [[host(s).reshape(wl.n_layers, s.shape[1], p.row_elems) for s, p in zip(per, wl.planes)]
                       for per in stubs]
            bt_out, freed, new_lens = _run_gpu(L, wl, pools, bt, free, stubs)
            planes = [oracle_plane(p) for p in wl.planes]
            flat = [b.reshape(b.shape[0], b.shape[1], b.shape[2], -1) for b in before]
            want, want_bt, want_lens, want_freed = O.splice_paged(
                flat, planes, dtype, bt_h, wl.seq_lens, _odirs(wl), stubs_h, list(free_h), page)
            assert new_lens == want_lens and np.array_equal(host(bt_out), want_bt)
            assert list(host(freed)) == want_freed
            for pi in range(len(planes)):
                got = host(pools[pi]).reshape(want[pi].shape)
                assert np.array_equal(got.view(np.uint8), want[pi].view(np.uint8)), f"page={page} case={ci} plane={pi}"


@pytest.mark.parametrize("kind", ["mla", "gqa"])
def test_rotation_in_place_is_bit_identical_to_the_oracle(L, kind):
    planes_d = [W.mla_plane()] if kind == "mla" else W.gqa_planes()
    wl = W.Workload(f"rot_{kind}", 3, "bf16", planes_d, [], [4096], capacity=4096, seed=71)
    tensors, _ = W.alloc_contig(wl, DEV)
    before = [host(t) for t in tensors]
    rows = torch.tensor(sorted(random.Random(5).sample(range(4096), 1500)), dtype=torch.int64, device=DEV)
    cache = L.make_cache(_specs(L, wl, tensors))
    for delta in (-6794, 1, 2000):
        print(f"[case] exact rotate {kind} delta={delta}", flush=True)
        L.leyline_rotate_delta(cache, delta, rows=rows)
        torch.cuda.synchronize()
        r = rows.cpu().numpy()
        for pi, desc in enumerate(wl.planes):
            plane = oracle_plane(desc)
            flat = before[pi].reshape(wl.n_layers, wl.capacity, -1)
            for layer in range(wl.n_layers):
                flat[layer, r] = O.rotate_rows(flat[layer, r], delta, plane, wl.dtype)
            got = host(tensors[pi]).reshape(flat.shape)
            assert np.array_equal(got, flat), f"{kind} plane {pi} delta {delta}"


def test_paged_131k_full_is_bit_identical(L):
    """The 8-directive 131K-token paged splice at full size (gather through the row table, bands
    packed into wavefronts of their own, each XCD gathering its own eighth)."""
    _check_sampled(L, W.mla_dsv3_paged_131k(), seed=23, exact=True)


@pytest.mark.parametrize("first", [20101, 20151])
def test_random_sweep_is_bit_identical(L, first):
    """The randomized sweep of test_gpu_random_sweep through the exact library, every element of
    every compared row bit for bit; seed 20168 is an fp32 pair that nearly cancels, whose result
    lies close to a float32 rounding boundary (it differed while the oracle's frequencies came from
    numpy's vectorized power and the kernel fused its fp64 products)."""
    from tests import test_gpu_contig as TC
    from tests import test_gpu_random_sweep as RS
    for seed in range(first, first + 50):
        rng = random.Random(seed)
        kind, dtype = RS.CONTIG_KINDS[seed % len(RS.CONTIG_KINDS)]
        n = rng.choice([1, 5, 63, 64, 65, 300, 1000, 2047, 3000])
        dirs = TC._random_dirs(rng, n, rng.randint(1, 8))
        wl = TC._small_workload(rng, kind, dtype, rng.randint(1, 4), n, dirs, extra=rng.randint(0, 40))
        print(f"[case] exact sweep contig seed {seed} {kind}/{dtype} n={n} dirs={dirs}", flush=True)
        planes_dev, stubs_dev = W.alloc_contig(wl, DEV, seed=seed)
        before = [host(t) for t in planes_dev]
        stubs_h = [[host(s) for s in per] for per in stubs_dev]
        cache = L.make_cache(TC._specs(L, wl, planes_dev))
        new_len = L.leyline_splice_contig(cache, n, L.make_directives(TC._dir_dicts(wl, stubs_dev)), len(wl.dirs))
        torch.cuda.synchronize()
        odirs = [O.Directive(d.span_start, d.span_end, d.stub_len, mode=d.mode) for d in wl.dirs]
        for pi, (desc, t) in enumerate(zip(wl.planes, planes_dev)):
            plane = oracle_plane(desc)
            shape = (wl.n_layers, wl.capacity, plane.row_elems)
            stubs = [s[pi].reshape(wl.n_layers, s[pi].shape[1], plane.row_elems) for s in stubs_h]
            want, n_want = O.splice_contig(before[pi].reshape(shape), n, odirs, stubs, plane, wl.dtype)
            assert new_len == n_want
            got = np.ascontiguousarray(host(t).reshape(shape)[:, :new_len])
            want = np.ascontiguousarray(want[:, :new_len])
            assert np.array_equal(got.view(np.uint8), want.view(np.uint8)), f"seed {seed} plane {pi}"
