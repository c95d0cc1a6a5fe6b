"""A wider randomized GPU parity sweep: for each seed one contiguous splice (1-8 directives of
both signs on 1-3000 rows, 1-4 layers, seven plane layouts and the split MLA layout, bf16 and
fp32) and one paged splice
(1-4 sequences, page sizes 1 to 64 including 3 and 48, some with copy-on-write), each compared
with the oracle as in the other GPU tests (Sec. 3.1 directive; Eq. "rotate")."""

import random

import numpy as np
import pytest

import workloads as W
from oracle import splice_oracle as O
from tests import test_gpu_contig as TC
from tests import test_gpu_paged as TP
from tests.parity_util import assert_rows_match, host, oracle_plane

pytestmark = pytest.mark.gpu

DEV = "cuda:0"
CONTIG_KINDS = [("mla", "bf16"), ("mla", "f32"), ("gqa", "bf16"), ("gqa", "f32"), ("mla_neox", "bf16"),
                ("heads", "bf16"), ("four", "bf16")]
PAGED_KINDS = [("mla", "bf16"), ("gqa", "bf16"), ("mla", "f32"), ("gqa", "f32"), ("mla_neox", "bf16"),
               ("four", "bf16"), ("gqa8", "bf16")]


@pytest.fixture(scope="module")
def L():
    from paper_2606_01065_amd import leyline
    return leyline


def _contig_case(L, seed, kinds=CONTIG_KINDS):
    rng = random.Random(seed)
    kind, dtype = kinds[seed % len(kinds)]
    n = rng.choice([1, 5, 63, 64, 65, 300, 1000, 2047, 3000])
    dirs = TC._random_dirs(rng, n, rng.randint(1, 8))
    wl = TC._small_workload(rng, kind, dtype, rng.randint(1, 4), n, dirs, extra=rng.randint(0, 40))
    planes_dev, stubs_dev = W.alloc_contig(wl, DEV, seed=seed)
    TC._run_and_check(L, wl, planes_dev, stubs_dev, f"sweep contig seed {seed} {kind}/{dtype} n={n} dirs={dirs}")
    return rng


def _paged_case(L, seed, rng, kinds=PAGED_KINDS):
    kind, dtype = kinds[seed % len(kinds)]
    page = rng.choice([1, 2, 3, 4, 16, 48, 64])
    wl = TP._random_workload(rng, page, kind, dtype, max_len=rng.choice([200, 900, 3000]))
    cow = rng.random() < 0.3
    print(f"[case] sweep paged seed {seed} {kind}/{dtype} page={page} cow={cow} lens={wl.seq_lens} "
          f"dirs={wl.dirs}", flush=True)
    odirs = TP._odirs(wl)
    plans = O.plan_paged(wl.seq_lens, odirs, page, remap=not cow)
    extra = sum(k == O.ASSEMBLE for p in plans for k in p.kinds) + 3
    pools, bt, free, stubs = W.alloc_paged(wl, DEV, spare_pages=extra)
    before = [host(p) for p in pools]
    bt_h, free_h = host(bt), host(free)
    stubs_h = [[host(s).reshape(wl.n_layers, s.shape[1], p.row_elems) for s, p in zip(per, wl.planes)]
               for per in stubs]
    bt_out, freed, new_lens = TP._run_gpu(L, wl, pools, bt, free, stubs,
                                          flags=L.PAGED_COPY_ON_WRITE if cow else 0)
    planes = [oracle_plane(p) for p in wl.planes]
    flat = [b.reshape(b.shape[0], b.shape[1], b.shape[2], -1) for b in before]
    want, want_bt, want_lens, want_freed = O.splice_paged(flat, planes, dtype, bt_h, wl.seq_lens, odirs,
                                                          stubs_h, list(free_h), page, remap=not cow)
    assert new_lens == want_lens
    assert np.array_equal(host(bt_out), want_bt)
    assert list(host(freed)) == want_freed
    for pi, plane in enumerate(planes):
        got = host(pools[pi]).reshape(want[pi].shape)
        assert_rows_match(got, want[pi], plane, dtype, what=f"sweep paged seed {seed} plane={pi}")


@pytest.mark.parametrize("first", [5001, 5051, 5101, 5151])
def test_random_sweep(L, first):
    for seed in range(first, first + 50):
        rng = _contig_case(L, seed)
        _paged_case(L, seed, rng)


@pytest.mark.parametrize("first", [6001])
def test_random_sweep_split_layout(L, first):
    """The same sweep on caches that keep K_pe and c_kv in two arrays (a plane that is all
    rotary band next to a move-only plane), bf16 and fp32."""
    kinds = [("mla_split", "bf16"), ("mla_split", "f32")]
    for seed in range(first, first + 40):
        rng = _contig_case(L, seed, kinds)
        _paged_case(L, seed, rng, kinds)


def _many_dirs(rng, n, k, seq=0):
    cuts = sorted(rng.sample(range(n + 1), min(2 * k, n + 1)))
    out = []
    for i in range(0, len(cuts) - 1, 2):
        s, e = cuts[i], cuts[i + 1]
        r = rng.choice([0, 1, e - s, rng.randint(0, 2 * (e - s) + 3), max(0, e - s - 1), e - s + 1])
        out.append(W.Dir(s, e, r, seq=seq))
    return out


@pytest.mark.parametrize("seed", [70001, 70002, 70003, 70004, 70005, 70006])
def test_many_directives(L, seed):
    """Calls of 20-400 directives on caches of 2,000-20,000 rows: many distinct shifts (the
    cos/sin table written by several prep launches), several ordered-tile launches and rounds
    (App. "Randomized edit-suite stress test" regime, at larger counts)."""
    rng = random.Random(seed)
    kind, dtype = [("mla", "bf16"), ("gqa", "bf16"), ("mla", "f32"), ("four", "bf16"), ("heads", "bf16")][seed % 5]
    n = rng.choice([2000, 8000, 20000])
    dirs = _many_dirs(rng, n, rng.randint(20, 400))
    wl = TC._small_workload(rng, kind, dtype, rng.randint(1, 2), n, dirs, extra=rng.randint(0, 3000))
    planes_dev, stubs_dev = W.alloc_contig(wl, DEV, seed=seed)
    TC._run_and_check(L, wl, planes_dev, stubs_dev, f"many directives seed {seed} {kind}/{dtype} n={n} k={len(dirs)}")
