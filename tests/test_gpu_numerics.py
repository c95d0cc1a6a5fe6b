"""GPU numerics of the re-anchoring (through the C ABI) against the oracle, across rotary shapes
and frequency schedules:

* the cross-architecture rotation-algebra sweep of the paper (App. "Cross-architecture
  rotation-algebra validation", Table "crossarch"): RoPE'd bf16 keys re-anchored by R(delta) on
  the GPU must match the oracle and stay within the paper's worst rel-L2 of R(delta)R(p)k against
  R(p+delta)k for each (head_dim, theta) configuration;
* splices on planes with rotary widths 64, 96 and 128, bases 1e4, 5e5 and 1e6, both pairings;
* a caller-given frequency table (a YaRN-style interpolation ramp, Sec. 3.3 "RoPE pairing
  convention" mentions the interpolated regime) through the contiguous, paged and rotate calls;
* chained in-place rotations (App. "Chained-rotation drift in bf16"): every step against the
  oracle applied to the GPU's previous state, and the end state against fresh RoPE at the final
  position within the paper's Table "drift" magnitudes;
* the precision-floor sweep (App. "bf16 K-storage precision floor"): keys at the paper's source
  positions re-anchored by shifts up to 6794 in fp32 and bf16 storage, against fresh RoPE.
"""

import random

import numpy as np
import pytest
import torch

import workloads as W
from oracle import splice_oracle as O
from tests.parity_util import assert_rows_match, device, host

pytestmark = pytest.mark.gpu

DEV = "cuda:0"


@pytest.fixture(scope="module")
def L():
    from paper_2606_01065_amd import leyline
    return leyline


def _spec(L, t, plane: O.Plane, inv_freq=None):
    return L.PlaneSpec(t, plane.n_heads, plane.head_stride, plane.rot_offset, plane.rot_dim,
                       plane.style, plane.base, inv_freq=inv_freq)


# Table "crossarch": (config, head_dim, rope_theta, worst rel-L2 printed by the paper).  The
# pairing follows Sec. 3.3: interleaved for MLA, half-split for the GQA families.
CROSSARCH = [
    ("mla_dsv2", 64, 3.2e7, O.INTERLEAVED, 4.3e-3),
    ("mla_alt", 64, 1e4, O.INTERLEAVED, 4.8e-3),
    ("gqa_llama31", 128, 5e5, O.NEOX, 4.6e-3),
    ("gqa_qwen3", 128, 1e6, O.NEOX, 4.7e-3),
    ("gqa_phi3", 96, 1e4, O.NEOX, 4.9e-3),
]
SOURCE_POSITIONS = (0, 517, 4096, 30000)
DELTAS = (-2000, -512, -21, 1, 48, 512, 2000)     # the paper's validation set, both signs


@pytest.mark.parametrize("name,d,theta,style,worst", CROSSARCH, ids=[c[0] for c in CROSSARCH])
def test_rotation_algebra_sweep_within_paper_bounds(L, name, d, theta, style, worst):
    """K = [batch 8, heads 32, head_dim d] in bf16, RoPE'd at p; R(delta) on the GPU; 5 seeds x
    the (p, delta) cases with p + delta in [0, 32768)."""
    heads, batch = 32, 8
    plane = O.Plane(row_elems=heads * d, n_heads=heads, head_stride=d, rot_offset=0, rot_dim=d,
                    style=style, base=theta)
    f = plane.frequencies()
    cases = [(p, dl) for p in SOURCE_POSITIONS for dl in DELTAS if 0 <= p + dl < 32768]
    rels = []
    for seed in range(5):
        print(f"[case] crossarch {name} seed {seed}", flush=True)
        rng = np.random.default_rng(1000 + seed)
        raw = rng.standard_normal((len(cases), batch * heads, d))
        stored = np.stack([O.encode(O.rope(raw[c], p, f, style), O.BF16) for c, (p, _) in enumerate(cases)])
        rows = stored.reshape(len(cases) * batch, heads * d)
        t = device(rows, DEV).view(1, len(cases) * batch, heads * d)
        cache = L.make_cache([_spec(L, t, plane)])
        for c, (_, dl) in enumerate(cases):
            L.leyline_rotate_delta(cache, dl, row0=c * batch, n_rows=batch)
        torch.cuda.synchronize()
        got = host(t).reshape(len(cases), batch, heads * d)
        for c, (p, dl) in enumerate(cases):
            src = stored[c].reshape(batch, heads * d)
            want = O.rotate_rows(src, dl, plane, O.BF16)
            assert_rows_match(got[c], want, plane, O.BF16, inputs=src, what=f"{name} p={p} delta={dl}")
            fresh = O.rope(raw[c], p + dl, f, style)
            g = O.decode(got[c], O.BF16).reshape(batch * heads, d)
            rels.append(np.linalg.norm(g - fresh) / np.linalg.norm(fresh))
    print(f"[info] {name}: worst rel-L2 {max(rels):.2e}, median {np.median(rels):.2e} "
          f"(paper worst {worst:.1e})")
    assert max(rels) <= worst


@pytest.mark.parametrize("d", [64, 96, 128])
@pytest.mark.parametrize("theta", [1e4, 5e5, 1e6])
@pytest.mark.parametrize("style", [O.INTERLEAVED, O.NEOX])
def test_splice_across_rotary_widths_and_bases(L, d, theta, style):
    """Two heads, each a 32-element non-rotary part then a d-wide rotary band; a move-only plane
    beside it; random multi-directive splices of both signs, whole cache against the oracle."""
    rng = random.Random(int(d * 7 + np.log10(theta) * 13 + style))
    planes = [W.PlaneDesc((2, d + 32), 2, d + 32, 32, d, style, theta), W.PlaneDesc((64,))]
    for ci in range(2):
        n = rng.randint(700, 1500)
        cuts = sorted(rng.sample(range(n + 1), 6))
        dirs = [W.Dir(cuts[i], cuts[i + 1], rng.choice([0, 3, cuts[i + 1] - cuts[i] + 40]))
                for i in range(0, 6, 2)]
        grow = max(0, sum(x.stub_len - (x.span_end - x.span_start) for x in dirs))
        wl = W.Workload("sweep", 2, "bf16", planes, dirs, [n], capacity=n + grow,
                        seed=rng.randint(0, 10 ** 6))
        print(f"[case] sweep d={d} theta={theta:g} style={style} case={ci} n={n} dirs={dirs}", flush=True)
        planes_dev, stubs_dev = W.alloc_contig(wl, DEV)
        _splice_and_check(L, wl, planes_dev, stubs_dev, [None, None], f"d={d} theta={theta:g}")


def _oplane(desc, freqs=None):
    row = desc.row_elems
    return O.Plane(row_elems=row, n_heads=desc.n_heads, head_stride=desc.head_stride or row,
                   rot_offset=desc.rot_offset, rot_dim=desc.rot_dim, style=desc.style, base=desc.base,
                   freqs=None if freqs is None else np.asarray(freqs, dtype=np.float64))


def _splice_and_check(L, wl, planes_dev, stubs_dev, inv_freqs, label):
    before = [host(t) for t in planes_dev]
    stubs_h = [[host(s) for s in per] for per in stubs_dev]
    oplanes = [_oplane(p, fq) for p, fq in zip(wl.planes, inv_freqs)]
    cache = L.make_cache([_spec(L, t, op, fq) for t, op, fq in zip(planes_dev, oplanes, inv_freqs)])
    dirs = L.make_directives([dict(span_start=x.span_start, span_end=x.span_end, stub=stubs_dev[j],
                                   stub_len=x.stub_len) for j, x in enumerate(wl.dirs)])
    n = wl.seq_lens[0]
    new_len = L.leyline_splice_contig(cache, n, dirs, len(wl.dirs))
    torch.cuda.synchronize()
    odirs = [O.Directive(x.span_start, x.span_end, x.stub_len) for x in wl.dirs]
    assert new_len == O.new_length(n, odirs)
    for pi, op in enumerate(oplanes):
        got = host(planes_dev[pi]).reshape(wl.n_layers, wl.capacity, op.row_elems)
        src = before[pi].reshape(wl.n_layers, wl.capacity, op.row_elems)
        stubs = [s[pi].reshape(wl.n_layers, s[pi].shape[1], op.row_elems) for s in stubs_h]
        want, _ = O.splice_contig(src, n, odirs, stubs, op, wl.dtype)
        assert_rows_match(got[:, :new_len], want[:, :new_len], op, wl.dtype, what=f"{label} plane {pi}")


def _yarn_like(rot_dim, base, factor=40.0, lo=4, hi=24):
    """A caller-given frequency table: the RoFormer schedule with its low frequencies divided by
    `factor`, blended linearly across pairs [lo, hi) (the shape of an NTK/YaRN-style
    interpolation; any table is allowed, this one exercises non-geometric frequencies)."""
    f = O.rope_frequencies(rot_dim, base)
    i = np.arange(rot_dim // 2, dtype=np.float64)
    ramp = np.clip((i - lo) / (hi - lo), 0.0, 1.0)
    return f * (1.0 - ramp) + (f / factor) * ramp


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_caller_frequency_table(L, dtype):
    """inv_freq given by the caller: contiguous splice, in-place rotation, token-slot splice."""
    rng = random.Random(5 if dtype == "bf16" else 6)
    mla = W.mla_plane()
    gqa_k, gqa_v = W.gqa_planes(heads=2, dim=128)
    for kind, planes in (("mla", [mla]), ("gqa", [gqa_k, gqa_v])):
        freqs = [_yarn_like(p.rot_dim, p.base) if p.rot_dim else None for p in planes]
        inv = [None if fq is None else [float(x) for x in fq] for fq in freqs]
        # contiguous splice
        n = 1200
        dirs = [W.Dir(100, 400, 17), W.Dir(700, 701, 90)]
        wl = W.Workload("yarn", 2, dtype, planes, dirs, [n], capacity=n, seed=rng.randint(0, 10 ** 6))
        print(f"[case] inv_freq {kind}/{dtype} contiguous splice", flush=True)
        planes_dev, stubs_dev = W.alloc_contig(wl, DEV)
        _splice_and_check(L, wl, planes_dev, stubs_dev, inv, f"inv_freq {kind}")
        # in-place rotation of a row range
        print(f"[case] inv_freq {kind}/{dtype} rotate", flush=True)
        oplanes = [_oplane(p, fq) for p, fq in zip(planes, inv)]
        before = [host(t) for t in planes_dev]
        cache = L.make_cache([_spec(L, t, op, fq) for t, op, fq in zip(planes_dev, oplanes, inv)])
        L.leyline_rotate_delta(cache, 4531, row0=10, n_rows=500)
        torch.cuda.synchronize()
        for pi, op in enumerate(oplanes):
            b = before[pi].reshape(2, n, op.row_elems)
            want = b.copy()
            for layer in range(2):
                want[layer, 10:510] = O.rotate_rows(b[layer, 10:510], 4531, op, dtype)
            got = host(planes_dev[pi]).reshape(2, n, op.row_elems)
            assert_rows_match(got, want, op, dtype, inputs=b, what=f"inv_freq rotate {kind}")
        # token-slot (page size 1) splice: downstream bands rotated in place
        print(f"[case] inv_freq {kind}/{dtype} token slots", flush=True)
        wl = W.Workload("yarn_slots", 2, dtype, planes, [W.Dir(50, 300, 5)], [800], page_size=1,
                        seed=rng.randint(0, 10 ** 6))
        pools, bt, free, stubs = W.alloc_paged(wl, DEV, spare_pages=3)
        pool_h = [host(p) for p in pools]
        stubs_h = [[host(s).reshape(2, s.shape[1], op.row_elems) for s, op in zip(per, oplanes)]
                   for per in stubs]
        cache = L.make_cache([_spec(L, t, op, fq) for t, op, fq in zip(pools, oplanes, inv)], paged=True)
        d = L.make_directives([dict(span_start=50, span_end=300, stub=stubs[0], stub_len=5)])
        new_lens, fresh, n_freed, ws_bytes = L.leyline_paged_query(cache, [800], bt.shape[1], d, 1)
        bt_out = torch.empty_like(bt)
        freed = torch.empty(max(1, n_freed), dtype=torch.int32, device=DEV)
        ws = torch.empty(max(256, ws_bytes), dtype=torch.uint8, device=DEV)
        L.leyline_splice_paged(cache, [800], bt, bt_out, d, 1, free, freed, ws)
        torch.cuda.synchronize()
        flat = [x.reshape(x.shape[0], x.shape[1], x.shape[2], -1) for x in pool_h]
        want, want_bt, want_lens, want_freed = O.splice_paged(
            flat, oplanes, dtype, host(bt), [800], [O.Directive(50, 300, 5)], stubs_h, list(host(free)), 1)
        assert np.array_equal(host(bt_out), want_bt) and new_lens == want_lens
        for pi, op in enumerate(oplanes):
            got = host(pools[pi]).reshape(want[pi].shape)
            assert_rows_match(got, want[pi], op, dtype, what=f"inv_freq slots {kind} plane {pi}")


# Table "drift": mean rel-L2 against fresh RoPE after N chained rotations (the paper's path also
# rounded cos/sin to bf16; ours keeps them in fp32, so these are upper bounds).
DRIFT_BOUND = {2: 4.3e-3, 5: 5.6e-3, 10: 7.5e-3, 20: 1.1e-2, 50: 1.7e-2, 100: 2.6e-2}


@pytest.mark.parametrize("style", [O.INTERLEAVED, O.NEOX])
def test_chained_rotations_step_by_step(L, style):
    """K = [batch 8, heads 32, head_dim 64] bf16, RoPE'd at 8192; N in-place rotations by signed
    shifts in [-512, 512] on the GPU.  Every step matches the oracle applied to the GPU's previous
    state; the drift against fresh RoPE at the final position, averaged over 10 seeds, stays
    within Table "drift"."""
    heads, d, batch = 32, 64, 8
    plane = O.Plane(row_elems=heads * d, n_heads=heads, head_stride=d, rot_offset=0, rot_dim=d,
                    style=style, base=10000.0)
    f = plane.frequencies()
    drift = {n: [] for n in DRIFT_BOUND}
    for seed in range(10):
        rng = np.random.default_rng(300 + seed)
        raw = rng.standard_normal((len(DRIFT_BOUND) * batch * heads, d))
        p0 = 8192
        t = device(O.encode(O.rope(raw, p0, f, style), O.BF16).reshape(len(DRIFT_BOUND) * batch, heads * d),
                   DEV).view(1, len(DRIFT_BOUND) * batch, heads * d)
        cache = L.make_cache([_spec(L, t, plane)])
        pos = {n: p0 for n in DRIFT_BOUND}
        prev = host(t).reshape(-1, heads * d)
        for step in range(max(DRIFT_BOUND)):
            shifts = {}
            for c, n in enumerate(DRIFT_BOUND):
                if step < n:
                    dl = int(rng.integers(-512, 513))
                    dl = max(-pos[n], dl)
                    shifts[c] = dl
                    pos[n] += dl
                    L.leyline_rotate_delta(cache, dl, row0=c * batch, n_rows=batch)
            torch.cuda.synchronize()
            cur = host(t).reshape(-1, heads * d)
            want = prev.copy()
            for c, dl in shifts.items():
                want[c * batch:(c + 1) * batch] = O.rotate_rows(prev[c * batch:(c + 1) * batch], dl, plane, O.BF16)
            assert_rows_match(cur, want, plane, O.BF16, inputs=prev, what=f"seed {seed} step {step}")
            prev = cur
        for c, n in enumerate(DRIFT_BOUND):
            g = O.decode(prev[c * batch:(c + 1) * batch], O.BF16).reshape(batch * heads, d)
            fresh = O.rope(raw.reshape(len(DRIFT_BOUND), batch * heads, d)[c], pos[n], f, style)
            drift[n].append(np.linalg.norm(g - fresh) / np.linalg.norm(fresh))
    for n, bound in DRIFT_BOUND.items():
        mean = float(np.mean(drift[n]))
        print(f"[info] style {style}: N={n} mean rel-L2 {mean:.2e} (paper {bound:.1e})")
        assert mean <= bound


FLOOR_SOURCES = (10, 100, 1000, 4000, 8000, 8836)
FLOOR_DELTAS = (1, -1, 48, -48, 512, 2000, 6794, -6794)


@pytest.mark.parametrize("dtype", [O.F32, O.BF16])
def test_precision_floor_sweep(L, dtype):
    """App. "bf16 K-storage precision floor": MLA K_pe keys RoPE'd at sources {10, ..., 8836}
    (theta 1e4, interleaved) and re-anchored in place by shifts up to |6794|, against a fresh fp64
    RoPE at p + delta, per entry relative to its pair's norm.  fp32 storage stays at fp32
    rounding at every (p, delta): angles are formed in fp64 (the paper's fp32 path, with fp32
    angles, grew to 1.6e-3 at (8836, 6794)).  bf16 storage sits at the storage floor (the
    stored key's rounding plus the result's, under 3 bf16 half-steps), the same for every
    shift."""
    plane = O.mla_plane()
    f = plane.frequencies()
    rng = np.random.default_rng(77)
    per = 64
    src = np.repeat(np.array(FLOOR_SOURCES), per)
    n = len(src)
    raw = rng.standard_normal((n, 64))
    rows = np.zeros((n, 576))
    rows[:, :512] = rng.standard_normal((n, 512))
    rows[:, 512:] = O.rope(raw, src, f, O.INTERLEAVED)
    stored = O.encode(rows, dtype)
    t = device(stored, DEV).view(1, n, 576)
    cache = L.make_cache([_spec(L, t, plane)])
    worst = {}
    for dl in FLOOR_DELTAS:
        t.copy_(device(stored, DEV).view(1, n, 576))
        print(f"[case] floor {dtype} delta={dl}", flush=True)
        L.leyline_rotate_delta(cache, dl, row0=0, n_rows=n)
        torch.cuda.synchronize()
        out = host(t).reshape(n, 576)
        assert np.array_equal(out[:, :512], stored[:, :512])                 # latent untouched
        got = O.decode(out[:, 512:], dtype)
        fresh = O.rope(raw, src + dl, f, O.INTERLEAVED)
        pair = np.repeat(np.hypot(fresh[:, 0::2], fresh[:, 1::2]), 2, axis=1)
        err = (np.abs(got - fresh) / pair).reshape(len(FLOOR_SOURCES), per, 64).max(axis=(1, 2))
        for p, e in zip(FLOOR_SOURCES, err):
            worst[(p, dl)] = float(e)
    print("[info] worst per-entry error / pair norm:", {k: f"{v:.2e}" for k, v in worst.items()})
    if dtype == O.F32:
        assert max(worst.values()) < 1e-5
    else:
        assert max(worst.values()) < 3 * 2.0 ** -8
        small = max(v for (p, dl), v in worst.items() if abs(dl) == 1)
        large = max(v for (p, dl), v in worst.items() if abs(dl) == 6794)
        assert large < 1.5 * small                                           # independent of delta
