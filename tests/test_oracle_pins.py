"""Pins of the CPU oracle against facts fixed by the paper and by mathematics (no GPU).

Each test checks the oracle against something other than itself: values printed or implied by
the paper (tests/golden), closed forms evaluated by a different route (complex arithmetic, the
textbook rotate-half formula), brute force with Python lists, library rounding, and invariants.
"""

import math
import os
import random

import numpy as np
import pytest
import torch

from oracle import splice_oracle as O

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _read_kv(name):
    out = {}
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            key, *vals = line.split()
            out[key] = vals
    return out


# --------------------------------------------------------------------------- index geometry ---

def test_worked_geometry_from_paper():
    g = {k: int(v[0]) for k, v in _read_kv("worked_splice_geometry.txt").items()}
    d = O.Directive(g["span_start"], g["span_end"], g["stub_len"])
    assert d.delta == g["delta"]
    assert O.new_length(g["n_old"], [d]) == g["n_new"]
    src = O.row_sources(g["n_old"], [d])
    new_pos = {r[1]: q for q, r in enumerate(src) if r[0] == "old"}
    assert new_pos[g["downstream_old_first"]] == g["downstream_new_first"]
    assert new_pos[g["downstream_old_last"]] == g["downstream_new_last"]
    assert all(new_pos[p] == p for p in range(g["span_start"]))
    assert all(new_pos[p] == p + g["delta"] for p in range(g["span_end"], g["n_old"]))
    stub_pos = [q for q, r in enumerate(src) if r[0] == "stub"]
    assert stub_pos == list(range(g["span_start"], g["span_start"] + g["stub_len"]))


def _random_dirs(rng, n, k_max=3, allow_insert=True):
    """Sorted non-overlapping directives; spans may be empty (insertions), stubs may be empty."""
    k = rng.randint(1, k_max)
    cuts = sorted(rng.sample(range(n + 1), min(2 * k, n + 1)))
    dirs = []
    for i in range(0, len(cuts) - 1, 2):
        s, e = cuts[i], cuts[i + 1]
        if not allow_insert and s == e:
            e = min(n, s + 1)
        dirs.append(O.Directive(s, e, rng.randint(0, 2 * (e - s) + 2)))
    return dirs


def test_splice_matches_python_list_brute_force():
    """Non-rotary rows: the splice is list surgery, applied right to left with del/insert."""
    rng = random.Random(11)
    plane = O.Plane(row_elems=4)
    for _ in range(300):
        n = rng.randint(0, 40)
        dirs = _random_dirs(rng, n) if n else [O.Directive(0, 0, rng.randint(0, 3))]
        rows = np.arange(n * 4, dtype=np.float32).reshape(n, 4)
        stubs = [np.full((d.stub_len, 4), -(j + 1), dtype=np.float32) for j, d in enumerate(dirs)]
        lst = [tuple(r) for r in rows]
        for j in reversed(range(len(dirs))):
            d = dirs[j]
            del lst[d.span_start:d.span_end]
            lst[d.span_start:d.span_start] = [tuple(r) for r in stubs[j]]
        got = O.splice_rows(rows, n, dirs, stubs, plane, O.F32)
        assert [tuple(r) for r in got] == lst
        assert len(got) == O.new_length(n, dirs)


def test_new_positions_are_a_bijection():
    rng = random.Random(5)
    for _ in range(200):
        n = rng.randint(1, 60)
        dirs = _random_dirs(rng, n)
        src = O.row_sources(n, dirs)
        olds = [r[1] for r in src if r[0] == "old"]
        deleted = set().union(*[set(range(d.span_start, d.span_end)) for d in dirs])
        assert sorted(olds) == [p for p in range(n) if p not in deleted]
        assert olds == sorted(olds)          # order preserved
        assert len(src) == O.new_length(n, dirs)
        # the shift recorded with a row is where it lands: new position = old position + shift
        assert all(q == r[1] + r[2] for q, r in enumerate(src) if r[0] == "old")


def test_rejects_overlap_unsorted_and_out_of_range():
    with pytest.raises(O.DirectiveError):
        O.check_directives(10, [O.Directive(2, 6, 1), O.Directive(5, 8, 0)])
    with pytest.raises(O.DirectiveError):
        O.check_directives(10, [O.Directive(5, 6, 1), O.Directive(2, 3, 0)])
    with pytest.raises(O.DirectiveError):
        O.check_directives(10, [O.Directive(5, 11, 1)])
    O.check_directives(10, [O.Directive(2, 5, 1), O.Directive(5, 8, 0)])   # adjacent is fine


# ------------------------------------------------------------------------------ rotation -----

def test_quarter_turn_pins_pairing_and_sign():
    g = _read_kv("quarter_turn.txt")
    x = np.array([float(v) for v in g["input"]])
    freqs = np.array([math.pi / 2, 0.0, 0.0, 0.0])
    for style, key in ((O.INTERLEAVED, "interleaved"), (O.NEOX, "neox")):
        want = np.array([float(v) for v in g[key]])
        got = O.rotate(x, 1, freqs, style)
        assert np.allclose(got, want, rtol=0, atol=1e-14), (key, got)


def test_interleaved_equals_complex_multiplication():
    """Interleaved RoPE = multiply the complex numbers (x[2i] + i x[2i+1]) by exp(i p theta_i)."""
    rng = np.random.default_rng(1)
    x = rng.standard_normal((50, 64))
    p = rng.integers(-5000, 5000, size=50).astype(np.float64)
    freqs = O.rope_frequencies(64, 10000.0)
    z = (x[:, 0::2] + 1j * x[:, 1::2]) * np.exp(1j * p[:, None] * freqs[None, :])
    want = np.empty_like(x)
    want[:, 0::2], want[:, 1::2] = z.real, z.imag
    assert np.max(np.abs(O.rotate(x, p, freqs, O.INTERLEAVED) - want)) < 1e-12


def test_neox_equals_rotate_half_formula():
    """Half-split RoPE in its rotate-half form: x cos + rotate_half(x) sin, with cos/sin tiled
    over both halves and rotate_half(x) = [-x2, x1]."""
    rng = np.random.default_rng(2)
    x = rng.standard_normal((40, 128))
    p = rng.integers(0, 100000, size=40).astype(np.float64)
    freqs = O.rope_frequencies(128, 500000.0)
    ang = np.concatenate([p[:, None] * freqs, p[:, None] * freqs], axis=1)
    rot_half = np.concatenate([-x[:, 64:], x[:, :64]], axis=1)
    want = x * np.cos(ang) + rot_half * np.sin(ang)
    assert np.max(np.abs(O.rotate(x, p, freqs, O.NEOX) - want)) < 1e-12


def test_frequency_schedule_values():
    f = O.rope_frequencies(64, 10000.0)
    assert f[0] == 1.0
    assert abs(f[16] - 0.01) < 1e-17                      # 10000 ** -0.5
    ratio = f[1:] / f[:-1]
    assert np.allclose(ratio, 10000.0 ** (-2 / 64), rtol=1e-14, atol=0)
    g = O.rope_frequencies(128, 500000.0)
    assert abs(g[32] - 500000.0 ** -0.5) < 1e-18


@pytest.mark.parametrize("style", [O.INTERLEAVED, O.NEOX])
def test_composition_and_identity(style):
    rng = np.random.default_rng(3)
    x = rng.standard_normal((30, 64))
    f = O.rope_frequencies(64, 10000.0)
    for a, b in [(1, 2), (-496, 4064), (2000, -2000), (131071, -65536)]:
        lhs = O.rotate(O.rotate(x, b, f, style), a, f, style)
        rhs = O.rotate(x, a + b, f, style)
        assert np.max(np.abs(lhs - rhs)) < 1e-9 * max(1, abs(a) + abs(b)) / 1000 + 1e-11
    assert np.array_equal(O.rotate(x, 0, f, style), x)


@pytest.mark.parametrize("style", [O.INTERLEAVED, O.NEOX])
def test_attention_scores_depend_only_on_relative_position(style):
    rng = np.random.default_rng(4)
    f = O.rope_frequencies(64, 10000.0)
    q, k = rng.standard_normal(64), rng.standard_normal(64)
    for m, n, d in [(300, 100, -46), (5000, 4000, -4064), (10, 9, 2000)]:
        before = O.rope(q, m, f, style) @ O.rope(k, n, f, style)
        after = O.rope(q, m + d, f, style) @ O.rotate(O.rope(k, n, f, style), d, f, style)
        assert abs(before - after) < 1e-11


@pytest.mark.parametrize("style", [O.INTERLEAVED, O.NEOX])
def test_splice_reanchors_to_fresh_rope_at_new_position(style):
    """Keys built as RoPE(raw, p) in f32 storage; after the splice each moved key must equal
    RoPE(raw, p + delta) up to f32 storage rounding (closure R(a)R(b) = R(a+b), Sec. 3.2)."""
    rng = np.random.default_rng(5)
    plane = O.mla_plane(style=style)
    n = 400
    raw = rng.standard_normal((n, 64))
    rows = np.zeros((n, plane.row_elems), dtype=np.float32)
    rows[:, :512] = rng.standard_normal((n, 512)).astype(np.float32)
    f = plane.frequencies()
    rows[:, 512:] = O.encode(O.rope(raw, np.arange(n), f, style), O.F32)
    d = O.Directive(100, 196, 16)
    stub = np.zeros((16, plane.row_elems), dtype=np.float32)
    out = O.splice_rows(rows, n, [d], [stub], plane, O.F32)
    new_pos = np.arange(d.span_end, n) + d.delta
    fresh = O.rope(raw[d.span_end:], new_pos, f, style)
    got = O.decode(out[new_pos, 512:], O.F32)
    err = np.abs(got - fresh)
    # input rounding (<= 0.5 ulp of |x|) carried through an isometry plus one output rounding
    assert np.all(err <= 2 * O.ulp(fresh, O.F32) + 2 * np.abs(fresh).max() * 2 ** -24)
    assert np.array_equal(out[new_pos, :512], rows[d.span_end:, :512])     # latent untouched


def test_mismatched_pairing_hides_at_small_delta_and_grows():
    """The failure mode described in App. "RoPE pairing convention": rotating an interleaved key
    with half-split pairing is nearly right for tiny shifts and wrong for large ones."""
    rng = np.random.default_rng(6)
    f = O.rope_frequencies(64, 10000.0)
    raw = rng.standard_normal((64, 64))
    key = O.rope(raw, 1000, f, O.INTERLEAVED)
    errs = []
    for d in (1, 21, 48, 76, 512, 2000):       # the shift set validated in Sec. 3.3
        good = O.rotate(key, d, f, O.INTERLEAVED)
        bad = O.rotate(key, d, f, O.NEOX)
        assert np.max(np.abs(good - O.rope(raw, 1000 + d, f, O.INTERLEAVED))) < 1e-10
        errs.append(np.linalg.norm(bad - good) / np.linalg.norm(good))
    assert errs[0] < errs[-1]
    assert errs[-1] > 0.1


# ----------------------------------------------------------------------------- rounding -----

def test_bf16_encode_matches_torch_round_to_nearest_even():
    rng = np.random.default_rng(7)
    x = np.concatenate([
        rng.standard_normal(200000).astype(np.float32),
        (rng.standard_normal(2000) * 1e-39).astype(np.float32),           # subnormals
        (rng.standard_normal(2000) * 1e38).astype(np.float32),
        np.array([0.0, -0.0, 1.0, -1.0, 3.3895314e38], dtype=np.float32),
    ])
    want = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    got = O.encode(x.astype(np.float64), O.BF16)
    assert np.array_equal(got, want)


def test_bf16_ties_round_to_even():
    one = 1.0
    assert O.encode(np.array([one + 2 ** -8]), O.BF16)[0] == 0x3F80          # halfway -> even (1.0)
    assert O.encode(np.array([one + 3 * 2 ** -8]), O.BF16)[0] == 0x3F82      # halfway -> even
    assert O.encode(np.array([one + 2 ** -8 + 2 ** -40]), O.BF16)[0] == 0x3F81  # above half -> up
    assert O.encode(np.array([2.0 ** -133]), O.BF16)[0] == 0x0001             # smallest subnormal
    assert np.array_equal(O.decode(O.encode(np.array([-2.5, 0.15625]), O.BF16), O.BF16),
                          [-2.5, 0.15625])


def _bf16_values(bits: np.ndarray) -> np.ndarray:
    """bf16 bit patterns -> float64 through torch's own bf16 type (not the oracle's decode)."""
    t = torch.from_numpy(np.asarray(bits, dtype=np.uint16).view(np.int16)).view(torch.bfloat16)
    return t.to(torch.float64).numpy()


def test_bf16_ulp_is_the_gap_to_the_next_value():
    """ulp() sets every bf16 parity tolerance (the one-ulp bar of App. "bf16 K-storage precision
    floor").  For every finite non-negative bf16 pattern b (zero and subnormals included),
    ulp(value(b)) must equal value(b + 1) - value(b), and ulp(-x) must equal ulp(x)."""
    b = np.arange(0, 0x7F7F, dtype=np.uint16)            # 0 .. one below the largest finite
    x = _bf16_values(b)
    gap = _bf16_values(b + 1) - x
    assert np.array_equal(O.ulp(x, O.BF16), gap)
    assert np.array_equal(O.ulp(-x, O.BF16), gap)
    assert O.ulp(np.array([0.0]), O.BF16)[0] == 2.0 ** -133
    assert O.ulp(np.array([1.0]), O.BF16)[0] == 2.0 ** -7


def test_f32_ulp_is_the_gap_to_the_next_value():
    """The same for float32 storage, against numpy's nextafter: random finite patterns, every
    binade edge (2**k and its predecessor), subnormals and zero."""
    rng = np.random.default_rng(21)
    bits = rng.integers(0, 0x7F7FFFFF, size=200000, dtype=np.uint32)
    edges = np.ldexp(np.float32(1.0), np.arange(-149, 128)).astype(np.float32)
    below = np.nextafter(edges, np.float32(0.0))
    x = np.concatenate([bits.view(np.float32), edges, below, np.float32([0.0, 1e-45, 1e-40, 1.0, 3.0])])
    gap = np.nextafter(x, np.float32(np.inf)).astype(np.float64) - x.astype(np.float64)
    assert np.array_equal(O.ulp(x.astype(np.float64), O.F32), gap)
    assert np.array_equal(O.ulp(-x.astype(np.float64), O.F32), gap)


def test_delta_zero_segment_is_bit_identical():
    rng = np.random.default_rng(8)
    plane = O.mla_plane()
    rows = O.encode(rng.standard_normal((64, 576)), O.BF16)
    d = O.Directive(10, 20, 10)             # Delta = 0: downstream rows must not change at all
    stub = O.encode(rng.standard_normal((10, 576)), O.BF16)
    out = O.splice_rows(rows, 64, [d], [stub], plane, O.BF16)
    assert np.array_equal(out[20:], rows[20:]) and np.array_equal(out[:10], rows[:10])
    assert np.array_equal(out[10:20], stub)


def test_chained_bf16_drift_order_of_magnitude():
    """Chained rotations with a bf16 store after each step drift slowly and sub-linearly
    (App. "Chained-rotation drift", Table "drift": 4.3e-3 rel-L2 at N=2, 2.6e-2 at N=100 for a
    path that also rounds cos/sin to bf16).  Rounding once per step from float64 must stay at or
    below those magnitudes and grow sub-linearly."""
    rng = np.random.default_rng(9)
    f = O.rope_frequencies(64, 10000.0)
    raw = rng.standard_normal((8 * 32, 64))
    res = {}
    for n_chain in (2, 100):
        pos = 4096
        cur = O.encode(O.rope(raw, pos, f, O.INTERLEAVED), O.BF16)
        for _ in range(n_chain):
            d = int(rng.integers(-512, 513))
            d = max(-pos, d)
            cur = O.encode(O.rotate(O.decode(cur, O.BF16), d, f, O.INTERLEAVED), O.BF16)
            pos += d
        fresh = O.rope(raw, pos, f, O.INTERLEAVED)
        res[n_chain] = np.linalg.norm(O.decode(cur, O.BF16) - fresh) / np.linalg.norm(fresh)
    assert 1e-4 < res[2] <= 4.3e-3
    assert res[100] <= 2.6e-2
    assert res[100] / res[2] < 50


# ------------------------------------------------------------------------- multi-directive ---

def test_one_call_equals_sequential_application():
    rng = random.Random(12)
    nrng = np.random.default_rng(12)
    for style, dtype in ((O.INTERLEAVED, O.BF16), (O.NEOX, O.F32)):
        plane = O.Plane(row_elems=48, n_heads=2, head_stride=24, rot_offset=8, rot_dim=16,
                        style=style, base=10000.0)
        for _ in range(25):
            n = rng.randint(20, 120)
            dirs = _random_dirs(rng, n, k_max=4)
            cap = n + sum(max(0, d.delta) for d in dirs) + 5
            cache = O.encode(nrng.standard_normal((2, cap, 48)), dtype)
            stubs = [O.encode(nrng.standard_normal((2, d.stub_len, 48)), dtype) for d in dirs]
            a, na = O.splice_contig(cache, n, dirs, stubs, plane, dtype)
            b, nb = O.splice_sequential(cache, n, dirs, stubs, plane, dtype)
            assert na == nb
            va, vb = O.decode(a[:, :na], dtype), O.decode(b[:, :nb], dtype)
            assert np.all(np.abs(va - vb) <= O.ulp(vb, dtype))


# ------------------------------------------------------------------------------------ paged --

def _paged_case(rng, nrng, n_seqs, page, dtype, plane, max_len=300, dirs_per_seq=2, remap=True):
    seq_lens = [rng.randint(1, max_len) for _ in range(n_seqs)]
    dirs = []
    for b, n in enumerate(seq_lens):
        for d in _random_dirs(rng, n, k_max=dirs_per_seq):
            d.seq = b
            dirs.append(d)
    plans = O.plan_paged(seq_lens, dirs, page, remap)
    bt_stride = max(max(O.pages_for(n, page), O.pages_for(p.new_len, page))
                    for n, p in zip(seq_lens, plans)) + 1
    used = sum(O.pages_for(n, page) for n in seq_lens)
    fresh = sum(k == O.ASSEMBLE for p in plans for k in p.kinds)
    n_pool = used + fresh + 3
    perm = nrng.permutation(n_pool)
    bt = np.full((n_seqs, bt_stride), -1, dtype=np.int32)
    c = 0
    for b, n in enumerate(seq_lens):
        for k in range(O.pages_for(n, page)):
            bt[b, k] = perm[c]
            c += 1
    free = [int(x) for x in perm[c:]]
    pool = O.encode(nrng.standard_normal((2, n_pool, page, plane.row_elems)), dtype)
    stubs = [[O.encode(nrng.standard_normal((2, d.stub_len, plane.row_elems)), dtype)] for d in dirs]
    return seq_lens, dirs, bt, free, pool, stubs


def test_paged_invariants_and_reconstruction():
    rng = random.Random(21)
    nrng = np.random.default_rng(21)
    plane = O.Plane(row_elems=16, n_heads=1, head_stride=16, rot_offset=8, rot_dim=8,
                    style=O.INTERLEAVED, base=10000.0)
    for page in (4, 8):
        for _ in range(20):
            seq_lens, dirs, bt, free, pool, stubs = _paged_case(rng, nrng, 3, page, O.BF16, plane,
                                                                max_len=60)
            (out,), bt_out, new_lens, freed = O.splice_paged(
                [pool], [plane], O.BF16, bt, seq_lens, dirs, stubs, free, page)
            referenced = [int(x) for x in bt_out.ravel() if x >= 0]
            assert len(referenced) == len(set(referenced))                     # unique pages
            old = {int(bt[b, k]) for b, n in enumerate(seq_lens) for k in range(O.pages_for(n, page))}
            used_fresh = set(referenced) - old
            assert used_fresh == set(free[:len(used_fresh)])
            assert set(referenced) | set(freed) == old | used_fresh            # nothing lost
            assert not (set(referenced) & set(freed))
            for plan in O.plan_paged(seq_lens, dirs, page):
                for k, (kind, src, delta) in enumerate(zip(plan.kinds, plan.sources, plan.deltas)):
                    if kind == O.IDENTITY:
                        assert src == k and delta == 0
                    elif kind == O.REMAP:                   # a whole page moved by whole pages
                        assert delta == (k - src) * page and delta != 0
            for b, n in enumerate(seq_lens):
                my = [d for d in dirs if d.seq == b]
                my_st = [stubs[i][0] for i, d in enumerate(dirs) if d.seq == b]
                assert O.pages_for(new_lens[b], page) == int((bt_out[b] >= 0).sum())
                for layer in range(2):
                    want = O.splice_rows(O.gather_logical(pool, layer, bt[b], n, page), n, my,
                                         [s[layer] for s in my_st], plane, O.BF16)
                    got = O.gather_logical(out, layer, bt_out[b], new_lens[b], page)
                    assert np.array_equal(got, want)


def test_paged_remap_only_for_whole_page_shifts():
    page = 8
    # delete exactly two pages' worth of tokens at a page boundary: downstream pages remap.
    dirs = [O.Directive(16, 32, 0)]
    (plan,) = O.plan_paged([64], dirs, page)
    assert plan.kinds[:2] == [O.IDENTITY, O.IDENTITY]
    assert plan.kinds[2:] == [O.REMAP] * 4 and plan.sources[2:] == [4, 5, 6, 7]
    assert plan.deltas[2:] == [-16] * 4
    assert plan.freed == [2, 3]
    # a shift that is not a multiple of the page size forces assembly of every downstream page
    (plan,) = O.plan_paged([64], [O.Directive(16, 33, 0)], page)
    assert plan.kinds[:2] == [O.IDENTITY, O.IDENTITY]
    assert all(k == O.ASSEMBLE for k in plan.kinds[2:])
    assert plan.freed == [2, 3, 4, 5, 6, 7]
    # a replacement of equal length leaves downstream pages in place (shift 0)
    (plan,) = O.plan_paged([64], [O.Directive(16, 20, 4)], page)
    assert plan.kinds == [O.IDENTITY, O.IDENTITY, O.ASSEMBLE] + [O.IDENTITY] * 5
    assert plan.freed == [2]


# ---------------------------------------------------------------------------- FORGET, copy-on-write

def test_forget_is_a_prefix_trim_after_the_earlier_edits():
    """FORGET hands the edit to a prefix-trimmed re-prefill (Sec. 3.1, "The FORGET mode"): with
    list surgery, the earlier directives are applied and the list is cut at the FORGET span's
    start (in post-edit coordinates); nothing from the span on is kept."""
    rng = random.Random(41)
    plane = O.Plane(row_elems=4)
    for _ in range(200):
        n = rng.randint(1, 40)
        dirs = _random_dirs(rng, n)
        tail_lo = dirs[-1].span_end if dirs else 0
        s = rng.randint(tail_lo, n)
        e = rng.randint(s, n)
        dirs = dirs + [O.Directive(s, e, 0, mode=O.FORGET)]
        rows = np.arange(n * 4, dtype=np.float32).reshape(n, 4)
        stubs = [np.full((d.stub_len, 4), -(j + 1), dtype=np.float32) for j, d in enumerate(dirs)]
        lst = [tuple(r) for r in rows]
        del lst[s:]                                   # the FORGET cut, in pre-call coordinates
        for j in reversed(range(len(dirs) - 1)):
            d = dirs[j]
            del lst[d.span_start:d.span_end]
            lst[d.span_start:d.span_start] = [tuple(r) for r in stubs[j]]
        got = O.splice_rows(rows, n, dirs, stubs, plane, O.F32)
        assert [tuple(r) for r in got] == lst
        assert O.new_length(n, dirs) == len(lst)


def test_forget_must_be_last_and_carry_no_replacement():
    with pytest.raises(O.DirectiveError):
        O.row_sources(20, [O.Directive(2, 4, 0, mode=O.FORGET), O.Directive(6, 8, 1)])
    # an insertion at the very end would not overlap the trimmed tail: refused all the same
    with pytest.raises(O.DirectiveError):
        O.row_sources(20, [O.Directive(2, 4, 0, mode=O.FORGET), O.Directive(20, 20, 1)])
    with pytest.raises(O.DirectiveError):
        O.row_sources(20, [O.Directive(2, 4, 3, mode=O.FORGET)])
    assert O.new_length(20, [O.Directive(5, 9, 0, mode=O.FORGET)]) == 5


def test_copy_on_write_plan_writes_no_old_page():
    """remap=False: no page is re-used with a shift, so every old page in the new tables keeps
    its contents bit for bit, and the logical content equals the in-place plan's."""
    rng = random.Random(43)
    nrng = np.random.default_rng(43)
    plane = O.Plane(row_elems=16, n_heads=1, head_stride=16, rot_offset=8, rot_dim=8,
                    style=O.INTERLEAVED, base=10000.0)
    for page in (1, 4, 8):
        for _ in range(15):
            seq_lens, dirs, bt, free, pool, stubs = _paged_case(rng, nrng, 3, page, O.BF16, plane,
                                                                max_len=60, remap=False)
            (cow,), bt_c, lens_c, freed_c = O.splice_paged([pool], [plane], O.BF16, bt, seq_lens, dirs,
                                                           stubs, free, page, remap=False)
            (inp,), bt_i, lens_i, _ = O.splice_paged([pool], [plane], O.BF16, bt, seq_lens, dirs,
                                                     stubs, free, page)
            plans = O.plan_paged(seq_lens, dirs, page, remap=False)
            assert all(k != O.REMAP for p in plans for k in p.kinds)
            assert any(k == O.REMAP for p in O.plan_paged(seq_lens, dirs, page) for k in p.kinds) or page > 1
            old = {int(bt[b, k]) for b, n in enumerate(seq_lens) for k in range(O.pages_for(n, page))}
            for pg in old:
                assert np.array_equal(cow[:, pg], pool[:, pg])               # old pages untouched
            assert lens_c == lens_i
            for b in range(len(seq_lens)):
                for layer in range(2):
                    a = O.gather_logical(cow, layer, bt_c[b], lens_c[b], page)
                    c = O.gather_logical(inp, layer, bt_i[b], lens_i[b], page)
                    assert np.array_equal(a, c)
