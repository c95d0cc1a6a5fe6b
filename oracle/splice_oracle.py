"""CPU oracle for Leyline's in-place KV-cache splice -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of ``bench.py`` may
import or call this module.  The product path (the HIP library under ``paper_2606_01065_amd``
and its Python binding) never does, and this module imports nothing from it.

What is computed, and where the paper defines it
-------------------------------------------------
* A directive replaces the cached token span ``[s, e)`` by a replacement of ``r`` tokens; every
  token downstream of the span moves by ``Delta = r - (e - s)`` (Sec. 3.1, "The directive").
* Only the rotary band of a moved key is modified: it is re-anchored with the closed-form
  rotation ``k' = R(Delta) k`` (Eq. "rotate", Sec. 3.2).  The latent / K_nope and V data of the
  moved rows are copied unchanged (Sec. 3.1 "Which tensors are modified"; App. "Kernel
  specification: tensors and composition", step (c)).
* The replacement's K/V come from an ordinary prefill at its final positions (App. "Kernel
  specification", step (b)); here it is an input, copied verbatim and never rotated.
* Several non-overlapping directives per call are processed left to right with a running
  (cumulative) shift of either sign; overlapping spans are rejected (App. "Kernel
  specification", paragraph on multiple directives).
* RoPE pairs are either interleaved (dims 2i, 2i+1) or half-split / NEOX (dims i, i+d/2)
  (Sec. 3.3 "RoPE pairing convention"; App. "RoPE pairing convention").
* Rotation arithmetic is carried out in higher precision than storage and rounded on the way
  back to the bf16 pool (Sec. 4.1 "bf16 K-storage precision floor"; App. "bf16 K-storage
  precision floor").  Here: float64 angles, float64 trig, float64 pair products, one
  round-to-nearest-even to the storage dtype.  The frequencies, cosines and sines come from the
  scalar functions of the platform's C math library (Python's ``math``), one value at a time:
  numpy's vectorized ``power`` can differ from them in the last place, and a float64 result one
  unit off can round to a different float32 when a pair nearly cancels.

* A FORGET directive hands the edit to a prefix-trimmed re-prefill (Sec. 3.1, "The FORGET
  mode"): on the cache, the sequence is cut at the span's start after the earlier directives.

The frequency schedule ``theta_i = base ** (-2 i / d_rot)`` is RoFormer's, which the paper cites
for RoPE without restating (Sec. 3.2).

Paged caches are not described by the paper at all.  The page-kind rule below (identity /
remap / assemble, fresh pages drawn in ascending (sequence, page) order, freed pages listed in
ascending (sequence, old page) order) is this project's reading, and so is its copy-on-write
variant (no page re-used with a shift), read from the Role A/B integration of Sec. 3.3 that writes
rotated KV to fresh destination slots.  Both are pinned by invariants and by reconstruction
against the contiguous definition, not by any value in the paper.

Everything here is deliberately plain: no blocking, no fusion, no reordering beyond what the
definition states.
"""

from __future__ import annotations

import math

from dataclasses import dataclass, field
from typing import List, Optional, Sequence, Tuple

import numpy as np

INTERLEAVED = 0
NEOX = 1

BF16 = "bf16"
F32 = "f32"

IDENTITY = 0
REMAP = 1
ASSEMBLE = 2


# ----------------------------------------------------------------------------------------------
# Storage dtypes
# ----------------------------------------------------------------------------------------------

def storage_numpy_dtype(dtype: str):
    """bf16 values are held as their 16-bit patterns (uint16); f32 as float32."""
    if dtype == BF16:
        return np.uint16
    if dtype == F32:
        return np.float32
    raise ValueError(f"unknown storage dtype {dtype!r}")


def decode(stored: np.ndarray, dtype: str) -> np.ndarray:
    """Storage -> float64 (exact: every bf16 and every f32 value is a float64 value)."""
    if dtype == BF16:
        bits = np.asarray(stored, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
        return bits.view(np.float32).astype(np.float64)
    if dtype == F32:
        return np.asarray(stored, dtype=np.float32).astype(np.float64)
    raise ValueError(f"unknown storage dtype {dtype!r}")


def encode(x: np.ndarray, dtype: str) -> np.ndarray:
    """float64 -> storage, one rounding to nearest, ties to even.

    bf16 keeps 8 significant bits and float32's exponent range.  The value is rounded directly
    from float64 (no intermediate float32 rounding): the quantum of the target binade is a power
    of two, so ``x / quantum`` is exact and ``np.round`` (ties to even) performs the rounding.
    """
    x = np.asarray(x, dtype=np.float64)
    if dtype == F32:
        return x.astype(np.float32)
    if dtype != BF16:
        raise ValueError(f"unknown storage dtype {dtype!r}")
    mag = np.abs(x)
    _, e = np.frexp(mag)                      # mag = m * 2**e, m in [0.5, 1)
    e = np.maximum(e, -125)                   # below 2**-126 the quantum stays 2**-133 (subnormals)
    quantum = np.ldexp(1.0, e - 8)            # 8 significant bits
    with np.errstate(invalid="ignore", over="ignore"):
        q = np.round(mag / quantum) * quantum
    q = np.where(q >= 2.0 ** 128, np.inf, q)  # rounds past the largest finite bf16
    q = np.copysign(q, x)
    bits = (q.astype(np.float32).view(np.uint32) >> np.uint32(16)).astype(np.uint16)
    return np.where(np.isnan(x), np.uint16(0x7FC0), bits).astype(np.uint16)


def ulp(x64: np.ndarray, dtype: str) -> np.ndarray:
    """Spacing of the storage format at |x|: for a storage value x, the gap between |x| and the
    next storage value away from zero (used by tests to express tolerances).

    A binade [2**(e-1), 2**e) of bf16 holds 2**7 values (8 significant bits), so its spacing is
    2**(e-8); float32 (24 significant bits) has 2**(e-24).  Zero and the subnormals share the
    spacing of the smallest normal binade (bf16 2**-133, float32 2**-149).
    """
    mag = np.abs(np.asarray(x64, dtype=np.float64))
    _, e = np.frexp(mag)                          # mag = m * 2**e, m in [0.5, 1); frexp(0) -> e = 0
    e = np.where(mag == 0, -125, np.maximum(e, -125))
    if dtype == BF16:
        return np.ldexp(1.0, e - 8)
    if dtype == F32:
        return np.ldexp(1.0, e - 24)
    raise ValueError(dtype)


# ----------------------------------------------------------------------------------------------
# RoPE geometry
# ----------------------------------------------------------------------------------------------

def rope_frequencies(rot_dim: int, base: float) -> np.ndarray:
    """theta_i = base ** (-2 i / d_rot), i in [0, d_rot/2)  (RoFormer schedule, Sec. 3.2), each
    evaluated by the C math library's pow."""
    return np.array([math.pow(float(base), -2.0 * i / rot_dim) for i in range(rot_dim // 2)],
                    dtype=np.float64)


def _cos_sin(shift, freqs: np.ndarray) -> Tuple[np.ndarray, np.ndarray]:
    """cos and sin of phi = shift * theta_i for every shift (scalar or array) and frequency:
    [..., d_rot/2] each, every value evaluated by the C math library (once per distinct shift)."""
    shift = np.asarray(shift, dtype=np.float64)
    u, inv = np.unique(shift, return_inverse=True)
    phi = u[:, None] * freqs                                              # [distinct shifts, d_rot/2]
    c = np.array([[math.cos(x) for x in row] for row in phi.tolist()], dtype=np.float64).reshape(phi.shape)
    s = np.array([[math.sin(x) for x in row] for row in phi.tolist()], dtype=np.float64).reshape(phi.shape)
    return c[inv].reshape(shift.shape + freqs.shape), s[inv].reshape(shift.shape + freqs.shape)


def pair_dims(rot_dim: int, style: int) -> Tuple[np.ndarray, np.ndarray]:
    """Which two dims of the rotary band form pair i (Sec. 3.3, "RoPE pairing convention").

    interleaved: (2i, 2i+1);  half-split (NEOX): (i, i + d/2).
    """
    half = rot_dim // 2
    i = np.arange(half)
    if style == INTERLEAVED:
        return 2 * i, 2 * i + 1
    if style == NEOX:
        return i, i + half
    raise ValueError(f"unknown rope style {style!r}")


def rotate(band: np.ndarray, shift, freqs: np.ndarray, style: int) -> np.ndarray:
    """Apply R(shift) to rotary bands: each pair (a, b) -> (a cos phi - b sin phi, a sin phi + b cos phi),
    phi = shift * theta_i (Eq. "rotate").

    band:  float64 [..., d_rot]
    shift: scalar or array broadcastable to band[..., 0] (a position or a position delta)
    """
    band = np.asarray(band, dtype=np.float64)
    d_rot = band.shape[-1]
    ia, ib = pair_dims(d_rot, style)
    c, s = _cos_sin(shift, freqs)                                         # [..., d_rot/2]
    a, b = band[..., ia], band[..., ib]
    out = np.empty(np.broadcast_shapes(band.shape, c.shape[:-1] + (d_rot,)), dtype=np.float64)
    out[..., ia] = a * c - b * s
    out[..., ib] = a * s + b * c
    return out


def rope(raw: np.ndarray, positions, freqs: np.ndarray, style: int) -> np.ndarray:
    """RoPE at absolute positions: RoPE(x, p) = R(p) x.  Used to build keys 'RoPE'd at their
    original position' and for the brute-force re-application checks."""
    return rotate(raw, positions, freqs, style)


@dataclass
class Plane:
    """One tensor family stored per token per layer (MLA: one plane; GQA: K and V planes).

    A row holds ``row_elems`` elements.  Heads ``h < n_heads`` start at ``h * head_stride`` and
    carry a rotary band of ``rot_dim`` elements at ``rot_offset`` within the head; ``rot_dim = 0``
    means the plane is moved only (latent c_kv is a non-rotary part of an MLA row; V is a plane
    with no rotary band).
    """
    row_elems: int
    n_heads: int = 1
    head_stride: int = 0
    rot_offset: int = 0
    rot_dim: int = 0
    style: int = INTERLEAVED
    base: float = 10000.0
    freqs: Optional[np.ndarray] = None

    def frequencies(self) -> np.ndarray:
        if self.freqs is not None:
            return np.asarray(self.freqs, dtype=np.float64)
        return rope_frequencies(self.rot_dim, self.base)

    def rotary_columns(self) -> List[np.ndarray]:
        """Row-element indices of each head's rotary band."""
        return [h * self.head_stride + self.rot_offset + np.arange(self.rot_dim)
                for h in range(self.n_heads)] if self.rot_dim else []


def mla_plane(base: float = 10000.0, kv_lora_rank: int = 512, rope_dim: int = 64,
              style: int = INTERLEAVED) -> Plane:
    """MLA row: latent c_kv[kv_lora_rank] then K_pe[rope_dim] (Sec. 3.2; DeepSeek layout)."""
    row = kv_lora_rank + rope_dim
    return Plane(row_elems=row, n_heads=1, head_stride=row, rot_offset=kv_lora_rank,
                 rot_dim=rope_dim, style=style, base=base)


def gqa_planes(n_kv_heads: int = 8, head_dim: int = 128, base: float = 500000.0,
               style: int = NEOX) -> List[Plane]:
    """GQA: K rotated over the whole head, V moved only (Sec. 6, "Extension to GQA and MHA")."""
    row = n_kv_heads * head_dim
    k = Plane(row_elems=row, n_heads=n_kv_heads, head_stride=head_dim, rot_offset=0,
              rot_dim=head_dim, style=style, base=base)
    v = Plane(row_elems=row)
    return [k, v]


def rotate_rows(rows: np.ndarray, shift, plane: Plane, dtype: str) -> np.ndarray:
    """R(shift) on every rotary band of storage rows [n, row_elems]; all other elements copied."""
    out = np.array(rows, copy=True)
    if plane.rot_dim == 0 or len(out) == 0:
        return out
    freqs = plane.frequencies()
    for cols in plane.rotary_columns():
        band = decode(rows[:, cols], dtype)
        out[:, cols] = encode(rotate(band, shift, freqs, plane.style), dtype)
    return out


# ----------------------------------------------------------------------------------------------
# Directives (Sec. 3.1; App. "Kernel specification: tensors and composition")
# ----------------------------------------------------------------------------------------------

AMORTIZE, FORGET = 0, 1     # directive modes (Sec. 3.1)


@dataclass
class Directive:
    span_start: int
    span_end: int
    stub_len: int
    seq: int = 0
    mode: int = AMORTIZE

    @property
    def delta(self) -> int:
        """Delta = |R| - (s_end - s_start)  (Sec. 3.1)."""
        return self.stub_len - (self.span_end - self.span_start)


class DirectiveError(ValueError):
    pass


def resolve_forget(n: int, dirs: Sequence[Directive]) -> List[Directive]:
    """FORGET (Sec. 3.1, "The FORGET mode") hands the edit to a prefix-trimmed re-prefill: the
    cache keeps what precedes the span and everything from the span start on is computed again
    by the model.  On the cache this is the deletion of [span_start, n) with no replacement.
    A FORGET directive must be the last of its sequence and carry no replacement KV (the
    replacement is part of what is re-prefilled)."""
    out = list(dirs)
    for j, d in enumerate(out):
        if d.mode == FORGET:
            if j != len(out) - 1:
                raise DirectiveError("a FORGET directive must be the last of its sequence")
            if d.stub_len != 0:
                raise DirectiveError("a FORGET directive carries no replacement")
            if not (0 <= d.span_start <= d.span_end <= n):
                raise DirectiveError(f"span [{d.span_start},{d.span_end}) outside [0,{n}]")
            out[j] = Directive(d.span_start, n, 0, d.seq)
        elif d.mode != AMORTIZE:
            raise DirectiveError("unknown mode")
    return out


def check_directives(n: int, dirs: Sequence[Directive]) -> None:
    """Ranges inside [0, n], sorted by span start, non-overlapping (adjacent allowed), |R| >= 0.
    Overlap is rejected at apply time (App. "Kernel specification", multiple directives)."""
    prev_end = 0
    for d in dirs:
        if not (0 <= d.span_start <= d.span_end <= n):
            raise DirectiveError(f"span [{d.span_start},{d.span_end}) outside [0,{n}]")
        if d.stub_len < 0:
            raise DirectiveError("negative stub length")
        if d.span_start < prev_end:
            raise DirectiveError("spans overlap or are not sorted")
        prev_end = d.span_end


def row_sources(n: int, dirs: Sequence[Directive]) -> List[tuple]:
    """Where each new row comes from, in new-position order.

    ('old', p, delta)  -> old row p, shifted by the cumulative delta of its segment
    ('stub', j, t)     -> token t of directive j's replacement
    """
    dirs = resolve_forget(n, dirs)
    check_directives(n, dirs)
    out: List[tuple] = []
    shift = 0
    cursor = 0
    for j, d in enumerate(dirs):
        for p in range(cursor, d.span_start):
            out.append(("old", p, shift))
        for t in range(d.stub_len):
            out.append(("stub", j, t))
        shift += d.delta
        cursor = d.span_end
    for p in range(cursor, n):
        out.append(("old", p, shift))
    return out


def new_length(n: int, dirs: Sequence[Directive]) -> int:
    return n + sum(d.delta for d in resolve_forget(n, dirs))


def splice_rows(rows: np.ndarray, n: int, dirs: Sequence[Directive],
                stubs: Sequence[np.ndarray], plane: Plane, dtype: str) -> np.ndarray:
    """One layer, one plane, logical rows: the plain definition of the splice.

    new = old[0:s1] ++ stub_1 ++ R(delta_1) old[e1:s2] ++ stub_2 ++ ... ++ R(delta_k) old[ek:n]
    with delta_j the running sum of the directives' Deltas.  Non-rotary elements are copied
    bit-for-bit; rotary bands are rotated in float64 and rounded once.
    """
    dirs = resolve_forget(n, dirs)
    check_directives(n, dirs)
    pieces = []
    shift = 0
    cursor = 0
    for j, d in enumerate(dirs):
        pieces.append(rotate_rows(rows[cursor:d.span_start], shift, plane, dtype))
        stub = np.asarray(stubs[j])
        if stub.shape[0] != d.stub_len:
            raise DirectiveError("stub rows do not match stub_len")
        pieces.append(np.array(stub, copy=True))
        shift += d.delta
        cursor = d.span_end
    pieces.append(rotate_rows(rows[cursor:n], shift, plane, dtype))
    if not pieces:
        return rows[:0].copy()
    return np.concatenate(pieces, axis=0)


def splice_contig(cache: np.ndarray, n: int, dirs: Sequence[Directive],
                  stubs: Sequence[np.ndarray], plane: Plane, dtype: str) -> Tuple[np.ndarray, int]:
    """Contiguous cache of one plane, storage [L, capacity, row_elems]; stubs[j] is
    [L, r_j, row_elems].  Returns (new cache, n').  Rows [n', capacity) keep whatever they held
    (their content after a splice is unspecified and never compared)."""
    n_new = new_length(n, dirs)
    if n_new > cache.shape[1]:
        raise DirectiveError("new length exceeds capacity")
    out = np.array(cache, copy=True)
    for layer in range(cache.shape[0]):
        out[layer, :n_new] = splice_rows(cache[layer], n, dirs, [s[layer] for s in stubs],
                                         plane, dtype)
    return out, n_new


def splice_sequential(cache: np.ndarray, n: int, dirs: Sequence[Directive],
                      stubs: Sequence[np.ndarray], plane: Plane, dtype: str) -> Tuple[np.ndarray, int]:
    """Multi-directive reference by sequential application (App. "Kernel specification"):
    directive j is applied alone to the result of directives < j, its span translated by the
    running shift.  Rows are carried in float64 between steps (one rounding at the end)."""
    dirs = resolve_forget(n, dirs)
    check_directives(n, dirs)
    n_layers = cache.shape[0]
    freqs = plane.frequencies() if plane.rot_dim else None
    cols = plane.rotary_columns()
    out = np.array(cache, copy=True)
    for layer in range(n_layers):
        cur = decode(cache[layer, :n], dtype)      # float64 rows
        running = 0
        for j, d in enumerate(dirs):
            s, e = d.span_start + running, d.span_end + running
            moved = cur[e:].copy()
            for c in cols:
                moved[:, c] = rotate(moved[:, c], d.delta, freqs, plane.style)
            cur = np.concatenate([cur[:s], decode(stubs[j][layer], dtype), moved], axis=0)
            running += d.delta
        out[layer, :len(cur)] = encode(cur, dtype)
    return out, new_length(n, dirs)


# ----------------------------------------------------------------------------------------------
# Paged caches (this project's reading; the paper describes no paging)
# ----------------------------------------------------------------------------------------------

@dataclass
class SeqPlan:
    old_len: int
    new_len: int
    kinds: List[int] = field(default_factory=list)     # per new logical page
    sources: List[int] = field(default_factory=list)   # old logical page (identity/remap) or fresh ordinal
    deltas: List[int] = field(default_factory=list)    # remap: the shift applied in place
    freed: List[int] = field(default_factory=list)     # old logical pages dropped


def pages_for(n: int, page: int) -> int:
    return (n + page - 1) // page


def plan_sequence(n: int, dirs: Sequence[Directive], page: int, fresh_base: int,
                  remap: bool = True) -> SeqPlan:
    """Page plan of one sequence.

    New logical page k is
      IDENTITY if every valid row comes from old row at the same position (shift 0);
      REMAP    if every valid row comes from one old page k' at the same in-page offset with one
               nonzero shift (necessarily a multiple of the page size): the page is re-used and only
               its rotary bands are rotated in place;
      ASSEMBLE otherwise: its rows are gathered into the next fresh page.
    Old pages referenced by neither an identity nor a remap page are freed.

    remap=False (copy-on-write, for pools whose pages other sequences share) never re-uses a page
    whose rows shift: such pages are assembled into fresh pages and no old page is written, as
    the paper's Role A/B integration writes the rotated downstream KV into fresh destination
    slots and leaves the originals to their other owners (Sec. 3.3, "Role B").
    """
    src = row_sources(n, dirs)
    n_new = len(src)
    plan = SeqPlan(old_len=n, new_len=n_new)
    kept = set()
    fresh = fresh_base
    for k in range(pages_for(n_new, page)):
        rows = src[k * page:min((k + 1) * page, n_new)]
        offs = range(k * page, k * page + len(rows))
        if all(r[0] == "old" and r[2] == 0 and r[1] == q for r, q in zip(rows, offs)):
            plan.kinds.append(IDENTITY)
            plan.sources.append(k)
            plan.deltas.append(0)
            kept.add(k)
            continue
        if remap and all(r[0] == "old" for r in rows):
            shifts = {r[2] for r in rows}
            old_pages = {r[1] // page for r in rows}
            same_off = all(r[1] % page == q % page for r, q in zip(rows, offs))
            if len(shifts) == 1 and len(old_pages) == 1 and same_off:
                kp = old_pages.pop()
                plan.kinds.append(REMAP)
                plan.sources.append(kp)
                plan.deltas.append(shifts.pop())
                kept.add(kp)
                continue
        plan.kinds.append(ASSEMBLE)
        plan.sources.append(fresh)
        plan.deltas.append(0)
        fresh += 1
    plan.freed = [kp for kp in range(pages_for(n, page)) if kp not in kept]
    return plan


def plan_paged(seq_lens: Sequence[int], dirs: Sequence[Directive], page: int,
               remap: bool = True) -> List[SeqPlan]:
    """Plans for all sequences; fresh ordinals run in ascending (sequence, new page) order.
    ``dirs`` is sorted by (seq, span_start)."""
    by_seq = [[d for d in dirs if d.seq == b] for b in range(len(seq_lens))]
    for b in range(1, len(dirs)):
        if (dirs[b].seq, dirs[b].span_start) < (dirs[b - 1].seq, dirs[b - 1].span_start):
            raise DirectiveError("directives not sorted by (seq, span_start)")
    plans = []
    fresh = 0
    for b, n in enumerate(seq_lens):
        p = plan_sequence(int(n), by_seq[b], page, fresh, remap)
        fresh += sum(1 for k in p.kinds if k == ASSEMBLE)
        plans.append(p)
    return plans


def gather_logical(pool: np.ndarray, layer: int, bt_row: np.ndarray, n: int, page: int) -> np.ndarray:
    """Logical rows [0, n) of one sequence, read through its block table."""
    idx = np.arange(n)
    return pool[layer, bt_row[idx // page], idx % page]


def paged_tables(block_table: np.ndarray, seq_lens: Sequence[int], dirs: Sequence[Directive],
                 free_pages: Sequence[int], page: int, remap: bool = True):
    """New block table (entries past a sequence's last page = -1), new lengths, the freed
    physical pages, and the plans, from the page plan and the old block table."""
    plans = plan_paged(seq_lens, dirs, page, remap)
    bt_out = np.full_like(block_table, -1)
    freed: List[int] = []
    for b, plan in enumerate(plans):
        if pages_for(plan.new_len, page) > block_table.shape[1]:
            raise DirectiveError("block table row too short for the new length")
        for k, (kind, srcp) in enumerate(zip(plan.kinds, plan.sources)):
            if kind == ASSEMBLE:
                if srcp >= len(free_pages):
                    raise DirectiveError("not enough free pages")
                bt_out[b, k] = free_pages[srcp]
            else:
                bt_out[b, k] = block_table[b, srcp]
        freed.extend(int(block_table[b, kp]) for kp in plan.freed)
    return bt_out, [p.new_len for p in plans], freed, plans


def splice_paged(pools: Sequence[np.ndarray], planes: Sequence[Plane], dtype: str,
                 block_table: np.ndarray, seq_lens: Sequence[int], dirs: Sequence[Directive],
                 stubs: Sequence[Sequence[np.ndarray]], free_pages: Sequence[int], page: int,
                 remap: bool = True):
    """Paged splice (remap=False: copy-on-write, see plan_sequence).

    pools[plane]:      storage [L, n_pool_pages, page, row_elems]
    block_table:       int32 [n_seqs, bt_stride] (old physical pages per logical page)
    stubs[j][plane]:   storage [L, r_j, row_elems]
    free_pages:        physical pages that ASSEMBLE pages draw from, in order

    Returns (new pools, new block table (unused entries = -1), new lengths, freed physical pages).
    Rows at or past the new length inside the last page of a sequence are unspecified.
    """
    bt_out, new_lens, freed, plans = paged_tables(block_table, seq_lens, dirs, free_pages, page, remap)
    out = [np.array(p, copy=True) for p in pools]
    for b, plan in enumerate(plans):
        my_dirs = [d for d in dirs if d.seq == b]
        my_stubs = [stubs[i] for i, d in enumerate(dirs) if d.seq == b]
        for pi, plane in enumerate(planes):
            for layer in range(pools[pi].shape[0]):
                old_rows = gather_logical(pools[pi], layer, block_table[b], plan.old_len, page)
                new_rows = splice_rows(old_rows, plan.old_len, my_dirs,
                                       [s[pi][layer] for s in my_stubs], plane, dtype)
                for k, kind in enumerate(plan.kinds):
                    if kind == IDENTITY:
                        continue
                    lo, hi = k * page, min((k + 1) * page, plan.new_len)
                    out[pi][layer, bt_out[b, k], :hi - lo] = new_rows[lo:hi]
    return out, bt_out, new_lens, freed
