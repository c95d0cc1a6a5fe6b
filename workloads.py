"""Seeded synthetic inputs shaped like the paper's splice workloads.

Shared by the tests, the benchmark and the smoke check.  This module only draws directive
positions (integers) and fills tensors with seeded N(0,1) values; it performs none of the
splice's or RoPE's arithmetic.  Keys that the workloads describe as "RoPE'd at their original
position" are drawn directly from N(0,1): a rotation of an isotropic Gaussian pair is again an
isotropic Gaussian pair, so the stored values have the described distribution.  Tests that need
the exact construction (raw key, then RoPE at its position) build it themselves.

Workloads (MLA rows: latent c_kv[512] + K_pe[64]; GQA rows: 8 KV heads x 128):
  mla_1l_4k_f32       1 layer, 4096 tokens, fp32, delete [1024,1536), 16-token stub
  mla_dsv3_32k        61 layers, 32768 tokens, bf16, 4096-token span at a seeded start in
                      [2048,16384), 32-token stub, contiguous in place
  mla_dsv3_paged_b64  61 layers, 64-token pages, 64 sequences of U[2048,32768] tokens, one
                      directive each (start in the first half, span U[64,4096], stub U[0,64])
  gqa_llama3_8b_16k   32 layers, K and V 8x128 bf16, theta 5e5 half-split, 16384 tokens,
                      delete [4096,6144), 24-token stub
  mla_dsv3_paged_131k 61 layers, 64-token pages, one 131072-token sequence, 8 non-overlapping
                      directives (spans U[256,8192], stubs U[0,64])
  mla_dsv3_paged_131k_inorder
                      the same with the pool's pages handed out in order (placement study)
  mla_dsv3_32k_edits8 the 32K MLA cache with 8 seeded edits (spans U[8,200], stubs U[0,2*span])
  mla_dsv3_32k_shift1 the 32K MLA cache with one token deleted (every downstream row moves by one)
  mla_dsv3_slots_32k, gqa_llama3_8b_slots_16k
                      the 32K MLA and 16K GQA splices on token-slot caches (page size 1)
  mla_dsv3_slots_cow_32k
                      the 32K MLA token-slot splice with copy-on-write (fresh slots downstream)
  mla_dsv3_rotate_32k, gqa_llama3_8b_rotate_16k
                      re-anchoring in place without movement: the downstream rows of the 32K MLA
                      and 16K GQA splices rotated by their shifts
  mla_dsv3_slots_rotate_32k
                      the same on a token-slot cache: the 32K MLA splice's downstream slots,
                      listed by physical slot, rotated in place
  mla_dsv3_32k_split, mla_dsv3_slots_split_32k, mla_dsv3_rotate_split_32k
                      the 32K MLA splice (contiguous, token slots) and in-place re-anchoring on a
                      cache that keeps K_pe[64] and c_kv[512] in two arrays (layout study)
"""

from __future__ import annotations

from dataclasses import dataclass, field
from typing import List, Tuple

import numpy as np
import torch

MLA_LATENT, MLA_ROPE = 512, 64


@dataclass
class PlaneDesc:
    row_shape: Tuple[int, ...]
    n_heads: int = 1
    head_stride: int = 0
    rot_offset: int = 0
    rot_dim: int = 0
    style: int = 0                # 0 interleaved, 1 half-split (NEOX)
    base: float = 10000.0

    @property
    def row_elems(self) -> int:
        return int(np.prod(self.row_shape))


@dataclass
class Dir:
    span_start: int
    span_end: int
    stub_len: int
    seq: int = 0
    mode: int = 0                 # 0 AMORTIZE, 1 FORGET


@dataclass
class Workload:
    name: str
    n_layers: int
    dtype: str                    # "bf16" | "f32"
    planes: List[PlaneDesc]
    dirs: List[Dir]
    seq_lens: List[int]
    page_size: int = 0            # 0: contiguous
    capacity: int = 0             # contiguous rows per layer
    paged_flags: int = 0          # paged splice flags (1: copy-on-write, no old page written)
    rotate: Tuple[int, int, int] = None   # (delta, row0, n_rows): re-anchoring in place, no move
    placement: str = "permuted"   # paged: pool pages handed to sequences and the free list in a
                                  # seeded random order ("permuted") or in pool order ("in_order")
    seed: int = 0
    notes: dict = field(default_factory=dict)

    @property
    def torch_dtype(self):
        return torch.bfloat16 if self.dtype == "bf16" else torch.float32


def mla_plane(base=10000.0) -> PlaneDesc:
    row = MLA_LATENT + MLA_ROPE
    return PlaneDesc((row,), 1, row, MLA_LATENT, MLA_ROPE, 0, base)


def mla_split_planes(base=10000.0) -> List[PlaneDesc]:
    """The MLA row stored as two planes: K_pe[64] (all of it rotary) and the latent c_kv[512]."""
    return [PlaneDesc((MLA_ROPE,), 1, MLA_ROPE, 0, MLA_ROPE, 0, base), PlaneDesc((MLA_LATENT,))]


def gqa_planes(heads=8, dim=128, base=500000.0) -> List[PlaneDesc]:
    return [PlaneDesc((heads, dim), heads, dim, 0, dim, 1, base), PlaneDesc((heads, dim))]


def mla_1l_4k_f32() -> Workload:
    return Workload("mla_1l_4k_f32", 1, "f32", [mla_plane()], [Dir(1024, 1536, 16)], [4096],
                    capacity=4096, seed=1)


def mla_dsv3_32k(seed: int = 2) -> Workload:
    rng = np.random.default_rng(seed)
    s = int(rng.integers(2048, 16384))
    return Workload("mla_dsv3_32k", 61, "bf16", [mla_plane()], [Dir(s, s + 4096, 32)], [32768],
                    capacity=32768, seed=seed)


def gqa_llama3_8b_16k() -> Workload:
    return Workload("gqa_llama3_8b_16k", 32, "bf16", gqa_planes(), [Dir(4096, 6144, 24)], [16384],
                    capacity=16384, seed=4)


def mla_dsv3_paged_b64(seed: int = 3, n_seqs: int = 64, n_layers: int = 61) -> Workload:
    rng = np.random.default_rng(seed)
    lens, dirs = [], []
    for b in range(n_seqs):
        n = int(rng.integers(2048, 32769))
        s = int(rng.integers(0, n // 2))
        ln = int(rng.integers(64, 4097))
        r = int(rng.integers(0, 65))
        lens.append(n)
        dirs.append(Dir(s, min(n, s + ln), r, seq=b))
    return Workload("mla_dsv3_paged_b64", n_layers, "bf16", [mla_plane()], dirs, lens,
                    page_size=64, seed=seed)


def mla_dsv3_paged_131k(seed: int = 5, n_layers: int = 61) -> Workload:
    rng = np.random.default_rng(seed)
    n = 131072
    spans: List[Tuple[int, int]] = []
    while len(spans) < 8:
        ln = int(rng.integers(256, 8193))
        s = int(rng.integers(0, n - ln + 1))
        if all(s + ln <= a or s >= b for a, b in spans):
            spans.append((s, s + ln))
    spans.sort()
    dirs = [Dir(a, b, int(rng.integers(0, 65))) for a, b in spans]
    return Workload("mla_dsv3_paged_131k", n_layers, "bf16", [mla_plane()], dirs, [n],
                    page_size=64, seed=seed)


def mla_dsv3_paged_131k_inorder() -> Workload:
    """The 131K-token 8-directive paged splice with the pool's pages handed out in pool order (the
    sequence's pages and the free list each contiguous and ascending) instead of permuted: the
    same bytes, without scattered pages to translate."""
    w = mla_dsv3_paged_131k()
    w.name = "mla_dsv3_paged_131k_inorder"
    w.placement = "in_order"
    return w


def mla_dsv3_32k_edits8(seed: int = 6) -> Workload:
    """The 32K MLA contiguous cache with 8 non-overlapping edits in one call, drawn like the
    paper's randomized edit suite: span sizes uniform in [8, 200] tokens at uniform positions,
    replacement lengths uniform in [0, 2 * span], so shifts take both signs and stay small."""
    rng = np.random.default_rng(seed)
    n = 32768
    spans: List[Tuple[int, int]] = []
    while len(spans) < 8:
        ln = int(rng.integers(8, 201))
        s = int(rng.integers(0, n - ln + 1))
        if all(s + ln <= a or s >= b for a, b in spans):
            spans.append((s, s + ln))
    spans.sort()
    dirs = [Dir(a, b, int(rng.integers(0, 2 * (b - a) + 1))) for a, b in spans]
    grow = max(0, max(int(x) for x in np.cumsum([d.stub_len - (d.span_end - d.span_start) for d in dirs])))
    return Workload("mla_dsv3_32k_edits8", 61, "bf16", [mla_plane()], dirs, [n], capacity=n + grow,
                    seed=seed)


def mla_dsv3_32k_shift1() -> Workload:
    """The 32K MLA contiguous cache with one token deleted at the headline's seeded start and no
    replacement: every downstream row moves by one row, the smallest shift (ordered tiles)."""
    w = mla_dsv3_32k()
    s = w.dirs[0].span_start
    return Workload("mla_dsv3_32k_shift1", w.n_layers, w.dtype, w.planes, [Dir(s, s + 1, 0)], w.seq_lens,
                    capacity=w.capacity, seed=w.seed)


def mla_dsv3_slots_32k() -> Workload:
    """The 32K MLA splice on a token-slot cache (page size 1, slots scattered over the pool): the
    downstream tokens keep their slots, only their K_pe bands are rotated in place."""
    w = mla_dsv3_32k()
    return Workload("mla_dsv3_slots_32k", w.n_layers, w.dtype, w.planes, w.dirs, w.seq_lens,
                    page_size=1, seed=w.seed)


def gqa_llama3_8b_slots_16k() -> Workload:
    """The 16K GQA splice on a token-slot cache: downstream K heads rotated in place, V untouched."""
    w = gqa_llama3_8b_16k()
    return Workload("gqa_llama3_8b_slots_16k", w.n_layers, w.dtype, w.planes, w.dirs, w.seq_lens,
                    page_size=1, seed=w.seed)


def mla_dsv3_slots_cow_32k() -> Workload:
    """The 32K MLA splice on a token-slot cache with copy-on-write: every downstream token is
    rotated into a fresh slot and its old slot is left as it was (other holders of those slots,
    such as a prefix tree, keep reading the original keys)."""
    w = mla_dsv3_slots_32k()
    return Workload("mla_dsv3_slots_cow_32k", w.n_layers, w.dtype, w.planes, w.dirs, w.seq_lens,
                    page_size=1, seed=w.seed, paged_flags=1)


def mla_dsv3_rotate_32k() -> Workload:
    """Re-anchoring without movement on the 32K MLA cache: the K_pe bands of the headline
    splice's downstream rows rotated in place by its shift (rows and shift of mla_dsv3_32k)."""
    w = mla_dsv3_32k()
    d = w.dirs[0]
    n = w.seq_lens[0]
    return Workload("mla_dsv3_rotate_32k", w.n_layers, w.dtype, w.planes, [], w.seq_lens, capacity=n,
                    rotate=(d.stub_len - (d.span_end - d.span_start), d.span_end, n - d.span_end), seed=w.seed)


def mla_dsv3_slots_rotate_32k() -> Workload:
    """Re-anchoring in place on a token-slot cache, the operation of the paper's own kernel
    (K_pe of re-keyed slots rotated where they are): the downstream slots of the 32K MLA
    token-slot splice, listed by physical slot, rotated by its shift; no replacement, no tables.
    The pool is the splice's own (same slots, same placement): its directive sizes the pool and
    nothing else, so the two workloads differ only by the splice's own work."""
    w = mla_dsv3_slots_32k()
    d = w.dirs[0]
    n = w.seq_lens[0]
    return Workload("mla_dsv3_slots_rotate_32k", w.n_layers, w.dtype, w.planes, w.dirs, w.seq_lens, page_size=1,
                    rotate=(d.stub_len - (d.span_end - d.span_start), d.span_end, n - d.span_end), seed=w.seed)


def gqa_llama3_8b_rotate_16k() -> Workload:
    """Re-anchoring without movement on the 16K GQA cache: whole K rows of the downstream rows
    [6144, 16384) rotated in place by -2024, V untouched."""
    w = gqa_llama3_8b_16k()
    return Workload("gqa_llama3_8b_rotate_16k", w.n_layers, w.dtype, w.planes, [], w.seq_lens,
                    capacity=w.capacity, rotate=(-2024, 6144, 16384 - 6144), seed=w.seed)


def _split(w: Workload, name: str) -> Workload:
    w.name = name
    w.planes = mla_split_planes()
    return w


def mla_dsv3_32k_split() -> Workload:
    """mla_dsv3_32k on a cache whose K_pe and c_kv live in separate arrays (same values, same
    directive, same bytes)."""
    return _split(mla_dsv3_32k(), "mla_dsv3_32k_split")


def mla_dsv3_slots_split_32k() -> Workload:
    """mla_dsv3_slots_32k with K_pe and c_kv in separate arrays: the in-place rotation of the
    downstream slots reads and writes 128-byte K_pe rows of one array instead of 128-byte bands
    of 1152-byte rows."""
    return _split(mla_dsv3_slots_32k(), "mla_dsv3_slots_split_32k")


def mla_dsv3_rotate_split_32k() -> Workload:
    """mla_dsv3_rotate_32k with K_pe and c_kv in separate arrays."""
    return _split(mla_dsv3_rotate_32k(), "mla_dsv3_rotate_split_32k")


WORKLOADS = {
    "mla_1l_4k_f32": mla_1l_4k_f32,
    "mla_dsv3_32k": mla_dsv3_32k,
    "mla_dsv3_paged_b64": mla_dsv3_paged_b64,
    "gqa_llama3_8b_16k": gqa_llama3_8b_16k,
    "mla_dsv3_paged_131k": mla_dsv3_paged_131k,
    "mla_dsv3_paged_131k_inorder": mla_dsv3_paged_131k_inorder,
    "mla_dsv3_32k_edits8": mla_dsv3_32k_edits8,
    "mla_dsv3_32k_shift1": mla_dsv3_32k_shift1,
    "mla_dsv3_slots_32k": mla_dsv3_slots_32k,
    "gqa_llama3_8b_slots_16k": gqa_llama3_8b_slots_16k,
    "mla_dsv3_slots_cow_32k": mla_dsv3_slots_cow_32k,
    "mla_dsv3_rotate_32k": mla_dsv3_rotate_32k,
    "gqa_llama3_8b_rotate_16k": gqa_llama3_8b_rotate_16k,
    "mla_dsv3_slots_rotate_32k": mla_dsv3_slots_rotate_32k,
    "mla_dsv3_32k_split": mla_dsv3_32k_split,
    "mla_dsv3_slots_split_32k": mla_dsv3_slots_split_32k,
    "mla_dsv3_rotate_split_32k": mla_dsv3_rotate_split_32k,
}


# --------------------------------------------------------------------------------- filling ---

def fill_normal(t: torch.Tensor, seed: int, chunk_elems: int = 1 << 27) -> torch.Tensor:
    """Fill t (any float dtype, any device) with seeded N(0,1) values, generated in fp32 chunks
    along the flattened leading dims and rounded to t's dtype."""
    flat = t.view(-1)
    g = torch.Generator(device=t.device)
    g.manual_seed(seed)
    for lo in range(0, flat.numel(), chunk_elems):
        hi = min(flat.numel(), lo + chunk_elems)
        flat[lo:hi] = torch.randn(hi - lo, generator=g, device=t.device, dtype=torch.float32).to(t.dtype)
    return t


def alloc_contig(w: Workload, device, seed: int = None, fill: bool = True):
    """Returns (plane tensors [L, capacity, *row], stubs[j][plane] = [L, r_j, *row])."""
    seed = w.seed if seed is None else seed
    planes = []
    for i, p in enumerate(w.planes):
        t = torch.empty((w.n_layers, w.capacity) + p.row_shape, dtype=w.torch_dtype, device=device)
        if fill:
            fill_normal(t, seed * 1000 + i)
        planes.append(t)
    stubs = []
    for j, d in enumerate(w.dirs):
        per = []
        for i, p in enumerate(w.planes):
            t = torch.empty((w.n_layers, d.stub_len) + p.row_shape, dtype=w.torch_dtype, device=device)
            fill_normal(t, seed * 1000 + 100 + 10 * j + i)
            per.append(t)
        stubs.append(per)
    return planes, stubs


def fresh_page_bound(w: Workload) -> int:
    """Upper bound on fresh pages a paged splice can consume: every new page from the page of
    the sequence's first span start onwards."""
    P = w.page_size
    total = 0
    for b, n in enumerate(w.seq_lens):
        mine = [d for d in w.dirs if d.seq == b]
        if not mine:
            continue
        n_new = n + sum(d.stub_len - (d.span_end - d.span_start) for d in mine)
        total += -(-n_new // P) - mine[0].span_start // P
    return total


def paged_new_lens(w: Workload) -> List[int]:
    return [n + sum(d.stub_len - (d.span_end - d.span_start) for d in w.dirs if d.seq == b)
            for b, n in enumerate(w.seq_lens)]


def paged_bt_stride(w: Workload) -> int:
    """Block-table width: pages of the longer of each sequence's old and new length."""
    P = w.page_size
    return max(-(-max(n, m) // P) for n, m in zip(w.seq_lens, paged_new_lens(w)))


def alloc_paged(w: Workload, device, seed: int = None, fill: bool = True, spare_pages: int = 8):
    """Pool tensors [L, n_pool, P, *row] per plane; block table int32 [n_seqs, bt_stride] with the
    sequences' pages drawn from a seeded permutation of the pool; the rest is the free list.
    Only pages referenced by a block table are filled."""
    seed = w.seed if seed is None else seed
    P = w.page_size
    rng = np.random.default_rng(seed + 77)
    old_pages = [-(-n // P) for n in w.seq_lens]
    bt_stride = paged_bt_stride(w)
    n_used = sum(old_pages)
    n_pool = n_used + fresh_page_bound(w) + spare_pages
    perm = (rng.permutation(n_pool) if w.placement == "permuted" else np.arange(n_pool)).astype(np.int32)
    bt = np.full((len(w.seq_lens), bt_stride), -1, dtype=np.int32)
    c = 0
    for b, k in enumerate(old_pages):
        bt[b, :k] = perm[c:c + k]
        c += k
    free = perm[c:].copy()
    pools = []
    for i, p in enumerate(w.planes):
        t = torch.empty((w.n_layers, n_pool, P) + p.row_shape, dtype=w.torch_dtype, device=device)
        if fill:
            gen_seed = seed * 1000 + i
            # fill layer by layer (keeps the fp32 staging small for very large pools)
            for layer in range(w.n_layers):
                fill_normal(t[layer], gen_seed * 100 + layer)
        pools.append(t)
    stubs = []
    for j, d in enumerate(w.dirs):
        per = []
        for i, p in enumerate(w.planes):
            t = torch.empty((w.n_layers, d.stub_len) + p.row_shape, dtype=w.torch_dtype, device=device)
            fill_normal(t, seed * 1000 + 500 + 10 * j + i)
            per.append(t)
        stubs.append(per)
    return pools, torch.from_numpy(bt).to(device), torch.from_numpy(free).to(device), stubs
