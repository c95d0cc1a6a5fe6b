"""Helpers shared by the GPU parity tests: host snapshots of device tensors, oracle plane specs
built from workload descriptions, and the tolerance checks.

Tolerances (the bar of the splice's parity tests):
* every non-rotary element and every index/table: bit-exact;
* rotary elements, fp32 storage: per rotary pair, ||gpu - oracle|| <= 2e-6 * ||input pair||
  (rotations preserve the pair norm, so this is the relative error of the fp32 compute);
* rotary elements, bf16 storage: per element, |gpu - oracle| <= max(1 bf16 ulp of the oracle
  value, 2e-6 * ||pair||).  The rotation is computed in fp32 and rounded once; the oracle is
  exact and rounded once.  When a pair's rotated component nearly cancels (e.g. (0.32, -1.98)
  turning into (-2.0, 1.4e-6)), the fp32 compute error (about 1e-7 of the pair norm) exceeds the
  bf16 spacing of that tiny component, so the 2e-6-of-fp32-compute arm applies; everywhere else
  the 1-ulp arm does.  The fraction of bf16 elements that are bit-identical is reported too.
"""

import numpy as np
import torch

from oracle import splice_oracle as O

F32_PAIR_RTOL = 2e-6
LAST_BF16_EXACT_FRACTION = None


def pair_norms(vals: np.ndarray, plane: O.Plane, rot: np.ndarray) -> np.ndarray:
    """For every rotary element (in the compressed rotary selection), the norm of its pair."""
    out = np.empty_like(vals)
    sel_all = np.flatnonzero(rot)
    ia, ib = O.pair_dims(plane.rot_dim, plane.style)
    for cols in plane.rotary_columns():
        sel = np.searchsorted(sel_all, cols)
        nrm = np.hypot(vals[..., sel[ia]], vals[..., sel[ib]])
        out[..., sel[ia]] = nrm
        out[..., sel[ib]] = nrm
    return out


def host(t: torch.Tensor) -> np.ndarray:
    """Device tensor -> numpy in oracle storage form (bf16 as uint16 bit patterns)."""
    t = t.detach().cpu()
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).numpy().view(np.uint16)
    if t.dtype == torch.float32:
        return t.numpy()
    return t.numpy()


def device(a: np.ndarray, dev) -> torch.Tensor:
    if a.dtype == np.uint16:
        return torch.from_numpy(a.view(np.int16)).view(torch.bfloat16).to(dev)
    return torch.from_numpy(a).to(dev)


def oracle_plane(desc) -> O.Plane:
    row = int(np.prod(desc.row_shape))
    return O.Plane(row_elems=row, n_heads=desc.n_heads, head_stride=desc.head_stride or row,
                   rot_offset=desc.rot_offset, rot_dim=desc.rot_dim, style=desc.style, base=desc.base)


def rotary_mask(plane: O.Plane) -> np.ndarray:
    m = np.zeros(plane.row_elems, dtype=bool)
    for cols in plane.rotary_columns():
        m[cols] = True
    return m


def assert_rows_match(got: np.ndarray, want: np.ndarray, plane: O.Plane, dtype: str,
                      inputs: np.ndarray = None, what: str = "") -> None:
    """got/want: storage arrays [..., row_elems].  inputs: the pre-splice rows whose rotation
    produced `want` (needed for the fp32 pair-relative bound; defaults to `want`)."""
    assert got.shape == want.shape, (what, got.shape, want.shape)
    rot = rotary_mask(plane)
    plain = ~rot
    if not np.array_equal(got[..., plain], want[..., plain]):
        bad = np.argwhere(got[..., plain] != want[..., plain])
        raise AssertionError(f"{what}: non-rotary mismatch at {bad[:5].tolist()} ({len(bad)} total)")
    if not rot.any():
        return
    g = O.decode(got[..., rot], dtype)
    w = O.decode(want[..., rot], dtype)
    src = w if inputs is None else O.decode(inputs[..., rot], dtype)
    norms = pair_norms(src, plane, rot)
    if dtype == O.BF16:
        err = np.abs(g - w)
        tol = np.maximum(O.ulp(w, O.BF16), F32_PAIR_RTOL * norms)
        if not np.all(err <= tol):
            bad = np.argwhere(err > tol)
            raise AssertionError(f"{what}: bf16 rotary error beyond max(1 ulp, 2e-6 |pair|) at "
                                 f"{bad[:5].tolist()} ({len(bad)} total, max err {err.max():.3g})")
        global LAST_BF16_EXACT_FRACTION
        same = got[..., rot] == want[..., rot]
        LAST_BF16_EXACT_FRACTION = float(np.mean(same)) if same.size else None
        return
    for cols in plane.rotary_columns():
        # positions of this head's band inside the compressed rotary selection
        sel = np.searchsorted(np.flatnonzero(rot), cols)
        ia, ib = O.pair_dims(plane.rot_dim, plane.style)
        ga, gb = g[..., sel[ia]], g[..., sel[ib]]
        wa, wb = w[..., sel[ia]], w[..., sel[ib]]
        sa, sb = src[..., sel[ia]], src[..., sel[ib]]
        num = np.hypot(ga - wa, gb - wb)
        den = np.hypot(sa, sb)
        ok = num <= F32_PAIR_RTOL * den + 1e-30
        if not np.all(ok):
            bad = np.argwhere(~ok)
            raise AssertionError(f"{what}: fp32 pair error above {F32_PAIR_RTOL} at {bad[:5].tolist()}")


def angle_tables(plane: O.Plane, shifts: np.ndarray, dev):
    """For rows moved by `shifts` (one per row, nonzero): the columns of every pair's two members
    within the plane's rotary selection (all heads), and cos/sin of every (row, pair) angle
    phi = shift * theta_i, taken from the oracle's rotation of unit pairs (one evaluation per
    distinct shift)."""
    uniq, which = np.unique(np.asarray(shifts, dtype=np.int64), return_inverse=True)
    ia, ib = O.pair_dims(plane.rot_dim, plane.style)
    unit = np.zeros((len(uniq), plane.rot_dim))
    unit[:, ia] = 1.0
    turned = O.rotate(unit, uniq, plane.frequencies(), plane.style)       # (cos, sin) per pair
    heads = range(plane.n_heads)
    cs = np.concatenate([turned[:, ia] for _ in heads], axis=1)[which]
    sn = np.concatenate([turned[:, ib] for _ in heads], axis=1)[which]
    cols = lambda x: torch.from_numpy(np.concatenate([x + h * plane.rot_dim for h in heads])).to(dev)
    return cols(ia), cols(ib), torch.from_numpy(cs).to(dev), torch.from_numpy(sn).to(dev)


def ulp_t(x: torch.Tensor, dtype: str) -> torch.Tensor:
    """Device twin of the oracle's ulp(): the spacing of the storage dtype at |x| (fp64 tensor),
    with zero and subnormals at the subnormal quantum."""
    _, e = torch.frexp(x)
    e = torch.where(x == 0, torch.full_like(e, -125), torch.clamp(e, min=-125))
    return torch.ldexp(torch.ones_like(x), e - (8 if dtype == O.BF16 else 24))


def assert_bands_rotated(before: torch.Tensor, after: torch.Tensor, tables, dtype: str, what: str = "") -> None:
    """before/after: rotary selections [rows, n_rot] of moved rows (device, storage dtype).  Every
    member of every pair must lie within 1.5 storage ulps of the exact rotation of its stored input
    (fp64 products with the oracle's cos/sin of the pair's angle, `tables`), or within
    2e-6 |pair| + 0.5 ulp where the pair nearly cancels.  An output within the oracle's bar (1 ulp
    of the oracle's rounded value, or 2e-6 |pair|; assert_rows_match) always passes: the rounded
    value lies within half an ulp of the exact one, and the ulp is taken of |exact| (1 + 2^-7) so
    that a value rounded up into the next binade is covered."""
    ia, ib, cs, sn = tables
    bm, gm = before.double(), after.double()
    a, b = bm[:, ia], bm[:, ib]
    norm = torch.sqrt(a * a + b * b)
    for name, want, got in (("first", a * cs - b * sn, gm[:, ia]), ("second", a * sn + b * cs, gm[:, ib])):
        u = ulp_t(want.abs() * (1.0 + 2.0 ** -7), dtype)
        tol = torch.maximum(1.5 * u, F32_PAIR_RTOL * norm + 0.5 * u)
        err = (got - want).abs()
        ok = err <= tol
        if not bool(ok.all()):
            bad = torch.nonzero(~ok)[:5].tolist()
            raise AssertionError(f"{what}: {name} pair members beyond 1.5 ulp of the exact rotation at {bad} "
                                 f"({int((~ok).sum())} total, max err/tol {float((err / tol).max()):.3g})")


def bits(t: torch.Tensor) -> torch.Tensor:
    """Bit patterns of a bf16 or fp32 device tensor, for exact comparison."""
    return t.contiguous().view(torch.int16 if t.dtype == torch.bfloat16 else torch.int32)

