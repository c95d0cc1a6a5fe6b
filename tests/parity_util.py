"""Helpers shared by the GPU parity tests: host snapshots of device tensors, oracle plane specs
built from workload descriptions, and the tolerance checks.

Tolerances (the bar of the splice's parity tests):
* every non-rotary element and every index/table: bit-exact;
* rotary elements stored in bf16: |gpu - oracle| <= 1 bf16 ulp of the oracle value (the GPU
  rounds an fp32 result once, the oracle rounds the fp64 value once);
* rotary elements stored in fp32: per rotary pair, ||gpu - oracle|| <= 2e-6 * ||input pair||
  (rotations preserve the pair norm, so this is the relative error of the fp32 compute).
"""

import numpy as np
import torch

from oracle import splice_oracle as O

F32_PAIR_RTOL = 2e-6


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
    if dtype == O.BF16:
        err = np.abs(g - w)
        tol = O.ulp(w, O.BF16)
        if not np.all(err <= tol):
            bad = np.argwhere(err > tol)
            raise AssertionError(f"{what}: bf16 rotary error beyond 1 ulp at {bad[:5].tolist()} "
                                 f"({len(bad)} total, max err {err.max():.3g})")
        return
    src = w if inputs is None else O.decode(inputs[..., rot], dtype)
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
