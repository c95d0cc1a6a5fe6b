"""The every-row rotary check of the GPU tests (parity_util.assert_bands_rotated), on the CPU: it
accepts the oracle's own rotated rows (bf16 and fp32 storage, both pairings, shifts of both signs,
pairs that nearly cancel) and rejects a row with one member two ulps off, so that its bar is
implied by, and close to, the oracle comparison of assert_rows_match."""

import numpy as np
import pytest
import torch

from oracle import splice_oracle as O
from tests.parity_util import angle_tables, assert_bands_rotated, device, rotary_mask


def _case(dtype, style, seed):
    rng = np.random.default_rng(seed)
    plane = O.Plane(row_elems=192, n_heads=2, head_stride=96, rot_offset=32, rot_dim=64, style=style, base=10000.0)
    n = 600
    x = rng.standard_normal((n, plane.row_elems))
    x[:40, :] *= 1e-3                                   # small pairs
    ia, ib = O.pair_dims(plane.rot_dim, plane.style)
    near = x[40:80]                                     # pairs that nearly cancel after rotation
    near[:, 32 + ib] = near[:, 32 + ia] * (1 + 1e-3 * rng.standard_normal((40, len(ia))))
    rows = O.encode(x, dtype)
    shifts = rng.choice([-4064, -1, 1, 7, 300, 2023], size=n)
    want = np.empty_like(rows)
    for c in np.unique(shifts):
        sel = shifts == c
        want[sel] = O.rotate_rows(rows[sel], int(c), plane, dtype)
    rot = rotary_mask(plane)
    return plane, rows, want, shifts, rot


@pytest.mark.parametrize("dtype", [O.BF16, O.F32])
@pytest.mark.parametrize("style", [O.INTERLEAVED, O.NEOX])
def test_oracle_rows_pass_and_two_ulp_errors_fail(dtype, style):
    plane, rows, want, shifts, rot = _case(dtype, style, 7 + style + (dtype == O.F32))
    tables = angle_tables(plane, shifts, "cpu")
    before = device(np.ascontiguousarray(rows[:, rot]), "cpu")
    assert_bands_rotated(before, device(np.ascontiguousarray(want[:, rot]), "cpu"), tables, dtype, "oracle rows")
    # one member of one pair moved past the oracle's bar (two ulps for bf16; 4e-6 of the pair's
    # norm for fp32, whose bar is 2e-6 of it) must be caught
    out = np.ascontiguousarray(want[:, rot])
    vals = O.decode(out, dtype)
    half = plane.rot_dim // 2
    for r, c in ((3, 0), (250, 17), (599, 63), (123, 100)):
        j = c % plane.rot_dim
        partner = c - j + ((j ^ 1) if style == O.INTERLEAVED else (j + half) % plane.rot_dim)
        norm = np.hypot(vals[r, c], vals[r, partner])
        v = vals[r, c]
        step = 2 * O.ulp(np.array([v]), dtype)[0] if dtype == O.BF16 else 4e-6 * norm
        bad = out.copy()
        bad[r, c] = O.encode(np.array([[v + (1.0 if v >= 0 else -1.0) * step]]), dtype)[0, 0]
        with pytest.raises(AssertionError):
            assert_bands_rotated(before, device(bad, "cpu"), tables, dtype, "planted")
