"""Planted mistakes in the oracle must be caught by its pins (no GPU).

Each mutant edits one function of the oracle's source in memory -- a flipped sign, swapped
operands, a dropped term, an off-by-one index or range, another rounding mode, a relaxed check,
a running shift that does not accumulate -- re-executes it in the oracle module's namespace, and
runs the pins of tests/test_oracle_pins.py against the mutated oracle: at least one pin must
fail.  The file on disk is never changed and every mutant is undone after its test.
"""

import inspect
import textwrap

import pytest

from oracle import splice_oracle as O
from tests import test_oracle_pins as PINS

# (function or class of the oracle, original snippet, planted mistake, what the mistake is)
MUTANTS = [
    # the rotation of Eq. "rotate"
    ("rotate", "out[..., ib] = a * s + b * c", "out[..., ib] = a * s - b * c", "sign of the second component"),
    ("rotate", "out[..., ia] = a * c - b * s", "out[..., ia] = a * c + b * s", "sign of the first component"),
    ("rotate", "out[..., ia] = a * c - b * s", "out[..., ia] = a * c", "dropped cross term"),
    ("rotate", "c, s = _cos_sin(shift, freqs)", "s, c = _cos_sin(shift, freqs)", "cos and sin swapped"),
    ("_cos_sin", "s = np.array([[math.sin(x) for x in row] for row in phi.tolist()], dtype=np.float64)",
     "s = np.array([[math.sin(-x) for x in row] for row in phi.tolist()], dtype=np.float64)",
     "sin of the negated angle"),
    ("_cos_sin", "return c[inv].reshape(shift.shape + freqs.shape), s[inv]",
     "return c[inv[::-1]].reshape(shift.shape + freqs.shape), s[inv]", "cos taken for other shifts"),
    ("rotate", "a, b = band[..., ia], band[..., ib]", "b, a = band[..., ia], band[..., ib]", "pair operands transposed"),
    ("_cos_sin", "phi = u[:, None] * freqs", "phi = u[:, None] * freqs[::-1]", "frequency index reversed"),
    # pairing convention (Sec. 3.3)
    ("pair_dims", "return 2 * i, 2 * i + 1", "return i, i + half", "interleaved paired as half-split"),
    ("pair_dims", "return i, i + half", "return 2 * i, 2 * i + 1", "half-split paired as interleaved"),
    ("pair_dims", "return i, i + half", "return i + half, i", "half-split pair members swapped"),
    # frequency schedule
    ("rope_frequencies", "-2.0 * i / rot_dim", "-1.0 * i / rot_dim", "exponent missing its factor 2"),
    ("rope_frequencies", "for i in range(rot_dim // 2)]",
     "for i in range(1, rot_dim // 2 + 1)]", "frequency index off by one"),
    # the directive and its signed shift (Sec. 3.1)
    ("Directive", "return self.stub_len - (self.span_end - self.span_start)",
     "return (self.span_end - self.span_start) - self.stub_len", "sign of Delta"),
    ("Directive", "return self.stub_len - (self.span_end - self.span_start)",
     "return self.stub_len - (self.span_end - self.span_start) + 1", "Delta off by one"),
    # the splice of one layer (list concatenation with running shifts)
    ("splice_rows", "pieces.append(rotate_rows(rows[cursor:d.span_start], shift, plane, dtype))",
     "pieces.append(rotate_rows(rows[cursor:d.span_start], shift + d.delta, plane, dtype))",
     "segment rotated by the next running shift"),
    ("splice_rows", "pieces.append(rotate_rows(rows[cursor:n], shift, plane, dtype))",
     "pieces.append(rotate_rows(rows[cursor:n], 0, plane, dtype))", "last segment not re-anchored"),
    ("splice_rows", "cursor = d.span_end", "cursor = d.span_start", "span not deleted"),
    ("splice_rows", "shift += d.delta", "shift = d.delta", "shift not cumulative"),
    ("row_sources", "cursor = d.span_end", "cursor = d.span_end + 1", "first downstream row dropped"),
    ("row_sources", "shift += d.delta", "shift = d.delta", "shift not cumulative (positions)"),
    ("rotate_rows", "rotate(band, shift, freqs, plane.style)", "rotate(band, -shift, freqs, plane.style)",
     "rotation by the opposite shift"),
    ("splice_sequential", "s, e = d.span_start + running, d.span_end + running",
     "s, e = d.span_start, d.span_end", "sequential reference not translated by the running shift"),
    # storage rounding
    ("encode", "q = np.round(mag / quantum) * quantum", "q = np.floor(mag / quantum) * quantum",
     "bf16 truncation instead of round to nearest even"),
    ("encode", "q = np.round(mag / quantum) * quantum", "q = np.floor(mag / quantum + 0.5) * quantum",
     "bf16 ties away from zero"),
    ("encode", "quantum = np.ldexp(1.0, e - 8)", "quantum = np.ldexp(1.0, e - 7)", "bf16 with 7 significant bits"),
    ("encode", "e = np.maximum(e, -125)", "e = np.maximum(e, -100)", "bf16 subnormal range"),
    # the spacing that sets every bf16 / f32 parity tolerance
    ("ulp", "return np.ldexp(1.0, e - 8)", "return np.ldexp(1.0, e - 7)", "bf16 ulp twice the spacing"),
    ("ulp", "np.maximum(e, -125))", "np.maximum(e, -126))", "bf16 / f32 subnormal spacing halved"),
    ("ulp", "np.where(mag == 0, -125,", "np.where(mag == 0, 0,", "spacing at zero taken from binade 0"),
    ("ulp", "return np.ldexp(1.0, e - 24)", "return np.ldexp(1.0, e - 23)", "f32 ulp twice the spacing"),
    # directive checks
    ("check_directives", "if d.span_start < prev_end:", "if d.span_start < prev_end - 1:", "overlap by one accepted"),
    ("check_directives", "if not (0 <= d.span_start <= d.span_end <= n):",
     "if not (0 <= d.span_start <= d.span_end <= n + 1):", "span past the sequence accepted"),
    # FORGET (Sec. 3.1)
    ("resolve_forget", "out[j] = Directive(d.span_start, n, 0, d.seq)",
     "out[j] = Directive(d.span_end, n, 0, d.seq)", "cut at the span end"),
    ("resolve_forget", "if j != len(out) - 1:", "if False:", "FORGET before other directives accepted"),
    # the paged rule (this project's reading, pinned by invariants and reconstruction)
    ("plan_sequence", "if len(shifts) == 1 and len(old_pages) == 1 and same_off:",
     "if len(shifts) == 1 and len(old_pages) == 1:", "page re-used at other in-page offsets"),
    ("plan_sequence", "for kp in range(pages_for(n, page)) if kp not in kept",
     "for kp in range(pages_for(n, page) - 1) if kp not in kept", "last old page never freed"),
    ("plan_sequence", "                kept.add(kp)\n", "", "re-used page also freed"),
    ("paged_tables", "bt_out[b, k] = block_table[b, srcp]", "bt_out[b, k] = block_table[b, k]",
     "re-used page looked up at the new logical index"),
    ("plan_paged", "fresh += sum(1 for k in p.kinds if k == ASSEMBLE)", "pass",
     "fresh pages handed out twice"),
    ("plan_sequence", 'if remap and all(r[0] == "old" for r in rows):', 'if all(r[0] == "old" for r in rows):',
     "copy-on-write flag ignored"),
    ("paged_tables", "for kp in plan.freed)", "for kp in plan.freed[1:])", "a freed page not reported"),
    ("splice_paged", "lo, hi = k * page, min((k + 1) * page, plan.new_len)",
     "lo, hi = k * page, min((k + 1) * page, plan.new_len - 1)", "last row of a page run not written"),
    ("gather_logical", "pool[layer, bt_row[idx // page], idx % page]",
     "pool[layer, bt_row[idx // page], (idx + 1) % page]", "in-page offset off by one"),
    # layout of a row and of a cache
    ("decode", "<< np.uint32(16)", "<< np.uint32(15)", "bf16 bits misplaced"),
    ("Plane", "h * self.head_stride + self.rot_offset + np.arange(self.rot_dim)",
     "h * self.head_stride + np.arange(self.rot_dim)", "rotary band offset dropped"),
    ("Plane", "h * self.head_stride + self.rot_offset + np.arange(self.rot_dim)",
     "self.rot_offset + np.arange(self.rot_dim)", "every head rotates head 0's band"),
    ("rotate_rows", "if plane.rot_dim == 0 or len(out) == 0:", "if plane.rot_dim == 0 or len(out) <= 1:",
     "single-row segment not re-anchored"),
    ("splice_contig", "out[layer, :n_new] = splice_rows(cache[layer]", "out[layer, :n_new] = splice_rows(cache[0]",
     "every layer spliced from layer 0"),
]


def _pins():
    """Every pin of the oracle as (label, zero-argument callable); parametrized pins expanded."""
    out = []
    for name, fn in inspect.getmembers(PINS, inspect.isfunction):
        if not name.startswith("test_") or fn.__module__ != PINS.__name__:
            continue
        marks = [m for m in getattr(fn, "pytestmark", []) if m.name == "parametrize"]
        if not marks:
            out.append((name, fn))
            continue
        assert len(marks) == 1, name
        argname, values = marks[0].args[0], marks[0].args[1]
        assert "," not in argname, name
        out.extend((f"{name}[{v}]", (lambda f=fn, a=argname, v=v: f(**{a: v}))) for v in values)
    return out


def _failing_pin(pins):
    """The first pin that fails, or None."""
    for label, call in pins:
        try:
            call()
        except (Exception, pytest.fail.Exception):
            return label
    return None


class _Mutant:
    """Re-executes one oracle function or class from its source with one snippet replaced."""

    def __init__(self, name, old, new):
        self.name, self.old, self.new = name, old, new

    def __enter__(self):
        self.saved = getattr(O, self.name)
        src = textwrap.dedent(inspect.getsource(self.saved))
        assert src.count(self.old) == 1, f"{self.name}: snippet must occur once: {self.old!r}"
        exec(compile(src.replace(self.old, self.new), f"<mutant of {self.name}>", "exec"), O.__dict__)
        assert getattr(O, self.name) is not self.saved
        return self

    def __exit__(self, *exc):
        O.__dict__[self.name] = self.saved
        return False


def test_every_pin_passes_on_the_oracle_itself():
    assert _failing_pin(_pins()) is None


def test_reexecuted_unchanged_sources_pass_every_pin():
    """The mutation harness itself changes nothing when the snippet is left as it is."""
    pins = _pins()
    for name in sorted({m[0] for m in MUTANTS}):
        old = next(m[1] for m in MUTANTS if m[0] == name)
        with _Mutant(name, old, old):
            assert _failing_pin(pins) is None, name


@pytest.mark.parametrize("name,old,new,what", MUTANTS, ids=[f"{m[0]}:{m[3]}" for m in MUTANTS])
def test_planted_mistake_is_caught(name, old, new, what):
    with _Mutant(name, old, new):
        caught = _failing_pin(_pins())
    assert caught is not None, f"no pin catches: {what} ({name})"
    print(f"[mutant] {name}: {what} -> caught by {caught}")
