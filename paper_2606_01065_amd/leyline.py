"""ctypes binding of libleyline.so (argument marshalling only).

Every entry point of ``include/leyline.h`` is exposed under its C name.  Device memory is
passed as torch tensors (their ``data_ptr()``), the stream as a torch stream or a raw HIP stream
handle.  All computation happens in the HIP library; if it is missing the import fails.
"""

from __future__ import annotations

import ctypes
import os
from ctypes import POINTER, Structure, c_double, c_int, c_int32, c_int64, c_uint32, c_void_p
from collections import namedtuple
from dataclasses import dataclass
from typing import List, Optional, Sequence

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libleyline.so")
#: the same entry points with fp64 pair arithmetic (results bit-identical to a float64 reference)
EXACT_LIB_PATH = os.path.join(HERE, "libleyline_exact.so")

MAX_PLANES = 4
OK, E_INVAL, E_RANGE, E_ORDER, E_OVERLAP, E_CAPACITY, E_MODE, E_WORKSPACE, E_HIP = 0, -1, -2, -3, -4, -5, -6, -7, -8
BF16, F32 = 0, 1
ROPE_INTERLEAVED, ROPE_NEOX = 0, 1
AMORTIZE, FORGET = 0, 1
STATUS_BAD_PAGE, STATUS_BAD_ROW, STATUS_TILE_TIMEOUT = 1, 2, 4
PAGE_IDENTITY, PAGE_REMAP, PAGE_ASSEMBLE, PAGE_NONE = 0, 1, 2, -1
PAGED_COPY_ON_WRITE = 1


class leyline_plane(Structure):
    _fields_ = [
        ("base", c_void_p),
        ("layer_stride", c_int64),
        ("token_stride", c_int64),
        ("page_stride", c_int64),
        ("row_elems", c_int32),
        ("n_heads", c_int32),
        ("head_stride", c_int32),
        ("rot_offset", c_int32),
        ("rot_dim", c_int32),
        ("rope_style", c_int32),
        ("rope_base", c_double),
        ("inv_freq", POINTER(c_double)),
    ]


class leyline_cache(Structure):
    _fields_ = [
        ("dtype", c_int32),
        ("n_layers", c_int32),
        ("n_planes", c_int32),
        ("page_size", c_int32),
        ("capacity", c_int64),
        ("planes", leyline_plane * MAX_PLANES),
    ]


class leyline_directive(Structure):
    _fields_ = [
        ("seq", c_int32),
        ("mode", c_int32),
        ("span_start", c_int64),
        ("span_end", c_int64),
        ("stub_len", c_int64),
        ("stub", c_void_p * MAX_PLANES),
    ]


class LeylineError(RuntimeError):
    def __init__(self, code: int, where: str):
        self.code = code
        detail = f": {_lib.leyline_last_hip_error().decode()}" if code == E_HIP else ""
        super().__init__(f"{where}: {strerror(code)} ({code}){detail}")


def _hip_runtimes_mapped():
    try:
        with open("/proc/self/maps") as f:
            return sorted({ln.split()[-1] for ln in f if "libamdhip64" in ln})
    except OSError:
        return []


def _load(path=None):
    path = path or LIB_PATH
    if not os.path.exists(path):
        raise ImportError(f"{path} is not built; run `python -m paper_2606_01065_amd.build`")
    # torch ships its own HIP runtime.  It must be loaded before the library so that the
    # library's HIP dependency resolves to that same copy: two HIP/HSA runtimes in one process
    # cannot both open the GPU.
    import torch  # noqa: F401
    lib = ctypes.CDLL(path)
    runtimes = _hip_runtimes_mapped()
    if len(runtimes) > 1:
        raise ImportError("more than one HIP runtime is loaded in this process "
                          f"({', '.join(runtimes)}); import torch before anything that loads "
                          "another libamdhip64")
    P = POINTER
    sig = {
        "leyline_strerror": (ctypes.c_char_p, [c_int]),
        "leyline_abi_version": (c_int, []),
        "leyline_pair_bits": (c_int, []),
        "leyline_last_hip_error": (ctypes.c_char_p, []),
        "leyline_contig_query": (c_int, [P(leyline_cache), c_int64, P(leyline_directive), c_int32,
                                         P(c_int64), P(c_int32), P(c_int32), P(c_int64)]),
        "leyline_splice_contig": (c_int, [P(leyline_cache), c_int64, P(leyline_directive), c_int32,
                                          P(c_int64), c_void_p, c_void_p, c_int64, c_void_p]),
        "leyline_splice_contig_noalloc": (c_int, [P(leyline_cache), c_int64, P(leyline_directive), c_int32,
                                                  P(c_int64), c_void_p, c_void_p]),
        "leyline_paged_query": (c_int, [P(leyline_cache), c_int32, P(c_int32), c_int32,
                                        P(leyline_directive), c_int32, c_uint32, P(c_int32),
                                        P(c_int32), P(c_int32), P(c_int64)]),
        "leyline_paged_plan": (c_int, [c_int32, c_int32, P(c_int32), P(leyline_directive), c_int32,
                                       c_uint32, c_int32, P(c_int32), P(c_int32), P(c_int32),
                                       P(c_int32), c_int32]),
        "leyline_splice_paged": (c_int, [P(leyline_cache), c_int32, P(c_int32), c_void_p, c_void_p,
                                         c_int32, P(leyline_directive), c_int32, c_uint32, c_void_p,
                                         c_int32, c_void_p, c_int32, P(c_int32), P(c_int32),
                                         P(c_int32), c_void_p, c_void_p, c_int64, c_void_p]),
        "leyline_rotate_delta": (c_int, [P(leyline_cache), c_int64, c_void_p, c_int64, c_int64,
                                         c_void_p, c_void_p]),
    }
    for name, (res, args) in sig.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    return lib


_lib = _load()


def use_library(exact: bool) -> None:
    """Route every call of this module to libleyline_exact.so (fp64 pair arithmetic) or back to
    libleyline.so (fp32 pair arithmetic)."""
    global _lib
    _lib = _load(EXACT_LIB_PATH if exact else LIB_PATH)

#: every symbol the header declares (checked by tests against the loaded library)
SYMBOLS = ("leyline_strerror", "leyline_abi_version", "leyline_pair_bits", "leyline_last_hip_error",
           "leyline_contig_query",
           "leyline_splice_contig", "leyline_splice_contig_noalloc", "leyline_paged_query",
           "leyline_paged_plan", "leyline_splice_paged", "leyline_rotate_delta")

#: bytes of the library's fixed per-GPU scratch array (leyline_splice_contig_noalloc)
SCRATCH_BYTES = 1 << 20


def strerror(code: int) -> str:
    return _lib.leyline_strerror(code).decode()


def leyline_abi_version() -> int:
    return _lib.leyline_abi_version()


def leyline_pair_bits() -> int:
    return _lib.leyline_pair_bits()


# ----------------------------------------------------------------------------- descriptors --

@dataclass
class PlaneSpec:
    """A cache plane given as a tensor.

    contiguous: tensor [layers, capacity, *row]   paged: tensor [layers, pages, page_size, *row]
    The row dims must be dense (last stride 1, row elements contiguous).
    """
    tensor: object
    n_heads: int = 1
    head_stride: int = 0
    rot_offset: int = 0
    rot_dim: int = 0
    rope_style: int = ROPE_INTERLEAVED
    rope_base: float = 10000.0
    inv_freq: Optional[Sequence[float]] = None


def _dtype_code(t) -> int:
    import torch
    if t.dtype == torch.bfloat16:
        return BF16
    if t.dtype == torch.float32:
        return F32
    raise TypeError(f"unsupported cache dtype {t.dtype}")


def make_cache(planes: Sequence[PlaneSpec], paged: bool = False) -> leyline_cache:
    """Fill a leyline_cache from tensors (pure marshalling; the library validates the layout)."""
    if not 1 <= len(planes) <= MAX_PLANES:
        raise ValueError("1..4 planes")
    t0 = planes[0].tensor
    c = leyline_cache()
    c.dtype = _dtype_code(t0)
    c.n_layers = t0.shape[0]
    c.n_planes = len(planes)
    lead = 3 if paged else 2
    c.page_size = t0.shape[2] if paged else 0
    c.capacity = t0.shape[1]
    keep = []
    for i, p in enumerate(planes):
        t = p.tensor
        if _dtype_code(t) != c.dtype or t.shape[0] != c.n_layers:
            raise ValueError("planes must share dtype and layer count")
        row = 1
        for d in t.shape[lead:]:
            row *= d
        pl = c.planes[i]
        pl.base = t.data_ptr()
        pl.layer_stride = t.stride(0)
        if paged:
            pl.page_stride = t.stride(1)
            pl.token_stride = t.stride(2)
        else:
            pl.token_stride = t.stride(1)
        pl.row_elems = row
        pl.n_heads = p.n_heads
        pl.head_stride = p.head_stride or row
        pl.rot_offset = p.rot_offset
        pl.rot_dim = p.rot_dim
        pl.rope_style = p.rope_style
        pl.rope_base = p.rope_base
        if p.inv_freq is not None:
            arr = (c_double * len(p.inv_freq))(*p.inv_freq)
            keep.append(arr)
            pl.inv_freq = ctypes.cast(arr, POINTER(c_double))
        keep.append(t)
    # the descriptor holds raw pointers: it keeps the plane tensors and its host tables alive
    c._keep = keep
    c._device = getattr(t0, "device", None)
    return c


def _cache_device(cache: leyline_cache):
    return getattr(cache, "_device", None) or "cuda"


def make_directives(dirs: Sequence[dict]) -> ctypes.Array:
    """dirs: dicts with span_start, span_end, stub (list of per-plane tensors or None), optional
    seq and mode.  stub_len is taken from the stub tensors' token dim (dim 1) or 'stub_len'."""
    arr = (leyline_directive * max(1, len(dirs)))()
    keep = []
    for i, d in enumerate(dirs):
        x = arr[i]
        x.seq = d.get("seq", 0)
        x.mode = d.get("mode", AMORTIZE)
        x.span_start = d["span_start"]
        x.span_end = d["span_end"]
        stubs = d.get("stub") or []
        x.stub_len = d.get("stub_len", stubs[0].shape[1] if stubs else 0)
        for p, s in enumerate(stubs):
            x.stub[p] = s.data_ptr() if s is not None and s.numel() else None
            if s is not None:
                keep.append(s)
    arr._keep = keep         # the array holds raw pointers: it keeps the replacement tensors alive
    return arr


def _stream(stream) -> Optional[int]:
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def _stream_workspace(nbytes: int, stream, device):
    """A device buffer allocated on the stream the call runs on: torch's caching allocator hands a
    freed block out again only in that stream's order, so dropping the buffer when the call
    returns cannot let later work reuse it while the call's kernels still run."""
    import torch
    if stream is None:
        s = torch.cuda.current_stream(device)
    elif isinstance(stream, int):
        s = torch.cuda.ExternalStream(stream, device=device)
    else:
        s = stream
    with torch.cuda.stream(s):
        return torch.empty(nbytes, dtype=torch.uint8, device=device)


def _ptr(t) -> Optional[int]:
    return None if t is None else t.data_ptr()


def _check(rc: int, where: str) -> None:
    if rc != OK:
        raise LeylineError(rc, where)


# ----------------------------------------------------------------------------- entry points --

ContigQuery = namedtuple("ContigQuery", "new_len launches tile_launches workspace_bytes")


def leyline_contig_query(cache: leyline_cache, seq_len: int, dirs, n_dirs: int) -> ContigQuery:
    """(new_len, launches, tile_launches, workspace_bytes), without enqueueing anything."""
    new_len, n_launch, n_tile, ws = c_int64(0), c_int32(0), c_int32(0), c_int64(0)
    rc = _lib.leyline_contig_query(ctypes.byref(cache), seq_len, dirs, n_dirs, ctypes.byref(new_len),
                                   ctypes.byref(n_launch), ctypes.byref(n_tile), ctypes.byref(ws))
    _check(rc, "leyline_contig_query")
    return ContigQuery(new_len.value, n_launch.value, n_tile.value, ws.value)


def contig_workspace(cache: leyline_cache, seq_len: int, dirs, n_dirs: int, device="cuda"):
    """A device workspace tensor of the size the splice needs (None when it needs none)."""
    import torch
    need = leyline_contig_query(cache, seq_len, dirs, n_dirs).workspace_bytes
    return torch.empty(need, dtype=torch.uint8, device=device) if need else None


def leyline_splice_contig(cache: leyline_cache, seq_len: int, dirs, n_dirs: int, stream=None,
                          workspace=None, device_status=None) -> int:
    """Returns the new sequence length.  workspace: a device tensor of at least the queried size;
    when None, the call queries the size and allocates one with torch if the splice needs it
    (a caller that splices repeatedly keeps one workspace instead and saves the extra planning
    and allocation per call).  device_status: optional int32 device tensor (status bits)."""
    if workspace is None:
        need = leyline_contig_query(cache, seq_len, dirs, n_dirs).workspace_bytes
        if need:
            workspace = _stream_workspace(need, stream, _cache_device(cache))
    ws_ptr = workspace.data_ptr() if workspace is not None else None
    ws_len = workspace.numel() * workspace.element_size() if workspace is not None else 0
    new_len = c_int64(0)
    rc = _lib.leyline_splice_contig(ctypes.byref(cache), seq_len, dirs, n_dirs,
                                    ctypes.byref(new_len), _ptr(device_status), ws_ptr, ws_len,
                                    _stream(stream))
    _check(rc, "leyline_splice_contig")
    return new_len.value


def leyline_splice_contig_noalloc(cache: leyline_cache, seq_len: int, dirs, n_dirs: int, stream=None,
                                  device_status=None) -> int:
    """leyline_splice_contig on the library's fixed per-GPU scratch array (no workspace argument,
    no device allocation).  Returns the new sequence length."""
    new_len = c_int64(0)
    rc = _lib.leyline_splice_contig_noalloc(ctypes.byref(cache), seq_len, dirs, n_dirs, ctypes.byref(new_len),
                                            _ptr(device_status), _stream(stream))
    _check(rc, "leyline_splice_contig_noalloc")
    return new_len.value


def leyline_paged_query(cache: leyline_cache, seq_lens: Sequence[int], bt_stride: int, dirs, n_dirs: int,
                        flags: int = 0):
    """Returns (new_seq_lens, n_fresh_needed, n_freed, workspace_bytes)."""
    n = len(seq_lens)
    lens = (c_int32 * max(1, n))(*seq_lens)
    new = (c_int32 * max(1, n))()
    fresh, freed, ws = c_int32(0), c_int32(0), c_int64(0)
    rc = _lib.leyline_paged_query(ctypes.byref(cache), n, lens, bt_stride, dirs, n_dirs, flags, new,
                                  ctypes.byref(fresh), ctypes.byref(freed), ctypes.byref(ws))
    _check(rc, "leyline_paged_query")
    return list(new)[:n], fresh.value, freed.value, ws.value


def leyline_paged_plan(page_size: int, seq_lens: Sequence[int], dirs, n_dirs: int, bt_stride: int,
                       freed_cap: int, flags: int = 0):
    """Host-only symbolic plan: (kinds [n*bt_stride], srcs, freed_seq, freed_page)."""
    n = len(seq_lens)
    lens = (c_int32 * max(1, n))(*seq_lens)
    kinds = (c_int32 * max(1, n * bt_stride))()
    srcs = (c_int32 * max(1, n * bt_stride))()
    fs = (c_int32 * max(1, freed_cap))()
    fp = (c_int32 * max(1, freed_cap))()
    rc = _lib.leyline_paged_plan(page_size, n, lens, dirs, n_dirs, flags, bt_stride, kinds, srcs, fs, fp,
                                 freed_cap)
    _check(rc, "leyline_paged_plan")
    return list(kinds)[:n * bt_stride], list(srcs)[:n * bt_stride], list(fs), list(fp)


def leyline_splice_paged(cache: leyline_cache, seq_lens: Sequence[int], block_table_in, block_table_out,
                         dirs, n_dirs: int, free_pages, freed_pages_out, workspace,
                         device_status=None, stream=None, flags: int = 0):
    """Returns (new_seq_lens, n_fresh_used, n_freed).  Tables are int32 device tensors."""
    n = len(seq_lens)
    lens = (c_int32 * max(1, n))(*seq_lens)
    new = (c_int32 * max(1, n))()
    fresh, freed = c_int32(0), c_int32(0)
    bt_stride = block_table_in.shape[1]
    rc = _lib.leyline_splice_paged(
        ctypes.byref(cache), n, lens, _ptr(block_table_in), _ptr(block_table_out), bt_stride,
        dirs, n_dirs, flags, _ptr(free_pages), 0 if free_pages is None else free_pages.numel(),
        _ptr(freed_pages_out), 0 if freed_pages_out is None else freed_pages_out.numel(),
        new, ctypes.byref(fresh), ctypes.byref(freed), _ptr(device_status),
        _ptr(workspace), 0 if workspace is None else workspace.numel() * workspace.element_size(),
        _stream(stream))
    _check(rc, "leyline_splice_paged")
    return list(new)[:n], fresh.value, freed.value


def leyline_rotate_delta(cache: leyline_cache, delta: int, rows=None, row0: int = 0, n_rows: int = 0,
                         device_status=None, stream=None) -> None:
    """rows: optional int64 device tensor of physical row indices."""
    if rows is not None:
        n_rows = rows.numel()
    rc = _lib.leyline_rotate_delta(ctypes.byref(cache), delta, _ptr(rows), row0, n_rows,
                                   _ptr(device_status), _stream(stream))
    _check(rc, "leyline_rotate_delta")
