"""Python binding of libgeot_hip (argument marshalling only).

Every call here forwards torch tensors' device pointers and the current HIP
stream to the extern "C" functions declared in include/geot.h; all arithmetic
runs in the library's HIP kernels. There is no fallback: if the library is
not built, or a tensor is not on the GPU, the call raises.
"""
from __future__ import annotations

import ctypes
import os

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libgeot_hip.so")

OPS = {"sum": 0, "mean": 1, "max": 2}
FAMILIES = {"auto": 0, "ep": 1, "sp": 2}
STATUS = {0: "success", 1: "invalid value", 2: "index not sorted", 3: "index out of range",
          4: "HIP runtime error", 5: "unsupported kernel choice"}


class GeotError(RuntimeError):
    def __init__(self, status: int, detail: str):
        super().__init__(f"{STATUS.get(status, status)}: {detail}")
        self.status = status
        self.detail = detail


class KernelChoice(ctypes.Structure):
    _fields_ = [("family", ctypes.c_int32), ("vec", ctypes.c_int32), ("lanes", ctypes.c_int32),
                ("rows", ctypes.c_int32), ("groups", ctypes.c_int32), ("flags", ctypes.c_int32)]

    def as_dict(self) -> dict:
        return {k: int(getattr(self, k)) for k, _ in self._fields_}


class IndexStats(ctypes.Structure):
    _fields_ = [("nnz", ctypes.c_int64), ("num_segments", ctypes.c_int64),
                ("max_len", ctypes.c_int64), ("num_empty", ctypes.c_int64),
                ("sum_len_sq", ctypes.c_int64), ("mean_len", ctypes.c_double),
                ("var_len", ctypes.c_double)]

    def as_dict(self) -> dict:
        return {k: getattr(self, k) for k, _ in self._fields_}


_lib = None


def lib() -> ctypes.CDLL:
    """The loaded C library (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise GeotError(4, f"{LIB_PATH} is missing: build it with __graft_entry__.build()")
    L = ctypes.CDLL(LIB_PATH)
    p, i64, i32 = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32
    pc = ctypes.POINTER(KernelChoice)
    L.geot_segment_reduce.argtypes = [p, p, i64, i64, i64, ctypes.c_int, p, p]
    L.geot_segment_reduce_with.argtypes = [p, p, i64, i64, i64, ctypes.c_int, p, p, pc]
    L.geot_gather_scatter.argtypes = [p, i64, p, p, p, i64, i64, i64, ctypes.c_int, p, p]
    L.geot_gather_scatter_with.argtypes = [p, i64, p, p, p, i64, i64, i64, ctypes.c_int, p, p, pc]
    L.geot_segment_reduce_typed.argtypes = [p, ctypes.c_int, p, ctypes.c_int, i64, i64, i64, ctypes.c_int,
                                            p, p, pc]
    L.geot_gather_scatter_typed.argtypes = [p, ctypes.c_int, i64, p, p, p, ctypes.c_int, i64, i64, i64,
                                            ctypes.c_int, p, p, pc]
    L.geot_select.argtypes = [i64, i64, i64, ctypes.c_int, i32, ctypes.POINTER(IndexStats), pc]
    L.geot_index_stats.argtypes = [p, i64, i64, ctypes.POINTER(IndexStats), p]
    L.geot_check_index.argtypes = [p, i64, i64, p, i64, p]
    L.geot_segment_reduce_backward.argtypes = [p, p, i64, i64, i64, ctypes.c_int, p, p, p, p]
    L.geot_segment_reduce_backward_typed.argtypes = [p, p, ctypes.c_int, i64, i64, i64, ctypes.c_int, p,
                                                     ctypes.c_int, p, p, p]
    L.geot_gather_scatter_backward.argtypes = [p, i64, p, p, p, i64, i64, i64, ctypes.c_int, p, p, p, p, p]
    L.geot_gather_scatter_backward_typed.argtypes = [p, ctypes.c_int, i64, p, p, p, ctypes.c_int, i64, i64, i64,
                                                     ctypes.c_int, p, p, p, p, p]
    L.geot_transpose_edges.argtypes = [p, i64, p, p, i64, i64, ctypes.c_int, p, p, p, p]
    L.geot_segment_reduce_max_arg.argtypes = [p, ctypes.c_int, p, ctypes.c_int, i64, i64, i64, p, p, p, pc]
    L.geot_gather_scatter_max_arg.argtypes = [p, ctypes.c_int, i64, p, p, p, ctypes.c_int, i64, i64, i64,
                                              p, p, p, pc]
    L.geot_segment_reduce_backward_max_arg.argtypes = [p, p, ctypes.c_int, i64, i64, i64, p, p,
                                                       ctypes.c_int, p]
    L.geot_gather_scatter_backward_max_arg.argtypes = [p, ctypes.c_int, i64, p, p, p, ctypes.c_int, i64, i64,
                                                       i64, p, p, p, p, p]
    sz = ctypes.c_size_t
    L.geot_segment_reduce_workspace_size.argtypes = [i64, i64, i64, ctypes.c_int, pc, ctypes.POINTER(sz)]
    L.geot_gather_scatter_workspace_size.argtypes = [i64, i64, i64, ctypes.c_int, i32, pc, ctypes.POINTER(sz)]
    L.geot_segment_reduce_ws.argtypes = [p, p, i64, i64, i64, ctypes.c_int, p, p, sz, p, pc]
    L.geot_gather_scatter_ws.argtypes = [p, i64, p, p, p, i64, i64, i64, ctypes.c_int, p, p, sz, p, pc]
    L.geot_segment_reduce_noalloc.argtypes = [p, p, i64, i64, i64, ctypes.c_int, p, p]
    L.geot_noalloc_scratch_bytes.argtypes = []
    L.geot_noalloc_scratch_bytes.restype = sz
    L.geot_last_choice.argtypes = [pc]
    L.geot_release_scratch.argtypes = []
    L.geot_profile_begin.argtypes = [i32]
    L.geot_profile_end.argtypes = [ctypes.POINTER(ctypes.c_float), i32, ctypes.POINTER(i32)]
    L.geot_status_string.argtypes = [ctypes.c_int]
    L.geot_status_string.restype = ctypes.c_char_p
    L.geot_last_error_detail.argtypes = []
    L.geot_last_error_detail.restype = ctypes.c_char_p
    L.geot_version.restype = i32
    for name in ("geot_segment_reduce", "geot_segment_reduce_with", "geot_gather_scatter",
                 "geot_gather_scatter_with", "geot_select", "geot_index_stats", "geot_check_index",
                 "geot_last_choice", "geot_profile_begin", "geot_profile_end", "geot_release_scratch",
                 "geot_segment_reduce_backward", "geot_gather_scatter_backward",
                 "geot_segment_reduce_workspace_size", "geot_gather_scatter_workspace_size",
                 "geot_segment_reduce_ws", "geot_gather_scatter_ws", "geot_segment_reduce_noalloc"):
        getattr(L, name).restype = ctypes.c_int
    _lib = L
    return L


def _raise(status: int):
    if status != 0:
        detail = lib().geot_last_error_detail().decode()
        raise GeotError(status, detail)


def _choice(choice) -> KernelChoice | None:
    if choice is None:
        return None
    if isinstance(choice, KernelChoice):
        return choice
    c = dict(choice)
    fam = c.get("family", 0)
    if isinstance(fam, str):
        fam = FAMILIES[fam]
    return KernelChoice(int(fam), int(c.get("vec", 0)), int(c.get("lanes", 0)),
                        int(c.get("rows", 0)), int(c.get("groups", 0)), int(c.get("flags", 0)))


def _dev(t: torch.Tensor, name: str, dtype, ndim):
    """Type, rank and layout of one tensor argument (its device is checked by _on_gpu, after
    the shapes, so that every size mismatch is reported before anything else)."""
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch tensor")
    if t.dtype not in (dtype if isinstance(dtype, tuple) else (dtype,)):
        raise TypeError(f"{name} must be {dtype}")
    if t.dim() != ndim:
        raise ValueError(f"{name} must have {ndim} dimensions")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return t


def _shape(t: torch.Tensor | None, name: str, shape: tuple):
    if t is not None and tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} must have shape {tuple(shape)}, got {tuple(t.shape)}")


def _on_gpu(**tensors):
    """Every given tensor is on the same GPU (the library reads them through raw pointers)."""
    dev = None
    for name, t in tensors.items():
        if t is None:
            continue
        if t.device.type != "cuda":
            raise ValueError(f"{name} must be on the GPU")
        if dev is None:
            dev = t.device
        elif t.device != dev:
            raise ValueError(f"{name} is on {t.device}, the other arguments on {dev}")


def _stream(device) -> int:
    return torch.cuda.current_stream(device).cuda_stream


class _OnDevice:
    """Make `device` current for the call (cheap when it already is)."""

    __slots__ = ("idx", "prev")

    def __init__(self, device):
        self.idx = device.index if device.index is not None else torch.cuda.current_device()

    def __enter__(self):
        self.prev = torch.cuda.current_device()
        if self.prev != self.idx:
            torch.cuda.set_device(self.idx)
        return self

    def __exit__(self, *exc):
        if self.prev != self.idx:
            torch.cuda.set_device(self.prev)
        return False


# storage types of src / x and index types accepted by the typed entry points
DTYPES = {torch.float32: 0, torch.bfloat16: 1, torch.float16: 2}
INDEX_TYPES = {torch.int64: 0, torch.int32: 1}


def _stats_choice(choice, stats, nnz, S, F, reduce, gather, weighted, plain):
    """The selector's choice with the index statistics `stats` (geot_index_stats of the same
    index, computed once by the caller, e.g. per static graph) when no choice is forced; the
    segment-parallel family it may pick takes fp32 data with int64 ids only (`plain`)."""
    if choice is not None or stats is None or not plain:
        return choice
    return select(nnz, S, F, reduce, gather=gather, stats=stats, weighted=weighted)


def segment_reduce(src: torch.Tensor, index: torch.Tensor, num_segments: int, reduce: str = "sum",
                   out: torch.Tensor | None = None, choice=None, stats: dict | None = None) -> torch.Tensor:
    """out[s] = reduce over rows i of src with index[i] == s (geot_segment_reduce).

    src may be fp32, bf16 or fp16 and index int64 or int32 (geot_segment_reduce_typed);
    out is fp32 in every case. `stats` (index_stats(index, num_segments), kept by the caller)
    lets the selector use the length spread (geot_select with statistics)."""
    _dev(src, "src", tuple(DTYPES), 2)
    _dev(index, "index", tuple(INDEX_TYPES), 1)
    if index.numel() != src.shape[0]:
        raise ValueError("index must have one entry per row of src")
    S, F = int(num_segments), src.shape[1]
    if out is not None:
        _dev(out, "out", torch.float32, 2)
        _shape(out, "out", (S, F))
    _on_gpu(src=src, index=index, out=out)
    if out is None:
        out = torch.empty((S, F), dtype=torch.float32, device=src.device)
    plain = src.dtype == torch.float32 and index.dtype == torch.int64
    c = _choice(_stats_choice(choice, stats, index.numel(), S, F, reduce, False, True, plain))
    cp = ctypes.byref(c) if c is not None else None
    with _OnDevice(src.device):
        if plain:
            st = lib().geot_segment_reduce_with(src.data_ptr(), index.data_ptr(), index.numel(), S, F,
                                                OPS[reduce], out.data_ptr(), _stream(src.device), cp)
        else:
            st = lib().geot_segment_reduce_typed(src.data_ptr(), DTYPES[src.dtype], index.data_ptr(),
                                                 INDEX_TYPES[index.dtype], index.numel(), S, F,
                                                 OPS[reduce], out.data_ptr(), _stream(src.device), cp)
    _raise(st)
    return out


def gather_scatter(x: torch.Tensor, col: torch.Tensor, weight: torch.Tensor | None,
                   row: torch.Tensor, num_rows: int, reduce: str = "sum",
                   out: torch.Tensor | None = None, choice=None, stats: dict | None = None) -> torch.Tensor:
    """out[r] = reduce over edges e with row[e] == r of weight[e] * x[col[e]] (geot_gather_scatter).

    x may be fp32, bf16 or fp16 and col / row int64 or int32 (both the same;
    geot_gather_scatter_typed); weight and out are fp32. `stats`: index_stats(row, num_rows),
    as for segment_reduce."""
    _dev(x, "x", tuple(DTYPES), 2)
    _dev(col, "col", tuple(INDEX_TYPES), 1)
    _dev(row, "row", (col.dtype,), 1)
    if weight is not None:
        _dev(weight, "weight", torch.float32, 1)
        if weight.numel() != row.numel():
            raise ValueError("weight must have one entry per edge")
    if col.numel() != row.numel():
        raise ValueError("col and row must have one entry per edge")
    R, F = int(num_rows), x.shape[1]
    if out is not None:
        _dev(out, "out", torch.float32, 2)
        _shape(out, "out", (R, F))
    _on_gpu(x=x, col=col, weight=weight, row=row, out=out)
    if out is None:
        out = torch.empty((R, F), dtype=torch.float32, device=x.device)
    plain = x.dtype == torch.float32 and col.dtype == torch.int64
    c = _choice(_stats_choice(choice, stats, row.numel(), R, F, reduce, True, weight is not None, plain))
    wp = weight.data_ptr() if weight is not None else None
    cp = ctypes.byref(c) if c is not None else None
    with _OnDevice(x.device):
        if plain:
            st = lib().geot_gather_scatter_with(x.data_ptr(), x.shape[0], col.data_ptr(), wp,
                                                row.data_ptr(), row.numel(), R, F, OPS[reduce],
                                                out.data_ptr(), _stream(x.device), cp)
        else:
            st = lib().geot_gather_scatter_typed(x.data_ptr(), DTYPES[x.dtype], x.shape[0], col.data_ptr(),
                                                 wp, row.data_ptr(), INDEX_TYPES[col.dtype], row.numel(),
                                                 R, F, OPS[reduce], out.data_ptr(), _stream(x.device), cp)
    _raise(st)
    return out


def segment_reduce_max_arg(src: torch.Tensor, index: torch.Tensor, num_segments: int, choice=None):
    """(out, arg): the max of segment_reduce and its recipients (geot_segment_reduce_max_arg).

    arg [num_segments, F] int32 holds the uint32 row numbers the library writes: the lowest
    row of each segment whose value equals the maximum, -1 (0xFFFFFFFF) where there is none.
    Requires fewer than 2^32 - 1 rows."""
    _dev(src, "src", tuple(DTYPES), 2)
    _dev(index, "index", tuple(INDEX_TYPES), 1)
    if index.numel() != src.shape[0]:
        raise ValueError("index must have one entry per row of src")
    _on_gpu(src=src, index=index)
    S, F = int(num_segments), src.shape[1]
    out = torch.empty((S, F), dtype=torch.float32, device=src.device)
    arg = torch.empty((S, F), dtype=torch.int32, device=src.device)
    c = _choice(choice)
    with _OnDevice(src.device):
        st = lib().geot_segment_reduce_max_arg(src.data_ptr(), DTYPES[src.dtype], index.data_ptr(),
                                               INDEX_TYPES[index.dtype], index.numel(), S, F, out.data_ptr(),
                                               arg.data_ptr(), _stream(src.device),
                                               ctypes.byref(c) if c is not None else None)
    _raise(st)
    return out, arg


def gather_scatter_max_arg(x: torch.Tensor, col: torch.Tensor, weight: torch.Tensor | None,
                           row: torch.Tensor, num_rows: int, choice=None):
    """(out, arg): the max of gather_scatter and its recipients (geot_gather_scatter_max_arg):
    arg [num_rows, F] int32 holds the uint32 edge numbers, -1 where there is none."""
    _dev(x, "x", tuple(DTYPES), 2)
    _dev(col, "col", tuple(INDEX_TYPES), 1)
    _dev(row, "row", (col.dtype,), 1)
    if weight is not None:
        _dev(weight, "weight", torch.float32, 1)
        if weight.numel() != row.numel():
            raise ValueError("weight must have one entry per edge")
    if col.numel() != row.numel():
        raise ValueError("col and row must have one entry per edge")
    _on_gpu(x=x, col=col, weight=weight, row=row)
    R, F = int(num_rows), x.shape[1]
    out = torch.empty((R, F), dtype=torch.float32, device=x.device)
    arg = torch.empty((R, F), dtype=torch.int32, device=x.device)
    c = _choice(choice)
    with _OnDevice(x.device):
        st = lib().geot_gather_scatter_max_arg(x.data_ptr(), DTYPES[x.dtype], x.shape[0], col.data_ptr(),
                                               weight.data_ptr() if weight is not None else None, row.data_ptr(),
                                               INDEX_TYPES[col.dtype], row.numel(), R, F, out.data_ptr(),
                                               arg.data_ptr(), _stream(x.device),
                                               ctypes.byref(c) if c is not None else None)
    _raise(st)
    return out, arg


def segment_reduce_backward_max_arg(grad_out: torch.Tensor, index: torch.Tensor, arg: torch.Tensor,
                                    dtype: torch.dtype = torch.float32) -> torch.Tensor:
    """Gradient of the max of segment_reduce w.r.t. src from recorded recipients (arg of
    segment_reduce_max_arg; geot_segment_reduce_backward_max_arg), in storage type `dtype`."""
    _dev(grad_out, "grad_out", torch.float32, 2)
    _dev(index, "index", tuple(INDEX_TYPES), 1)
    _dev(arg, "arg", torch.int32, 2)
    if dtype not in DTYPES:
        raise TypeError(f"the gradient's type must be one of {tuple(DTYPES)}")
    S, F = grad_out.shape
    _shape(arg, "arg", (S, F))
    _on_gpu(grad_out=grad_out, index=index, arg=arg)
    grad_src = torch.empty((index.numel(), F), dtype=dtype, device=grad_out.device)
    with _OnDevice(grad_out.device):
        st = lib().geot_segment_reduce_backward_max_arg(grad_out.data_ptr(), index.data_ptr(),
                                                        INDEX_TYPES[index.dtype], index.numel(), S, F,
                                                        arg.data_ptr(), grad_src.data_ptr(), DTYPES[dtype],
                                                        _stream(grad_out.device))
    _raise(st)
    return grad_src


def gather_scatter_backward_max_arg(x: torch.Tensor, col: torch.Tensor, weight: torch.Tensor | None,
                                    row: torch.Tensor, grad_out: torch.Tensor, arg: torch.Tensor,
                                    need_x: bool = True, need_weight: bool = True):
    """(grad_x or None, grad_weight or None) of the max of gather_scatter from recorded
    recipients (arg of gather_scatter_max_arg; geot_gather_scatter_backward_max_arg)."""
    _dev(x, "x", tuple(DTYPES), 2)
    _dev(col, "col", tuple(INDEX_TYPES), 1)
    _dev(row, "row", (col.dtype,), 1)
    _dev(grad_out, "grad_out", torch.float32, 2)
    _dev(arg, "arg", torch.int32, 2)
    R, F = grad_out.shape
    n = row.numel()
    if col.numel() != n:
        raise ValueError("col and row must have one entry per edge")
    if x.shape[1] != F:
        raise ValueError(f"x has {x.shape[1]} columns, grad_out {F}")
    _shape(arg, "arg", (R, F))
    if weight is not None:
        _dev(weight, "weight", torch.float32, 1)
        _shape(weight, "weight", (n,))
    _on_gpu(x=x, col=col, weight=weight, row=row, grad_out=grad_out, arg=arg)
    gx = torch.empty(x.shape, dtype=torch.float32, device=x.device) if need_x else None
    gw = torch.empty_like(weight) if (need_weight and weight is not None) else None
    with _OnDevice(x.device):
        st = lib().geot_gather_scatter_backward_max_arg(
            x.data_ptr(), DTYPES[x.dtype], x.shape[0], col.data_ptr(),
            weight.data_ptr() if weight is not None else None, row.data_ptr(), INDEX_TYPES[col.dtype], n, R, F,
            grad_out.data_ptr(), arg.data_ptr(), gx.data_ptr() if gx is not None else None,
            gw.data_ptr() if gw is not None else None, _stream(x.device))
    _raise(st)
    return gx, gw


def workspace_size(nnz: int, num_segments: int, F: int, reduce: str = "sum", gather: bool = False,
                   weighted: bool = True, choice=None) -> int:
    """Bytes of caller workspace that segment_reduce_ws (gather_scatter_ws with `gather`) needs
    for these sizes, whatever the alignment of the arrays (the *_workspace_size queries; host only)."""
    c = _choice(choice)
    cp = ctypes.byref(c) if c is not None else None
    n = ctypes.c_size_t()
    if gather:
        st = lib().geot_gather_scatter_workspace_size(int(nnz), int(num_segments), int(F), OPS[reduce],
                                                      1 if weighted else 0, cp, ctypes.byref(n))
    else:
        st = lib().geot_segment_reduce_workspace_size(int(nnz), int(num_segments), int(F), OPS[reduce], cp,
                                                      ctypes.byref(n))
    _raise(st)
    return int(n.value)


def _workspace(ws: torch.Tensor | None):
    if ws is None:
        return None, 0
    if not isinstance(ws, torch.Tensor) or not ws.is_contiguous():
        raise ValueError("workspace must be a contiguous tensor")
    return ws.data_ptr(), ws.numel() * ws.element_size()


def segment_reduce_ws(src: torch.Tensor, index: torch.Tensor, num_segments: int, reduce: str,
                      workspace: torch.Tensor | None, out: torch.Tensor | None = None, choice=None) -> torch.Tensor:
    """segment_reduce (fp32 src, int64 index) with its temporary memory in `workspace`
    (geot_segment_reduce_ws): any contiguous device tensor of at least workspace_size(...) bytes."""
    _dev(src, "src", torch.float32, 2)
    _dev(index, "index", torch.int64, 1)
    if index.numel() != src.shape[0]:
        raise ValueError("index must have one entry per row of src")
    S, F = int(num_segments), src.shape[1]
    if out is not None:
        _dev(out, "out", torch.float32, 2)
        _shape(out, "out", (S, F))
    _on_gpu(src=src, index=index, out=out, workspace=workspace)
    if out is None:
        out = torch.empty((S, F), dtype=torch.float32, device=src.device)
    wp, wb = _workspace(workspace)
    c = _choice(choice)
    with _OnDevice(src.device):
        st = lib().geot_segment_reduce_ws(src.data_ptr(), index.data_ptr(), index.numel(), S, F, OPS[reduce],
                                          out.data_ptr(), wp, wb, _stream(src.device),
                                          ctypes.byref(c) if c is not None else None)
    _raise(st)
    return out


def gather_scatter_ws(x: torch.Tensor, col: torch.Tensor, weight: torch.Tensor | None, row: torch.Tensor,
                      num_rows: int, reduce: str, workspace: torch.Tensor | None,
                      out: torch.Tensor | None = None, choice=None) -> torch.Tensor:
    """gather_scatter (fp32 x, int64 col / row) with its temporary memory in `workspace`
    (geot_gather_scatter_ws)."""
    _dev(x, "x", torch.float32, 2)
    _dev(col, "col", torch.int64, 1)
    _dev(row, "row", torch.int64, 1)
    if weight is not None:
        _dev(weight, "weight", torch.float32, 1)
        if weight.numel() != row.numel():
            raise ValueError("weight must have one entry per edge")
    if col.numel() != row.numel():
        raise ValueError("col and row must have one entry per edge")
    R, F = int(num_rows), x.shape[1]
    if out is not None:
        _dev(out, "out", torch.float32, 2)
        _shape(out, "out", (R, F))
    _on_gpu(x=x, col=col, weight=weight, row=row, out=out, workspace=workspace)
    if out is None:
        out = torch.empty((R, F), dtype=torch.float32, device=x.device)
    wp, wb = _workspace(workspace)
    c = _choice(choice)
    with _OnDevice(x.device):
        st = lib().geot_gather_scatter_ws(x.data_ptr(), x.shape[0], col.data_ptr(),
                                          weight.data_ptr() if weight is not None else None, row.data_ptr(),
                                          row.numel(), R, F, OPS[reduce], out.data_ptr(), wp, wb,
                                          _stream(x.device), ctypes.byref(c) if c is not None else None)
    _raise(st)
    return out


def segment_reduce_noalloc(src: torch.Tensor, index: torch.Tensor, num_segments: int, reduce: str,
                           out: torch.Tensor) -> torch.Tensor:
    """segment_reduce (fp32 src, int64 index) into a given `out`, with no allocation anywhere:
    the library's static per-GPU array holds its temporaries (geot_segment_reduce_noalloc)."""
    _dev(src, "src", torch.float32, 2)
    _dev(index, "index", torch.int64, 1)
    _dev(out, "out", torch.float32, 2)
    if index.numel() != src.shape[0]:
        raise ValueError("index must have one entry per row of src")
    S, F = int(num_segments), src.shape[1]
    _shape(out, "out", (S, F))
    _on_gpu(src=src, index=index, out=out)
    with _OnDevice(src.device):
        st = lib().geot_segment_reduce_noalloc(src.data_ptr(), index.data_ptr(), index.numel(), S, F,
                                               OPS[reduce], out.data_ptr(), _stream(src.device))
    _raise(st)
    return out


def noalloc_scratch_bytes() -> int:
    """Size of the static per-GPU array of segment_reduce_noalloc."""
    return int(lib().geot_noalloc_scratch_bytes())


def segment_reduce_backward(grad_out: torch.Tensor, index: torch.Tensor, reduce: str = "sum",
                            src: torch.Tensor | None = None, out: torch.Tensor | None = None,
                            grad_src: torch.Tensor | None = None, dtype: torch.dtype | None = None
                            ) -> torch.Tensor:
    """Gradient of segment_reduce w.r.t. src (geot_segment_reduce_backward_typed).

    The gradient has src's storage type: that of `grad_src` when given, else of `src`
    (max), else `dtype` (default fp32). The index may be int64 or int32."""
    _dev(grad_out, "grad_out", torch.float32, 2)
    _dev(index, "index", tuple(INDEX_TYPES), 1)
    S, F = grad_out.shape
    typ = grad_src.dtype if grad_src is not None else (src.dtype if src is not None else (dtype or torch.float32))
    if typ not in DTYPES:
        raise TypeError(f"the gradient's type must be one of {tuple(DTYPES)}")
    if reduce not in OPS:
        raise ValueError(f"unknown reduce {reduce!r}")
    if reduce == "max":
        if src is None or out is None:
            raise ValueError("max needs src and out")
        _dev(src, "src", typ, 2)
        _dev(out, "out", torch.float32, 2)
        _shape(src, "src", (index.numel(), F))
        _shape(out, "out", (S, F))
    else:   # read for max only
        src = out = None
    if grad_src is not None:
        _dev(grad_src, "grad_src", typ, 2)
        _shape(grad_src, "grad_src", (index.numel(), F))
    _on_gpu(grad_out=grad_out, index=index, src=src, out=out, grad_src=grad_src)
    if grad_src is None:
        grad_src = torch.empty((index.numel(), F), dtype=typ, device=grad_out.device)
    with _OnDevice(grad_out.device):
        st = lib().geot_segment_reduce_backward_typed(
            grad_out.data_ptr(), index.data_ptr(), INDEX_TYPES[index.dtype], index.numel(), S, F, OPS[reduce],
            src.data_ptr() if src is not None else None, DTYPES[typ],
            out.data_ptr() if out is not None else None, grad_src.data_ptr(), _stream(grad_out.device))
    _raise(st)
    return grad_src


def gather_scatter_backward(x: torch.Tensor, col: torch.Tensor, weight: torch.Tensor | None,
                            row: torch.Tensor, grad_out: torch.Tensor, reduce: str = "sum",
                            out: torch.Tensor | None = None, need_x: bool = True,
                            need_weight: bool = True):
    """(grad_x or None, grad_weight or None) of gather_scatter (geot_gather_scatter_backward_typed).

    x may be fp32, bf16 or fp16 and col / row int64 or int32 (the same type); grad_x and
    grad_weight are fp32."""
    _dev(x, "x", tuple(DTYPES), 2)
    _dev(col, "col", tuple(INDEX_TYPES), 1)
    _dev(row, "row", (col.dtype,), 1)
    _dev(grad_out, "grad_out", torch.float32, 2)
    if reduce not in OPS:
        raise ValueError(f"unknown reduce {reduce!r}")
    R, F = grad_out.shape
    n = row.numel()
    if col.numel() != n:
        raise ValueError("col and row must have one entry per edge")
    if x.shape[1] != F:
        raise ValueError(f"x has {x.shape[1]} columns, grad_out {F}")
    if weight is not None:
        _dev(weight, "weight", torch.float32, 1)
        _shape(weight, "weight", (n,))
    if reduce == "max":
        if out is None:
            raise ValueError("max needs out")
        _dev(out, "out", torch.float32, 2)
        _shape(out, "out", (R, F))
    else:   # read for max only
        out = None
    _on_gpu(x=x, col=col, weight=weight, row=row, grad_out=grad_out, out=out)
    gx = torch.empty(x.shape, dtype=torch.float32, device=x.device) if need_x else None
    gw = torch.empty_like(weight) if (need_weight and weight is not None) else None
    with _OnDevice(x.device):
        st = lib().geot_gather_scatter_backward_typed(
            x.data_ptr(), DTYPES[x.dtype], x.shape[0], col.data_ptr(),
            weight.data_ptr() if weight is not None else None, row.data_ptr(), INDEX_TYPES[col.dtype],
            row.numel(), R, F, OPS[reduce], grad_out.data_ptr(),
            out.data_ptr() if out is not None else None, gx.data_ptr() if gx is not None else None,
            gw.data_ptr() if gw is not None else None, _stream(x.device))
    _raise(st)
    return gx, gw


def transpose_edges(col: torch.Tensor, weight: torch.Tensor | None, row: torch.Tensor, num_x_rows: int,
                    num_rows: int, reduce: str = "sum"):
    """The edge list sorted by column (geot_transpose_edges): (sorted_col, row_t, coef).

    gather_scatter(grad_out, row_t, coef, sorted_col, num_x_rows, "sum") is then the
    gradient w.r.t. x of gather_scatter(x, col, weight, row, num_rows, reduce)."""
    _dev(col, "col", torch.int64, 1)
    _dev(row, "row", torch.int64, 1)
    if weight is not None:
        _dev(weight, "weight", torch.float32, 1)
        if weight.numel() != row.numel():
            raise ValueError("weight must have one entry per edge")
    if col.numel() != row.numel():
        raise ValueError("col and row must have one entry per edge")
    _on_gpu(col=col, weight=weight, row=row)
    n = row.numel()
    sc = torch.empty(n, dtype=torch.int64, device=row.device)
    rt = torch.empty(n, dtype=torch.int64, device=row.device)
    cf = torch.empty(n, dtype=torch.float32, device=row.device)
    wp = weight.data_ptr() if weight is not None else None
    with _OnDevice(row.device):
        st = lib().geot_transpose_edges(col.data_ptr(), int(num_x_rows), wp, row.data_ptr(), n, int(num_rows),
                                        OPS[reduce], sc.data_ptr(), rt.data_ptr(), cf.data_ptr(),
                                        _stream(row.device))
    _raise(st)
    return sc, rt, cf


def index_stats(index: torch.Tensor, num_segments: int) -> dict:
    """Segment-length statistics of a sorted index (geot_index_stats; synchronizes)."""
    _dev(index, "index", torch.int64, 1)
    _on_gpu(index=index)
    o = IndexStats()
    with _OnDevice(index.device):
        st = lib().geot_index_stats(index.data_ptr(), index.numel(), int(num_segments),
                                    ctypes.byref(o), _stream(index.device))
    _raise(st)
    return o.as_dict()


def check_index(index: torch.Tensor, num_segments: int, col: torch.Tensor | None = None,
                num_x_rows: int = 0) -> int:
    """Precondition check (geot_check_index; synchronizes). Returns the status code."""
    _dev(index, "index", torch.int64, 1)
    cp = None
    if col is not None:
        _dev(col, "col", torch.int64, 1)
        cp = col.data_ptr()
    _on_gpu(index=index, col=col)
    with _OnDevice(index.device):
        return int(lib().geot_check_index(index.data_ptr(), index.numel(), int(num_segments), cp,
                                          int(num_x_rows), _stream(index.device)))


def select(nnz: int, num_segments: int, F: int, reduce: str = "sum", gather: bool = False,
           stats: dict | None = None, weighted: bool = True) -> dict:
    """The selector's kernel choice for a shape (geot_select; host only). `weighted`
    says whether a fused gather has edge weights."""
    c = KernelChoice()
    sp = None
    if stats is not None:
        s = IndexStats(**{k: stats[k] for k, _ in IndexStats._fields_})
        sp = ctypes.byref(s)
    g = 0 if not gather else (1 if weighted else 2)
    _raise(lib().geot_select(int(nnz), int(num_segments), int(F), OPS[reduce], g, sp, ctypes.byref(c)))
    return c.as_dict()


def last_choice() -> dict:
    c = KernelChoice()
    _raise(lib().geot_last_choice(ctypes.byref(c)))
    return c.as_dict()


def profile_begin(max_records: int):
    _raise(lib().geot_profile_begin(int(max_records)))


def profile_end(capacity: int = 4096) -> list:
    buf = (ctypes.c_float * capacity)()
    n = ctypes.c_int32()
    _raise(lib().geot_profile_end(buf, capacity, ctypes.byref(n)))
    return [float(buf[i]) for i in range(min(n.value, capacity))]


def release_scratch():
    """Free the library's cached per-stream temporary buffers (geot_release_scratch)."""
    _raise(lib().geot_release_scratch())


def version() -> int:
    return int(lib().geot_version())
