"""The C-ABI library: loads, exports every declared symbol, and its host-side logic
(argument checks, forced-choice validation, selector) runs without a GPU.

Every call here returns before any device work: invalid arguments and
impossible kernel choices are rejected on the host, and geot_select touches
no device memory. Fake (never dereferenced) pointer values stand in for
device buffers.
"""
import ctypes
import os
import re

import pytest

import paper_2404_03019_amd as geot
from paper_2404_03019_amd.geot import KernelChoice, lib

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "geot.h")

SUCCESS, INVALID, NOT_SORTED, OUT_OF_RANGE, HIP, UNSUPPORTED = range(6)
FAKE = 0x10000000  # 256-byte aligned, never dereferenced


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(geot_[a-z_0-9]+)\s*\(", text)))


def test_header_declares_the_entry_points():
    names = declared_functions()
    for n in ("geot_segment_reduce", "geot_gather_scatter", "geot_select", "geot_index_stats",
              "geot_check_index", "geot_segment_reduce_with", "geot_gather_scatter_with"):
        assert n in names


def test_library_exports_every_declared_symbol():
    L = lib()
    missing = [n for n in declared_functions() if not hasattr(L, n)]
    assert not missing, missing


def test_version_and_status_strings():
    L = lib()
    assert geot.version() == 1
    assert L.geot_status_string(0) == b"success"
    assert L.geot_status_string(2) == b"index not sorted"
    assert L.geot_status_string(99) == b"unknown status"


def _sr(src, idx, nnz, S, F, op, out, choice=None):
    L = lib()
    return L.geot_segment_reduce_with(src, idx, nnz, S, F, op, out, None,
                                      ctypes.byref(choice) if choice is not None else None)


def _gs(X, nx, col, w, row, nnz, R, F, op, out, choice=None):
    L = lib()
    return L.geot_gather_scatter_with(X, nx, col, w, row, nnz, R, F, op, out, None,
                                      ctypes.byref(choice) if choice is not None else None)


def _detail():
    return lib().geot_last_error_detail().decode()


def test_invalid_arguments_are_rejected_on_the_host():
    out = FAKE + (1 << 30)
    assert _sr(FAKE, FAKE + (1 << 28), 10, 4, 3, 7, out) == INVALID and "op" in _detail()
    st = geot.geot.IndexStats()
    assert lib().geot_index_stats(FAKE, 10, 1 << 31, ctypes.byref(st), None) == INVALID and "2^31" in _detail()
    assert _sr(FAKE, FAKE + (1 << 28), -1, 4, 3, 0, out) == INVALID
    assert _sr(FAKE, FAKE + (1 << 28), 10, -4, 3, 0, out) == INVALID
    assert _sr(FAKE, FAKE + (1 << 28), 10, 4, -3, 0, out) == INVALID
    assert _sr(None, FAKE, 10, 4, 3, 0, out) == INVALID and "src" in _detail()
    assert _sr(FAKE, None, 10, 4, 3, 0, out) == INVALID and "index" in _detail()
    assert _sr(FAKE, FAKE + (1 << 28), 10, 4, 3, 0, None) == INVALID and "out" in _detail()
    # out overlapping src, or the index
    assert _sr(FAKE, FAKE + (1 << 28), 100, 4, 8, 0, FAKE + 64) == INVALID and "overlap" in _detail()
    assert _sr(FAKE, FAKE + (1 << 28), 100, 4, 8, 0, FAKE + (1 << 28) + 8) == INVALID
    # size overflow
    assert _sr(FAKE, FAKE, 1 << 61, 4, 8, 0, out) == INVALID


def test_noops_return_success_without_device_work():
    assert _sr(None, None, 0, 0, 5, 0, None) == SUCCESS
    assert _sr(None, None, 10, 5, 0, 0, None) == SUCCESS
    assert _gs(None, 0, None, None, None, 10, 0, 4, 0, None) == SUCCESS


def test_gather_arguments_are_checked():
    out = FAKE + (1 << 30)
    assert _gs(FAKE, 10, None, None, FAKE + (1 << 26), 5, 3, 4, 0, out) == INVALID and "col" in _detail()
    assert _gs(None, 10, FAKE, None, FAKE + (1 << 26), 5, 3, 4, 0, out) == INVALID and "X" in _detail()
    assert _gs(FAKE, 0, FAKE + (1 << 27), None, FAKE + (1 << 26), 5, 3, 4, 0, out) == INVALID
    assert _gs(FAKE, -1, FAKE, None, FAKE, 5, 3, 4, 0, out) == INVALID


@pytest.mark.parametrize("choice", [
    dict(family=7), dict(vec=3), dict(lanes=3), dict(lanes=128), dict(rows=-1), dict(rows=5000),
    dict(family=2, lanes=16, groups=8), dict(family=2, groups=3), dict(flags=8), dict(flags=3), dict(flags=7),
    dict(vec=8), dict(flags=1, lanes=2),   # a 2-lane x 4-float tile is 32 bytes: no non-temporal rows
    dict(flags=1, family=2),
])
def test_impossible_forced_choices_are_unsupported(choice):
    c = geot.geot._choice(choice)
    out = FAKE + (1 << 30)
    assert _sr(FAKE, FAKE + (1 << 28), 1000, 10, 32, 0, out, c) == UNSUPPORTED


def test_non_temporal_loads_are_refused_for_the_gather_form():
    c = geot.geot._choice(dict(flags=1))
    out = FAKE + (1 << 30)
    assert _gs(FAKE, 10, FAKE + (1 << 27), None, FAKE + (1 << 26), 5, 3, 32, 0, out, c) == UNSUPPORTED


def test_selector_reports_the_load_policy():
    assert geot.select(114_615_892, 232_965, 32, "sum")["flags"] == 1       # 128-byte rows
    assert geot.select(2_000_000, 100_000, 8, "sum")["flags"] == 0          # 32-byte rows
    # the SpMM shape: ordinary loads, two 64-column tiles one after another
    c = geot.select(61_859_140, 2_449_029, 128, "sum", gather=True)
    assert c["flags"] == 4 and c["lanes"] * c["vec"] == 64, c


def test_selector_is_a_host_function():
    c = geot.select(114_615_892, 232_965, 32, "sum")
    assert c["family"] == 1 and c["vec"] == 4 and c["lanes"] == 8 and c["rows"] >= 1
    c = geot.select(61_859_140, 2_449_029, 128, "sum", gather=True)
    assert c["vec"] == 4 and c["lanes"] in (8, 16, 32)
    for F in (1, 2, 3, 4, 5, 8, 15, 16, 17, 33, 64, 100, 128, 255, 256, 257, 1000):
        c = geot.select(2_000_000, 100_000, F, "max")
        # fp32 rows of any width >= 3 move in 4-float vectors (the last overlapping), 3 -> 3
        want = F if F < 3 else (3 if F == 3 else 4)
        assert c["family"] in (1, 2) and c["vec"] == (want if c["family"] == 1 else c["vec"])
        assert c["family"] == 1 or F % c["vec"] == 0
        assert c["lanes"] in (1, 2, 4, 8, 16, 32, 64)
        if F <= 256:  # one column tile covers the row
            nt = 1 if c["lanes"] < 64 else max(1, -(-F // (64 * c["vec"])))
            assert c["lanes"] * c["vec"] * nt >= F
    assert lib().geot_select(10, 10, 4, 9, 0, None, ctypes.byref(KernelChoice())) == INVALID
    assert lib().geot_select(-1, 10, 4, 0, 0, None, ctypes.byref(KernelChoice())) == INVALID


def test_selector_uses_stats_when_given():
    even = dict(nnz=16 * 1000, num_segments=1000, max_len=16, num_empty=0, sum_len_sq=256 * 1000,
                mean_len=16.0, var_len=0.0)
    skew = dict(nnz=16 * 1000, num_segments=1000, max_len=9000, num_empty=900,
                sum_len_sq=9000 ** 2, mean_len=16.0, var_len=8.0e4)
    assert geot.select(16000, 1000, 64, "mean", stats=skew)["family"] == 1
    assert geot.select(16000, 1000, 64, "mean", stats=even)["family"] in (1, 2)


def test_backward_arguments_are_checked_on_the_host():
    L = lib()
    g, idx, out, gs = FAKE, FAKE + (1 << 26), FAKE + (1 << 27), FAKE + (1 << 30)
    # unknown op, negative sizes, max without src/out, overlap, no rows = no-op
    assert L.geot_segment_reduce_backward(g, idx, 10, 4, 3, 9, None, None, gs, None) == INVALID
    assert L.geot_segment_reduce_backward(g, idx, -1, 4, 3, 0, None, None, gs, None) == INVALID
    assert L.geot_segment_reduce_backward(g, idx, 10, 4, 3, 2, None, out, gs, None) == INVALID
    assert L.geot_segment_reduce_backward(g, idx, 10, 4, 8, 0, None, None, g + 16, None) == INVALID
    assert L.geot_segment_reduce_backward(g, idx, 10, 0, 3, 0, None, None, gs, None) == INVALID
    assert L.geot_segment_reduce_backward(None, None, 0, 4, 3, 0, None, None, None, None) == SUCCESS
    X, col, row, gx, gw = FAKE, FAKE + (1 << 25), FAKE + (1 << 26), FAKE + (1 << 31), FAKE + (1 << 32)
    # grad_weight without weight, max without out, nothing requested = no-op
    assert L.geot_gather_scatter_backward(X, 10, col, None, row, 5, 3, 4, 0, g, None, gx, gw, None) == INVALID
    assert L.geot_gather_scatter_backward(X, 10, col, None, row, 5, 3, 4, 2, g, None, gx, None, None) == INVALID
    assert L.geot_gather_scatter_backward(X, 10, None, None, row, 5, 3, 4, 0, g, None, gx, None, None) == INVALID
    assert L.geot_gather_scatter_backward(X, 10, col, None, row, 5, 3, 4, 0, g, None, None, None, None) == SUCCESS


def test_typed_arguments_are_checked_on_the_host():
    L = lib()
    src, idx, out = FAKE, FAKE + (1 << 28), FAKE + (1 << 30)
    sp = geot.geot._choice(dict(family="sp"))
    # unknown storage or index type
    assert L.geot_segment_reduce_typed(src, 3, idx, 0, 10, 4, 8, 0, out, None, None) == INVALID
    assert "data type" in _detail()
    assert L.geot_segment_reduce_typed(src, 1, idx, 2, 10, 4, 8, 0, out, None, None) == INVALID
    assert "index type" in _detail()
    assert L.geot_gather_scatter_typed(src, 5, 10, idx, None, idx + 4096, 0, 5, 3, 4, 0, out, None,
                                       None) == INVALID
    # overlap is judged with the element sizes: 100 x 8 bf16 = 1600 bytes, 100 int32 ids = 400 bytes
    assert L.geot_segment_reduce_typed(src, 1, idx, 1, 100, 4, 8, 0, src + 1500, None, None) == INVALID
    assert L.geot_segment_reduce_typed(src, 1, idx, 1, 100, 4, 8, 0, idx + 396, None, None) == INVALID
    # the segment-parallel family takes fp32 with int64 ids only
    assert L.geot_segment_reduce_typed(src, 1, idx, 0, 1000, 10, 32, 0, out, None, ctypes.byref(sp)) == UNSUPPORTED
    assert L.geot_segment_reduce_typed(src, 0, idx, 1, 1000, 10, 32, 0, out, None, ctypes.byref(sp)) == UNSUPPORTED
    # no-ops as in the fp32 call
    assert L.geot_segment_reduce_typed(None, 1, None, 1, 0, 0, 5, 0, None, None, None) == SUCCESS


def test_transpose_arguments_are_checked_on_the_host():
    L = lib()
    col, row, w = FAKE, FAKE + (1 << 26), FAKE + (1 << 27)
    a, b, c = FAKE + (1 << 30), FAKE + (1 << 31), FAKE + (1 << 32)
    assert L.geot_transpose_edges(col, 10, w, row, 100, 5, 2, a, b, c, None) == INVALID   # max
    assert L.geot_transpose_edges(col, 10, w, row, -1, 5, 0, a, b, c, None) == INVALID
    assert L.geot_transpose_edges(col, 10, w, row, 100, 5, 0, None, b, c, None) == INVALID
    assert L.geot_transpose_edges(col, 10, w, row, 100, 5, 0, col + 8, b, c, None) == INVALID  # overlap
    assert L.geot_transpose_edges(col, 10, w, row, 100, 5, 0, a, a + 64, c, None) == INVALID  # outputs overlap
    assert L.geot_transpose_edges(None, 10, None, None, 0, 5, 0, None, None, None, None) == SUCCESS


def test_workspace_size_query_on_the_host():
    """The *_workspace_size queries are host functions: sizes, errors, and monotone in the
    input (a larger input never needs less)."""
    c1 = geot.workspace_size(65_536, 4096, 32)
    assert c1 >= 1_500_000   # the empty-run list's counters and records, at least
    assert geot.workspace_size(0, 4096, 32) == 0 and geot.workspace_size(10, 0, 32) == 0
    assert geot.workspace_size(10, 4, 0) == 0
    big = geot.workspace_size(114_615_892, 232_965, 32)
    assert big > c1
    assert geot.workspace_size(61_859_140, 2_449_029, 128, gather=True) > c1
    assert geot.workspace_size(61_859_140, 2_449_029, 128, gather=True, weighted=False) > c1
    # segment-parallel: the segment starts
    sp = geot.workspace_size(10_000, 5_000, 8, choice=dict(family="sp"))
    assert sp >= 5_001 * 8
    for bad in ((-1, 4, 3), (10, -4, 3), (10, 4, -3), (10, 1 << 31, 3)):
        with pytest.raises(geot.GeotError):
            geot.workspace_size(*bad)
    with pytest.raises(geot.GeotError):
        geot.workspace_size(10, 4, 3, choice=dict(family="ep", lanes=3))
    n = ctypes.c_size_t()
    assert lib().geot_segment_reduce_workspace_size(10, 4, 3, 7, None, ctypes.byref(n)) == INVALID
    assert lib().geot_segment_reduce_workspace_size(10, 4, 3, 0, None, None) == INVALID


def test_workspace_calls_check_on_the_host():
    """A workspace that is missing, misaligned, too small or overlapping an argument is
    rejected before any device work."""
    L = lib()
    need = geot.workspace_size(1000, 10, 4)
    src, idx, out, ws = FAKE, FAKE + (1 << 24), FAKE + (1 << 26), FAKE + (1 << 28)
    call = lambda w, b: L.geot_segment_reduce_ws(src, idx, 1000, 10, 4, 0, out, w, b, None, None)
    assert call(None, need) == INVALID and "NULL" in _detail()
    assert call(ws + 64, need) == INVALID and "aligned" in _detail()
    assert call(ws, 1 << 20) == INVALID and "needs" in _detail()   # below the empty-run list alone
    assert call(out, need) == INVALID and "overlaps" in _detail()
    assert L.geot_gather_scatter_ws(src, 100, idx, None, idx + 8192, 1000, 10, 4, 0, out, ws, 16, None,
                                    None) == INVALID and "needs" in _detail()
    # nothing to do: no workspace needed
    assert L.geot_segment_reduce_ws(src, idx, 1000, 0, 4, 0, out, None, 0, None, None) == SUCCESS


def test_recipient_calls_check_on_the_host():
    """The max-with-recipients calls: a missing or overlapping arg, 2^32 - 1 rows or more,
    a segment-parallel choice, and an op other than max for the recorded gradient, all
    rejected before any device work."""
    L = lib()
    src, idx, out, arg = FAKE, FAKE + (1 << 28), FAKE + (1 << 30), FAKE + (1 << 31)
    F32, I64 = 0, 0
    fwd = lambda a, n=1000, c=None: L.geot_segment_reduce_max_arg(src, F32, idx, I64, n, 10, 4, out, a, None,
                                                                  ctypes.byref(c) if c is not None else None)
    assert fwd(None) == INVALID and "arg" in _detail()
    assert fwd(out + 16) == INVALID and "overlap" in _detail()
    assert fwd(src + 64) == INVALID and "overlap" in _detail()
    far = lambda k: FAKE + (k << 40)   # room for 2^32 rows of every array
    assert L.geot_segment_reduce_max_arg(far(0), F32, far(1), I64, (1 << 32) - 1, 10, 4, far(2), far(3), None,
                                         None) == UNSUPPORTED and "2^32" in _detail()
    assert fwd(arg, c=KernelChoice(2, 0, 0, 0, 0, 0)) == UNSUPPORTED and "element-parallel" in _detail()
    X, col, row = FAKE, FAKE + (1 << 26), FAKE + (1 << 27)
    assert L.geot_gather_scatter_max_arg(X, F32, 100, col, None, row, I64, 1000, 10, 4, out, None, None,
                                         None) == INVALID
    g, gs = FAKE + (1 << 32), FAKE + (1 << 33)
    assert L.geot_segment_reduce_backward_max_arg(g, idx, I64, 1000, 10, 4, None, gs, F32, None) == INVALID
    assert L.geot_segment_reduce_backward_max_arg(g, idx, I64, (1 << 32) - 1, 10, 4, arg, gs, F32,
                                                  None) == UNSUPPORTED
    assert L.geot_gather_scatter_backward_max_arg(X, F32, 100, col, None, row, I64, 1000, 10, 4, g, None, gs,
                                                  None, None) == INVALID
    # no rows: nothing to do, no device work
    assert L.geot_segment_reduce_backward_max_arg(g, idx, I64, 0, 10, 4, arg, gs, F32, None) == SUCCESS
