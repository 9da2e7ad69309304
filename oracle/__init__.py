"""CPU oracle for the SpMM hot path -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.  The GPU library never calls it and
shares no code with it.  The arithmetic lives in ``oracle.c`` (plain C, fp64
accumulation, sequential within each row); this module only marshals numpy
arrays.  Each function names the passage of the paper it follows.

Parity status: every function below is pinned by the ``-m "not gpu"`` tests
in ``tests/test_oracle_pins.py``.  ``shape_class`` inside ``stats`` follows a
reading of the row-length shape classes, which the paper names without
thresholds; hand-built row-length vectors on each side of every threshold
of that reading pin it.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SO = os.path.join(_HERE, "liboracle.so")
_SRC = os.path.join(_HERE, "oracle.c")

INT_FIELDS = (
    "m", "k", "nnz", "row_min", "row_max", "row_q25", "row_q50", "row_q75", "empty_rows",
    "col_deg_max", "row_span_median", "diag_nnz", "nnzb4", "nnzb8", "nnzb16", "dense_tiles16",
    "dense_tile_nnz16", "bell16_width", "sell16_slots", "sell32_slots", "sell512_slots", "shape_class",
)
REAL_FIELDS = (
    "density", "row_mean", "row_cv", "empty_row_frac", "col_deg_mean", "col_deg_cv", "row_span_mean",
    "row_span_norm", "col_gap_mean", "diag_frac", "tile16_coverage", "dense_tile_frac",
    "dense_tile_nnz_frac", "rho_ell", "rho_sell16", "rho_sell32", "rho_sell512", "rho_bsr4", "rho_bsr8",
    "rho_bsr16", "rho_bell16", "nnz_per_tile16",
)
SHAPE_CLASSES = ("uniform", "moderate", "skewed", "power-law", "bimodal")


def build(force: bool = True) -> str:
    """Compile the oracle with gcc (test infrastructure; compiling it runs none of it)."""
    if force or not os.path.exists(_SO):
        tmp = _SO + ".tmp"
        subprocess.check_call(["gcc", "-O2", "-ffp-contract=off", "-fopenmp", "-fPIC", "-shared",
                               "-o", tmp, _SRC, "-lm"])
        os.replace(tmp, _SO)
    return _SO


_lib = None


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_SO):
            build()
        lib = ctypes.CDLL(_SO)
        P, i32, i64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64
        lib.oracle_spmm_csr.argtypes = [i32, i32, P, P, P, i32, P, P, P]
        lib.oracle_spmm_csr_rows.argtypes = [P, i64, P, P, P, i32, P, P, P]
        lib.oracle_spmm_csr_transposed.argtypes = [i32, i32, P, P, P, i32, P, P, P]
        lib.oracle_spmm_blocks.argtypes = [i32, i32, i32, P, i32, P, P, i32, P, P, P]
        lib.oracle_transpose.argtypes = [i32, i32, P, P, P, P, P, P]
        lib.oracle_block_counts.restype = i64
        lib.oracle_block_counts.argtypes = [i32, P, P, i32, P]
        lib.oracle_to_bsr.argtypes = [i32, P, P, P, i32, P, P, P]
        lib.oracle_to_bell.argtypes = [i32, P, P, P, i32, i32, P, P]
        lib.oracle_heavy_split.argtypes = [i32, P, i32, i32, P, P, P]
        lib.oracle_light_by_last_col.argtypes = [i32, P, P, i64, P, P]
        lib.oracle_chunks_by_mid_col.argtypes = [P, i64, P, P]
        lib.oracle_split_layout.argtypes = [i32, P, P, P, i32, i32, i64, P, P, P, P, P]
        lib.oracle_to_ell.argtypes = [i32, P, P, P, i32, P, P]
        lib.oracle_spmm_ell.argtypes = [i32, i32, P, P, i32, P, P, P]
        lib.oracle_to_sell.restype = i64
        lib.oracle_to_sell.argtypes = [i32, P, P, P, i32, i32, P, P, P, P]
        lib.oracle_spmm_sell.argtypes = [i32, i32, P, P, P, P, i32, P, P, P]
        lib.oracle_split_windows.restype = i64
        lib.oracle_split_windows.argtypes = [i64, P, P, i64, i32, i32, P, P, P]
        lib.oracle_spmm_split_windows.argtypes = [i32, i64, P, P, i64, P, P, P, i32, P, P, i32, P, P, P]
        lib.oracle_merge_split.argtypes = [i32, P, i32, P]
        lib.oracle_stats.argtypes = [i32, i32, P, P, i32, P, P, P, P]
        lib.oracle_threads.restype = i32
        lib.oracle_threads.argtypes = [i32]
        _lib = lib
    return _lib


def _p(a):
    return None if a is None else ctypes.c_void_p(a.ctypes.data)


def _i32(a):
    return np.ascontiguousarray(a, dtype=np.int32)


def _f32(a):
    return np.ascontiguousarray(a, dtype=np.float32)


def spmm(A, B):
    """C = A.B in fp64 with S = |A|.|B| (Sec. "Sparse Matrix Operators on GPUs").

    Returns (C64, S), both m x n float64."""
    B = _f32(B)
    n = B.shape[1]
    C = np.empty((A.m, n), np.float64)
    S = np.empty((A.m, n), np.float64)
    _load().oracle_spmm_csr(A.m, A.k, _p(_i32(A.rowptr)), _p(_i32(A.colidx)), _p(_f32(A.values)), n, _p(B),
                            _p(C), _p(S))
    return C, S


def threads(n: int = 0) -> int:
    """Sets the oracle's OpenMP thread count when n > 0; returns the count in
    effect.  No result depends on it (each row is summed by one thread)."""
    return int(_load().oracle_threads(int(n)))


def spmm_rows(A, B, rows, out=None):
    """Rows `rows` of (C64, S) only, for row-chunked checks at full size.
    `out` may pass a (C64, S) pair of float64 arrays of at least
    len(rows) x n elements to be filled (and returned) instead of new ones."""
    B = _f32(B)
    rows = _i32(rows)
    n = B.shape[1]
    if out is None:
        C = np.empty((rows.size, n), np.float64)
        S = np.empty((rows.size, n), np.float64)
    else:
        C, S = (np.asarray(x).reshape(-1)[:rows.size * n].reshape(rows.size, n) for x in out)
        if C.dtype != np.float64 or S.dtype != np.float64 or not (C.flags.c_contiguous and S.flags.c_contiguous):
            raise ValueError("out must hold two contiguous float64 arrays")
    _load().oracle_spmm_csr_rows(_p(rows), rows.size, _p(_i32(A.rowptr)), _p(_i32(A.colidx)),
                                 _p(_f32(A.values)), n, _p(B), _p(C), _p(S))
    return C, S


def spmm_transposed(A, B):
    """C = A^T.B by a scatter over the rows of A (no transposed copy)."""
    B = _f32(B)
    n = B.shape[1]
    C = np.empty((A.k, n), np.float64)
    S = np.empty((A.k, n), np.float64)
    _load().oracle_spmm_csr_transposed(A.m, A.k, _p(_i32(A.rowptr)), _p(_i32(A.colidx)), _p(_f32(A.values)), n,
                                       _p(B), _p(C), _p(S))
    return C, S


def transpose(A):
    """A^T as (rowptr[k+1], colidx[nnz], values[nnz]) by counting sort."""
    tr = np.empty(A.k + 1, np.int32)
    tc = np.empty(A.nnz, np.int32)
    tv = np.empty(A.nnz, np.float32)
    _load().oracle_transpose(A.m, A.k, _p(_i32(A.rowptr)), _p(_i32(A.colidx)), _p(_f32(A.values)), _p(tr), _p(tc),
                             _p(tv))
    return tr, tc, tv


def block_counts(A, b):
    """Occupied b x b blocks per block-row (Eq. format-expansion, nnzb_b)."""
    mb = (A.m + b - 1) // b
    counts = np.empty(mb, np.int32)
    total = _load().oracle_block_counts(A.m, _p(_i32(A.rowptr)), _p(_i32(A.colidx)), b, _p(counts))
    return total, counts


def to_bsr(A, b):
    """BSR(b): (bptr[mb+1], bcol[nnzb], bval[nnzb, b, b])."""
    nnzb, _ = block_counts(A, b)
    mb = (A.m + b - 1) // b
    bptr = np.empty(mb + 1, np.int32)
    bcol = np.empty(nnzb, np.int32)
    bval = np.empty((nnzb, b, b), np.float32)
    _load().oracle_to_bsr(A.m, _p(_i32(A.rowptr)), _p(_i32(A.colidx)), _p(_f32(A.values)), b, _p(bptr), _p(bcol),
                          _p(bval))
    return bptr, bcol, bval


def to_bell(A, b):
    """Blocked-ELL(b): (width, bcol[mb, width], bval[mb, width, b, b])."""
    _, counts = block_counts(A, b)
    mb = (A.m + b - 1) // b
    width = int(counts.max()) if counts.size else 0
    bcol = np.empty((mb, width), np.int32)
    bval = np.empty((mb, width, b, b), np.float32)
    _load().oracle_to_bell(A.m, _p(_i32(A.rowptr)), _p(_i32(A.colidx)), _p(_f32(A.values)), b, width, _p(bcol),
                           _p(bval))
    return width, bcol, bval


def spmm_bsr(m, k, b, bptr, bcol, bval, B):
    """Block SpMM in fp64 over every stored slot, zero fill included."""
    B = _f32(B)
    n = B.shape[1]
    C = np.empty((m, n), np.float64)
    S = np.empty((m, n), np.float64)
    _load().oracle_spmm_blocks(m, k, b, _p(_i32(bptr)), 0, _p(_i32(bcol)), _p(_f32(bval)), n, _p(B), _p(C), _p(S))
    return C, S


def spmm_bell(m, k, b, width, bcol, bval, B):
    B = _f32(B)
    n = B.shape[1]
    C = np.empty((m, n), np.float64)
    S = np.empty((m, n), np.float64)
    _load().oracle_spmm_blocks(m, k, b, None, width, _p(_i32(bcol)), _p(_f32(bval)), n, _p(B), _p(C), _p(S))
    return C, S


def to_ell(A):
    """ELL: (width, ecol[m, width], eval[m, width]); padding column -1, value +0."""
    width = int(np.diff(A.rowptr).max()) if A.m else 0
    ecol = np.empty((A.m, width), np.int32)
    evals = np.empty((A.m, width), np.float32)
    _load().oracle_to_ell(A.m, _p(_i32(A.rowptr)), _p(_i32(A.colidx)), _p(_f32(A.values)), width, _p(ecol),
                          _p(evals))
    return width, ecol, evals


def spmm_ell(m, width, ecol, evals, B):
    """ELL SpMM in fp64, padding skipped."""
    B = _f32(B)
    n = B.shape[1]
    C = np.empty((m, n), np.float64)
    S = np.empty((m, n), np.float64)
    _load().oracle_spmm_ell(m, width, _p(_i32(ecol)), _p(_f32(evals)), n, _p(B), _p(C), _p(S))
    return C, S


def to_sell(A, C, sigma):
    """SELL-C-sigma: (perm[m], slice_ptr[ns+1] int64, col[total], val[total])."""
    ns = (A.m + C - 1) // C
    rp, ci, vv = _i32(A.rowptr), _i32(A.colidx), _f32(A.values)
    perm = np.empty(A.m, np.int32)
    sp = np.empty(ns + 1, np.int64)
    total = _load().oracle_to_sell(A.m, _p(rp), _p(ci), _p(vv), C, sigma, _p(perm), _p(sp), None, None)
    col = np.empty(total, np.int32)
    val = np.empty(total, np.float32)
    _load().oracle_to_sell(A.m, _p(rp), _p(ci), _p(vv), C, sigma, _p(perm), _p(sp), _p(col), _p(val))
    return perm, sp, col, val


def spmm_sell(m, C, perm, slice_ptr, col, val, B):
    B = _f32(B)
    n = B.shape[1]
    Cm = np.empty((m, n), np.float64)
    S = np.empty((m, n), np.float64)
    _load().oracle_spmm_sell(m, C, _p(_i32(perm)), _p(np.ascontiguousarray(slice_ptr, np.int64)), _p(_i32(col)),
                             _p(_f32(val)), n, _p(B), _p(Cm), _p(S))
    return Cm, S


def split_windows(lptr, colidx, n_light, R, cap):
    """Packed column windows over a heavy-split layout (lptr, colidx as
    split_layout returns them): windows of R light-list positions, each
    staging the columns two or more of its rows use (at most `cap`, the most
    used kept, ties to the smaller column), ascending.  Returns (win_ptr,
    win_cols, code) with code[p] = -2 - (staged position) or the column."""
    lptr, colidx = _i32(lptr), _i32(colidx)
    nnz = colidx.size
    nw = (int(n_light) + R - 1) // R
    total = _load().oracle_split_windows(int(n_light), _p(lptr), _p(colidx), nnz, R, cap, None, None, None)
    win_ptr = np.empty(nw + 1, np.int32)
    win_cols = np.empty(max(total, 0), np.int32)
    code = np.empty(nnz, np.int32)
    _load().oracle_split_windows(int(n_light), _p(lptr), _p(colidx), nnz, R, cap, _p(win_ptr), _p(win_cols), _p(code))
    return win_ptr, win_cols, code


def spmm_split_windows(m, light, lptr, chunks, code, vals, R, win_ptr, win_cols, B):
    """C = A.B in fp64 over the windowed split layout (light rows through their
    windows' codes, heavy rows through their chunks)."""
    B = _f32(B)
    n = B.shape[1]
    light, lptr = _i32(light), _i32(lptr)
    chunks = np.ascontiguousarray(np.asarray(chunks, np.int32).reshape(-1, 3))
    C = np.empty((m, n), np.float64)
    S = np.empty((m, n), np.float64)
    _load().oracle_spmm_split_windows(m, light.size, _p(light), _p(lptr), len(chunks), _p(chunks), _p(_i32(code)),
                                      _p(_f32(vals)), R, _p(_i32(win_ptr)), _p(_i32(win_cols)), n, _p(B), _p(C), _p(S))
    return C, S


def heavy_split(A_rowptr, m, T, c):
    """Light rows (r < T) and (row, begin, end) chunks of at most c nonzeros."""
    rowptr = _i32(A_rowptr)
    counts = np.zeros(2, np.int64)
    _load().oracle_heavy_split(m, _p(rowptr), T, c, None, None, _p(counts))
    light = np.empty(int(counts[0]), np.int32)
    chunks = np.empty((int(counts[1]), 3), np.int32)
    _load().oracle_heavy_split(m, _p(rowptr), T, c, _p(light), _p(chunks), _p(counts))
    return light, chunks


def light_by_last_col(A, light):
    """The light rows ordered by the column of their last nonzero, ties by row
    (an empty row last)."""
    light = _i32(light)
    out = np.empty_like(light)
    _load().oracle_light_by_last_col(A.k, _p(_i32(A.rowptr)), _p(_i32(A.colidx)), light.size, _p(light), _p(out))
    return out


def chunks_by_mid_col(colidx, chunks):
    """Processing order of the split layout's chunks (row, begin, end): by
    the column of the entry at floor((begin + end) / 2), ties by chunk index.
    `colidx` is the split layout's column array."""
    chunks = np.ascontiguousarray(np.asarray(chunks, np.int32).reshape(-1, 3))
    order = np.empty(len(chunks), np.int32)
    _load().oracle_chunks_by_mid_col(_p(_i32(colidx)), len(chunks), _p(chunks), _p(order))
    return order


def split_layout(A, T, c, light):
    """The heavy-split layout: the light rows' entries in the order of `light`,
    then the heavy rows' (r >= T) in ascending order.  Returns (lptr, colidx,
    values, chunks) with chunks (row, begin, end) in the new coordinates."""
    light = _i32(light)
    _, chunks0 = heavy_split(A.rowptr, A.m, T, c)
    lptr = np.empty(light.size + 1, np.int32)
    col = np.empty(A.nnz, np.int32)
    val = np.empty(A.nnz, np.float32)
    chunks = np.empty((len(chunks0), 3), np.int32)
    _load().oracle_split_layout(A.m, _p(_i32(A.rowptr)), _p(_i32(A.colidx)), _p(np.ascontiguousarray(A.values, np.float32)),
                                T, c, light.size, _p(light), _p(lptr), _p(col), _p(val), _p(chunks))
    return lptr, col, val, chunks


def merge_split(A_rowptr, m, U):
    """(U+1) x 2 merge-path coordinates (rows consumed, nonzeros consumed)."""
    rowptr = _i32(A_rowptr)
    coords = np.empty((U + 1, 2), np.int32)
    _load().oracle_merge_split(m, _p(rowptr), U, _p(coords))
    return coords


def stats(A, dense_threshold: int = 128) -> dict:
    """Structural statistics (Sec. "Structural Features and Overhead Modeling")."""
    ints = np.zeros(len(INT_FIELDS), np.int64)
    reals = np.zeros(len(REAL_FIELDS), np.float64)
    rh = np.zeros(33, np.int64)
    fh = np.zeros(8, np.int64)
    _load().oracle_stats(A.m, A.k, _p(_i32(A.rowptr)), _p(_i32(A.colidx)), dense_threshold, _p(ints), _p(reals),
                         _p(rh), _p(fh))
    out = {name: int(v) for name, v in zip(INT_FIELDS, ints)}
    out.update({name: float(v) for name, v in zip(REAL_FIELDS, reals)})
    out["row_hist"] = rh
    out["fill16_hist"] = fh
    return out
