"""Python binding of the MI355X SpMM library (libsparseditto.so).

Argument marshalling only: every step of the path (validation, analysis,
planning, conversion, and the SpMM itself) runs inside the native library,
whose C ABI is declared in ``include/sparseditto.h``.  The functions keep the
C names.  Dense operands are passed as device pointers: either integers or
objects with ``data_ptr()`` (PyTorch tensors); PyTorch is used by callers for
device memory and streams only.

If the shared library is missing, importing this package raises: there is no
fallback implementation.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libsparseditto.so")

SD_OK = 0
SD_ERR_INVALID_VALUE = 1
SD_ERR_INVALID_CSR = 2
SD_ERR_UNSUPPORTED = 3
SD_ERR_OUT_OF_MEMORY = 4
SD_ERR_HIP = 5
SD_ERR_OVERFLOW = 6
SD_ERR_NO_DEVICE = 7
SD_ERR_IO = 8

SD_FMT_AUTO, SD_FMT_CSR_ROW, SD_FMT_CSR_SPLIT, SD_FMT_CSR_MERGE, SD_FMT_BSR, SD_FMT_BELL, SD_FMT_ELL = range(7)
FAMILIES = {"auto": 0, "csr_row": 1, "csr_split": 2, "csr_merge": 3, "bsr": 4, "bell": 5, "ell": 6, "win": 7, "sell": 8}
FAMILY_NAMES = {v: k for k, v in FAMILIES.items()}
WG_ORDERS = {"auto": 0, "xcd_contiguous": 1, "round_robin": 2, "chunked": 3}
SD_ENGINE_AUTO, SD_ENGINE_MFMA, SD_ENGINE_VALU = 0, 1, 2
ENGINES = {"auto": 0, "mfma": 1, "valu": 2}
CACHE_POLICIES = {"auto": 0, "normal": 1, "tiered": 2, "nontemporal": 3}
PLACEMENT_CURRENT, PLACEMENT_DEVICE, PLACEMENT_HOST = 0, 1, 2

SD_EXPORT_ROWPTR = 1
SD_EXPORT_COLIDX = 2
SD_EXPORT_VALUES = 3
SD_EXPORT_LIGHT_ROWS = 4
SD_EXPORT_CHUNKS = 5
SD_EXPORT_MERGE_COORDS = 6
SD_EXPORT_BLOCK_PTR = 7
SD_EXPORT_BLOCK_COL = 8
SD_EXPORT_BLOCK_VAL = 9
SD_EXPORT_ELL_COL = 10
SD_EXPORT_ELL_VAL = 11
SD_EXPORT_WIN_PTR = 12
SD_EXPORT_WIN_COLS = 13
SD_EXPORT_WIN_CODE = 14
SD_EXPORT_WIN_VAL = 15
SD_EXPORT_SELL_PERM = 16
SD_EXPORT_SELL_SLICE_PTR = 17
SD_EXPORT_SELL_COL = 18
SD_EXPORT_SELL_VAL = 19
SD_EXPORT_CHUNK_ORDER = 20
_EXPORT_DTYPE = {1: np.int32, 2: np.int32, 3: np.float32, 4: np.int32, 5: np.int32, 6: np.int32, 7: np.int32,
                 8: np.int32, 9: np.float32, 10: np.int32, 11: np.float32, 12: np.int32, 13: np.int32,
                 14: np.int32, 15: np.float32, 16: np.int32, 17: np.int64, 18: np.int32, 19: np.float32,
                 20: np.int32}

_i32, _i64, _dbl, _P = ctypes.c_int32, ctypes.c_int64, ctypes.c_double, ctypes.c_void_p


class sd_csr_t(ctypes.Structure):
    _fields_ = [("m", _i32), ("k", _i32), ("nnz", _i64), ("rowptr", _P), ("colidx", _P), ("values", _P)]


_STATS_INT = ["m", "k", "nnz", "row_min", "row_max", "row_q25", "row_q50", "row_q75", "empty_rows",
              "col_deg_max", "row_span_median", "diag_nnz", "nnzb4", "nnzb8", "nnzb16", "dense_tiles16",
              "dense_tile_nnz16", "bell16_width", "sell16_slots", "sell32_slots", "sell512_slots", "shape_class",
              "dense_threshold"]
_STATS_REAL = ["density", "row_mean", "row_cv", "empty_row_frac", "col_deg_mean", "col_deg_cv", "row_span_mean",
               "row_span_norm", "col_gap_mean", "diag_frac", "tile16_coverage", "dense_tile_frac",
               "dense_tile_nnz_frac", "rho_ell", "rho_sell16", "rho_sell32", "rho_sell512", "rho_bsr4", "rho_bsr8",
               "rho_bsr16", "rho_bell16", "nnz_per_tile16"]


class sd_stats_t(ctypes.Structure):
    _fields_ = ([(f, _i64) for f in _STATS_INT] + [(f, _dbl) for f in _STATS_REAL] +
                [("row_hist", _i64 * 33), ("fill16_hist", _i64 * 8)])


class sd_plan_opts_t(ctypes.Structure):
    _fields_ = [("force", _i32), ("heavy_threshold", _i32), ("chunk_nnz", _i32), ("units", _i32),
                ("engine", _i32), ("transpose", _i32), ("placement", _i32), ("device", _i32),
                ("dense_threshold", _i32), ("rows_per_group", _i32), ("gather_unroll", _i32),
                ("cache_policy", _i32), ("hot_budget_kib", _i32), ("search", _i32), ("col_tile", _i32),
                ("window_rows", _i32), ("wg_order", _i32), ("wg_chunk", _i32), ("sell_sigma", _i32),
                ("row_slices", _i32), ("light_order", _i32), ("chunk_order", _i32)]


_INFO_FIELDS = [
    ("family", _i32), ("engine", _i32), ("transpose", _i32), ("device", _i32),
    ("m", _i64), ("k", _i64), ("n", _i64), ("nnz", _i64),
    ("heavy_threshold", _i64), ("chunk_nnz", _i64), ("n_light", _i64), ("n_heavy", _i64), ("n_chunks", _i64),
    ("units", _i64), ("merge_len", _i64),
    ("block", _i64), ("nnzb", _i64), ("bell_width", _i64), ("block_rows", _i64),
    ("m_rep", _i64), ("workspace", _i64), ("d_r", _i64), ("d_s", _i64), ("m_r", _i64), ("m_t", _i64),
    ("compulsory_bytes", _i64), ("l2_bytes", _i64), ("mall_bytes", _i64),
    ("q_r", _dbl), ("q_t", _dbl), ("q_r_mall", _dbl), ("q_t_mall", _dbl),
    ("work_units", _i64), ("units_per_cu", _dbl), ("cu_count", _i32),
    ("block_threads", _i32), ("max_threads", _i32), ("regs_per_thread", _i32), ("lds_bytes", _i32),
    ("max_lds_bytes", _i32), ("legal", _i32), ("rows_per_group", _i32), ("lanes_per_row", _i32),
    ("gather_unroll", _i32), ("cache_policy", _i32), ("row_slices", _i32), ("light_order", _i32),
    ("chunk_order", _i32), ("reserved", _i32 * 1),
    ("hot_columns", _i64), ("hot_nnz", _i64), ("ell_width", _i64),
    ("search_candidates", _i32), ("search_cache_hit", _i32), ("search_best_ms", _dbl), ("search_rule_ms", _dbl),
    ("col_tile", _i32), ("col_passes", _i32), ("window_rows", _i32), ("window_max", _i32),
    ("window_staged", _i64), ("window_staged_uses", _i64), ("wg_order", _i32), ("wg_chunk", _i32), ("device_built", _i32), ("reserved2", _i32 * 1), ("reach", _i64),
    ("sell_c", _i32), ("sell_sigma", _i32), ("sell_slices", _i64), ("sell_slots", _i64),
]


class sd_plan_info_t(ctypes.Structure):
    _fields_ = _INFO_FIELDS


class SparseDittoError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        detail = _lib.sd_last_error().decode() if status == SD_ERR_HIP else ""
        super().__init__(f"{where}: {_lib.sd_status_string(status).decode()}" + (f" ({detail})" if detail else ""))


def _load():
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built; run __graft_entry__.build() or "
                          "python paper_2608_05033_amd/_build.py")
    lib = ctypes.CDLL(LIB_PATH)
    lib.sd_analyze.argtypes = [ctypes.POINTER(sd_csr_t), _i32, ctypes.POINTER(sd_stats_t)]
    lib.sd_analyze_device.argtypes = [ctypes.POINTER(sd_csr_t), _i32, ctypes.POINTER(sd_stats_t), _P]
    lib.sd_plan.argtypes = [ctypes.POINTER(sd_csr_t), _i32, ctypes.POINTER(_P)]
    lib.sd_plan_ex.argtypes = [ctypes.POINTER(sd_csr_t), _i32, ctypes.POINTER(sd_plan_opts_t), ctypes.POINTER(_P)]
    lib.sd_plan_device.argtypes = [ctypes.POINTER(sd_csr_t), _i32, ctypes.POINTER(sd_plan_opts_t), _P,
                                   ctypes.POINTER(_P)]
    lib.sd_spmm.argtypes = [_P, _P, _P, _P]
    lib.sd_spmm_merge_noalloc.argtypes = [ctypes.POINTER(sd_csr_t), _i32, _i32, _P, _P, _P]
    lib.sd_plan_info.argtypes = [_P, ctypes.POINTER(sd_plan_info_t)]
    lib.sd_plan_export_size.argtypes = [_P, _i32, ctypes.POINTER(ctypes.c_size_t)]
    lib.sd_plan_export.argtypes = [_P, _i32, _P, ctypes.c_size_t]
    lib.sd_plan_destroy.argtypes = [_P]
    lib.sd_plan_destroy.restype = None
    lib.sd_plan_cache_clear.argtypes = []
    lib.sd_plan_cache_clear.restype = None
    lib.sd_plan_cache_size.argtypes = [ctypes.POINTER(_i64)]
    lib.sd_plan_cache_save.argtypes = [ctypes.c_char_p]
    lib.sd_plan_cache_load.argtypes = [ctypes.c_char_p]
    lib.sd_status_string.argtypes = [ctypes.c_int]
    lib.sd_status_string.restype = ctypes.c_char_p
    lib.sd_last_error.argtypes = []
    lib.sd_last_error.restype = ctypes.c_char_p
    for f in ("sd_analyze", "sd_analyze_device", "sd_plan", "sd_plan_ex", "sd_spmm", "sd_plan_info", "sd_plan_export_size",
              "sd_plan_export", "sd_plan_device", "sd_plan_cache_size", "sd_plan_cache_save", "sd_plan_cache_load"):
        getattr(lib, f).restype = ctypes.c_int
    return lib


_lib = _load()
EXPORTED = ("sd_analyze", "sd_analyze_device", "sd_plan", "sd_plan_ex", "sd_plan_device", "sd_spmm", "sd_spmm_merge_noalloc", "sd_plan_info", "sd_plan_export_size",
            "sd_plan_export", "sd_plan_destroy", "sd_plan_cache_clear", "sd_plan_cache_size", "sd_plan_cache_save", "sd_plan_cache_load", "sd_status_string", "sd_last_error")


def _check(status: int, where: str):
    if status != SD_OK:
        raise SparseDittoError(status, where)


class _Csr:
    """Keeps contiguous host copies alive for the duration of a call."""

    def __init__(self, rowptr, colidx, values, m, k):
        self.rowptr = np.ascontiguousarray(rowptr, dtype=np.int32)
        self.colidx = np.ascontiguousarray(colidx, dtype=np.int32)
        self.values = np.ascontiguousarray(values, dtype=np.float32)
        nnz = int(self.rowptr[-1]) if self.rowptr.size else 0
        self.c = sd_csr_t(int(m), int(k), nnz, self.rowptr.ctypes.data, self.colidx.ctypes.data or None,
                          self.values.ctypes.data or None)


def _csr_args(A, rowptr, colidx, values, m, k):
    if A is not None:
        return _Csr(A.rowptr, A.colidx, A.values, A.m, A.k)
    return _Csr(rowptr, colidx, values, m, k)


def sd_analyze(A=None, *, rowptr=None, colidx=None, values=None, m=None, k=None, dense_threshold: int = 0,
               raw: bool = False):
    """Structural statistics of a host CSR matrix (any object with m, k,
    rowptr, colidx, values, or the arrays as keywords).  raw=True returns
    the sd_stats_t struct itself."""
    csr = _csr_args(A, rowptr, colidx, values, m, k)
    st = sd_stats_t()
    _check(_lib.sd_analyze(ctypes.byref(csr.c), dense_threshold, ctypes.byref(st)), "sd_analyze")
    return st if raw else _stats_dict(st)


def _stats_dict(st) -> dict:
    out = {f: int(getattr(st, f)) for f in _STATS_INT}
    out.update({f: float(getattr(st, f)) for f in _STATS_REAL})
    out["row_hist"] = np.array(st.row_hist[:], np.int64)
    out["fill16_hist"] = np.array(st.fill16_hist[:], np.int64)
    return out


def sd_analyze_device(rowptr, colidx, values, m: int, k: int, nnz: int, dense_threshold: int = 0,
                      stream=None, raw: bool = False):
    """Structural statistics of a CSR matrix already in device memory.
    rowptr, colidx, values are device pointers (ints) or tensors on the
    current device; stream is an int hipStream_t, a torch stream, or None.
    raw=True returns the sd_stats_t struct itself."""
    if stream is not None and not isinstance(stream, int):
        stream = int(stream.cuda_stream)
    c = sd_csr_t(int(m), int(k), int(nnz), _devptr(rowptr), _devptr(colidx), _devptr(values))
    st = sd_stats_t()
    _check(_lib.sd_analyze_device(ctypes.byref(c), int(dense_threshold), ctypes.byref(st), stream),
           "sd_analyze_device")
    return st if raw else _stats_dict(st)


class Plan:
    """Owns an sd_plan_t handle; destroyed with sd_plan_destroy."""

    def __init__(self, handle: int):
        self.handle = handle
        self.info = sd_plan_info(self)

    def destroy(self):
        if self.handle:
            _lib.sd_plan_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.destroy()
        except Exception:
            pass

    def __enter__(self):
        return self

    def __exit__(self, *a):
        self.destroy()

    @property
    def family(self) -> str:
        return FAMILY_NAMES[self.info["family"]]


def _plan_opts(force="auto", heavy_threshold=0, chunk_nnz=0, units=0, engine="auto", transpose=False,
               placement=PLACEMENT_CURRENT, device=0, dense_threshold=0, rows_per_group=0, gather_unroll=0,
               cache_policy=0, hot_budget_kib=0, search=False, col_tile=0, window_rows=0, wg_order=0, wg_chunk=0,
               sell_sigma=0, row_slices=0, light_order=0, chunk_order=0) -> sd_plan_opts_t:
    o = sd_plan_opts_t()
    o.force = FAMILIES[force] if isinstance(force, str) else int(force)
    o.heavy_threshold, o.chunk_nnz, o.units = int(heavy_threshold), int(chunk_nnz), int(units)
    o.engine = ENGINES[engine] if isinstance(engine, str) else int(engine)
    o.transpose = 1 if transpose else 0
    o.placement, o.device, o.dense_threshold = int(placement), int(device), int(dense_threshold)
    o.rows_per_group, o.gather_unroll = int(rows_per_group), int(gather_unroll)
    o.cache_policy = CACHE_POLICIES[cache_policy] if isinstance(cache_policy, str) else int(cache_policy)
    o.hot_budget_kib = int(hot_budget_kib)
    o.search = 1 if search else 0
    o.col_tile = int(col_tile)
    o.window_rows = int(window_rows)
    o.wg_order = WG_ORDERS[wg_order] if isinstance(wg_order, str) else int(wg_order)
    o.wg_chunk = int(wg_chunk)
    o.sell_sigma = int(sell_sigma)
    o.row_slices = int(row_slices)
    o.light_order = {"auto": 0, "ascending": 1, "last_col": 2}[light_order] if isinstance(light_order, str) \
        else int(light_order)
    o.chunk_order = {"auto": 0, "list": 1, "mid_col": 2}[chunk_order] if isinstance(chunk_order, str) \
        else int(chunk_order)
    return o


def sd_plan_ex(A=None, n: int = 1, *, rowptr=None, colidx=None, values=None, m=None, k=None, **opts) -> Plan:
    """Plan for a host CSR matrix (an object with m, k, rowptr, colidx,
    values, or the arrays themselves); keyword options are sd_plan_opts_t's."""
    csr = _csr_args(A, rowptr, colidx, values, m, k)
    o = _plan_opts(**opts)
    h = _P()
    _check(_lib.sd_plan_ex(ctypes.byref(csr.c), int(n), ctypes.byref(o), ctypes.byref(h)), "sd_plan_ex")
    return Plan(h.value)


def sd_plan_device(rowptr, colidx, values, m: int, k: int, nnz: int, n: int, stream=None, **opts) -> Plan:
    """Plan for a CSR matrix already in device memory: rowptr, colidx, values
    are device pointers (ints) or tensors on the current device; stream is an
    int hipStream_t, a torch stream, or None.  Keyword options as sd_plan_ex."""
    if stream is not None and not isinstance(stream, int):
        stream = int(stream.cuda_stream)
    c = sd_csr_t(int(m), int(k), int(nnz), _devptr(rowptr), _devptr(colidx), _devptr(values))
    o = _plan_opts(**opts)
    h = _P()
    _check(_lib.sd_plan_device(ctypes.byref(c), int(n), ctypes.byref(o), stream, ctypes.byref(h)),
           "sd_plan_device")
    return Plan(h.value)


def sd_plan(A=None, n: int = 1, **kw) -> Plan:
    """sd_plan with default options (keyword options go to sd_plan_ex)."""
    if kw and any(key not in ("rowptr", "colidx", "values", "m", "k") for key in kw):
        return sd_plan_ex(A, n, **kw)
    csr = _csr_args(A, kw.get("rowptr"), kw.get("colidx"), kw.get("values"), kw.get("m"), kw.get("k"))
    h = _P()
    _check(_lib.sd_plan(ctypes.byref(csr.c), int(n), ctypes.byref(h)), "sd_plan")
    return Plan(h.value)


def _devptr(x):
    if x is None:
        return None
    if isinstance(x, int):
        return x
    return int(x.data_ptr())


def sd_spmm(plan: Plan, B, C, stream=None) -> None:
    """C = op(A).B on `stream` (an int hipStream_t, a torch stream, or None
    for the null stream).  B and C are device pointers or tensors."""
    if stream is not None and not isinstance(stream, int):
        stream = int(stream.cuda_stream)
    _check(_lib.sd_spmm(plan.handle, _devptr(B), _devptr(C), stream), "sd_spmm")


def sd_spmm_merge_noalloc(rowptr, colidx, values, m: int, k: int, nnz: int, n: int, B, C, units: int = 0,
                          stream=None) -> None:
    """C = A.B by the merge-path kernels straight from a device CSR, with no
    plan and no allocation (the library's fixed device scratch).  Pointers
    are ints or tensors on the current device; stream as for sd_spmm."""
    if stream is not None and not isinstance(stream, int):
        stream = int(stream.cuda_stream)
    c = sd_csr_t(int(m), int(k), int(nnz), _devptr(rowptr), _devptr(colidx), _devptr(values))
    _check(_lib.sd_spmm_merge_noalloc(ctypes.byref(c), int(n), int(units), _devptr(B), _devptr(C), stream),
           "sd_spmm_merge_noalloc")


def sd_plan_info(plan: Plan) -> dict:
    info = sd_plan_info_t()
    _check(_lib.sd_plan_info(plan.handle, ctypes.byref(info)), "sd_plan_info")
    return {name: getattr(info, name) for name, _ in _INFO_FIELDS if not name.startswith("reserved")}


def sd_plan_export(plan: Plan, what: int) -> np.ndarray:
    size = ctypes.c_size_t()
    _check(_lib.sd_plan_export_size(plan.handle, int(what), ctypes.byref(size)), "sd_plan_export_size")
    dt = _EXPORT_DTYPE[int(what)]
    out = np.empty(size.value // np.dtype(dt).itemsize, dt)
    _check(_lib.sd_plan_export(plan.handle, int(what), out.ctypes.data or None, size.value), "sd_plan_export")
    return out


def sd_plan_destroy(plan: Plan) -> None:
    plan.destroy()


def sd_plan_cache_clear() -> None:
    _lib.sd_plan_cache_clear()


def sd_plan_cache_size() -> int:
    n = _i64()
    _check(_lib.sd_plan_cache_size(ctypes.byref(n)), "sd_plan_cache_size")
    return n.value


def sd_plan_cache_save(path) -> None:
    """Writes the recorded search choices to `path`."""
    _check(_lib.sd_plan_cache_save(os.fsencode(path)), "sd_plan_cache_save")


def sd_plan_cache_load(path) -> None:
    """Adds the search choices recorded in a file written by sd_plan_cache_save."""
    _check(_lib.sd_plan_cache_load(os.fsencode(path)), "sd_plan_cache_load")


def sd_status_string(status: int) -> str:
    return _lib.sd_status_string(int(status)).decode()


def sd_last_error() -> str:
    return _lib.sd_last_error().decode()
