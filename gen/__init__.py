"""Seeded synthetic SpMM inputs shared by the tests and the benchmark.

This module builds input matrices (CSR, int32 indices, fp32 values) and
dense operands only.  It contains none of the SpMM arithmetic, no format
conversion and no work partitioning; the CPU oracle and the GPU library both
consume what it produces.  The random numbers are SplitMix64 in counter mode
(see ``sdgen.c`` for the exact definition), so every array is a pure function
of its seed and sizes.

Workloads (the five synthetic stand-ins for the paper's matrix families; the
paper's own SuiteSparse matrices and the Reddit graph are not available):

* ``uniform``   1024 x 1024, exactly 8 distinct uniform columns per row, N=32
* ``laplace``   7-point Laplacian on a 64^3 grid (Dirichlet), N=64
* ``rmat20``    R-MAT scale 20, 16 Mi edges, GCN-normalised, N=128
* ``block16``   131072^2 built from 16x16 blocks, 32 per block-row, 90 % fill, N=64
* ``gcn``       R-MAT on 2.4 M vertices, 62 M edges, GCN-normalised; four
                products A.X (N=128), A.H (N=64), A^T.G (N=64), A^T.G (N=128)
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from dataclasses import dataclass, field

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SO = os.path.join(_HERE, "libsdgen.so")
_SRC = os.path.join(_HERE, "sdgen.c")

RMAT_ABC = (0.57, 0.19, 0.19)  # d = 0.05


def build(force: bool = True) -> str:
    """Compile the generator library with gcc (host code only)."""
    if force or not os.path.exists(_SO):
        tmp = _SO + ".tmp"
        subprocess.check_call(["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-o", tmp, _SRC, "-lm"])
        os.replace(tmp, _SO)
    return _SO


_lib = None


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_SO):
            build()
        lib = ctypes.CDLL(_SO)
        P = ctypes.c_void_p
        i32, i64, u64, dbl = ctypes.c_int32, ctypes.c_int64, ctypes.c_uint64, ctypes.c_double
        lib.sdg_key.restype = u64
        lib.sdg_key.argtypes = [u64, u64]
        lib.sdg_draw.restype = u64
        lib.sdg_draw.argtypes = [u64, u64]
        lib.sdg_dense_uniform.argtypes = [u64, u64, i64, P]
        lib.sdg_dense_normal.argtypes = [u64, u64, i64, P]
        lib.sdg_csr_nnz.restype = i64
        lib.sdg_csr_nnz.argtypes = [P]
        lib.sdg_csr_m.restype = i32
        lib.sdg_csr_m.argtypes = [P]
        lib.sdg_csr_k.restype = i32
        lib.sdg_csr_k.argtypes = [P]
        lib.sdg_csr_copy.argtypes = [P, P, P, P]
        lib.sdg_csr_free.argtypes = [P]
        for name, args in (
            ("sdg_uniform_rows", [i32, i32, i32, u64]),
            ("sdg_random_rows", [i32, i32, P, u64]),
            ("sdg_laplacian3d", [i32, i32, i32]),
            ("sdg_rmat", [i32, i64, i32, dbl, dbl, dbl, u64]),
            ("sdg_block", [i32, i32, i32, i32, i32, dbl, u64]),
        ):
            f = getattr(lib, name)
            f.restype = P
            f.argtypes = args
        _lib = lib
    return _lib


def _ptr(a: np.ndarray):
    return ctypes.c_void_p(a.ctypes.data)


@dataclass
class CSR:
    """A host CSR matrix: rowptr[m+1], colidx[nnz], values[nnz]."""

    m: int
    k: int
    rowptr: np.ndarray
    colidx: np.ndarray
    values: np.ndarray
    name: str = ""

    @property
    def nnz(self) -> int:
        return int(self.rowptr[-1]) if self.rowptr.size else 0

    def row_lengths(self) -> np.ndarray:
        return np.diff(self.rowptr.astype(np.int64))


def _take(h, name: str) -> CSR:
    lib = _load()
    try:
        m, k, nnz = lib.sdg_csr_m(h), lib.sdg_csr_k(h), lib.sdg_csr_nnz(h)
        rowptr = np.empty(m + 1, np.int32)
        colidx = np.empty(nnz, np.int32)
        values = np.empty(nnz, np.float32)
        lib.sdg_csr_copy(h, _ptr(rowptr), _ptr(colidx), _ptr(values))
    finally:
        lib.sdg_csr_free(h)
    return CSR(m, k, rowptr, colidx, values, name)


def uniform_rows(m: int, k: int, per_row: int, seed: int = 0) -> CSR:
    return _take(_load().sdg_uniform_rows(m, k, per_row, seed), f"uniform_{m}x{k}_{per_row}")


def random_rows(m: int, k: int, lengths, seed: int = 0) -> CSR:
    lengths = np.ascontiguousarray(lengths, dtype=np.int32)
    assert lengths.shape == (m,)
    return _take(_load().sdg_random_rows(m, k, _ptr(lengths), seed), f"random_{m}x{k}")


def laplacian3d(nx: int, ny: int | None = None, nz: int | None = None) -> CSR:
    ny = nx if ny is None else ny
    nz = nx if nz is None else nz
    return _take(_load().sdg_laplacian3d(nx, ny, nz), f"laplace_{nx}x{ny}x{nz}")


def rmat(scale: int, edges: int, nmax: int | None = None, seed: int = 0, abc=RMAT_ABC) -> CSR:
    nmax = (1 << scale) if nmax is None else nmax
    a, b, c = abc
    return _take(_load().sdg_rmat(scale, edges, nmax, a, b, c, seed), f"rmat_s{scale}_e{edges}_n{nmax}")


def block(nbr: int, nbc: int, b: int, per_row: int, window: int, fill: float, seed: int = 0) -> CSR:
    return _take(_load().sdg_block(nbr, nbc, b, per_row, window, fill, seed),
                 f"block_{nbr}x{nbc}_b{b}_{per_row}")


def dense_uniform(rows: int, cols: int, seed: int = 0, stream: int = 1) -> np.ndarray:
    out = np.empty((rows, cols), np.float32)
    _load().sdg_dense_uniform(seed, stream, rows * cols, _ptr(out))
    return out


def dense_normal(rows: int, cols: int, seed: int = 0, stream: int = 1) -> np.ndarray:
    out = np.empty((rows, cols), np.float32)
    _load().sdg_dense_normal(seed, stream, rows * cols, _ptr(out))
    return out


@dataclass
class Product:
    """One SpMM of a workload: C = op(A) . B with op = identity or transpose."""

    n: int
    transpose: bool
    dist: str  # "uniform" or "normal"
    stream: int

    def dense(self, rows: int, seed: int = 0) -> np.ndarray:
        f = dense_uniform if self.dist == "uniform" else dense_normal
        return f(rows, self.n, seed, self.stream)


@dataclass
class Workload:
    name: str
    description: str
    products: list = field(default_factory=list)

    def matrix(self, seed: int = 0) -> CSR:
        raise NotImplementedError


class _Uniform(Workload):
    def matrix(self, seed=0):
        return uniform_rows(1024, 1024, 8, seed)


class _Laplace(Workload):
    def matrix(self, seed=0):
        return laplacian3d(64)


class _Rmat20(Workload):
    def matrix(self, seed=0):
        return rmat(20, 16 << 20, seed=seed)


class _Block16(Workload):
    def matrix(self, seed=0):
        return block(8192, 8192, 16, 32, 512, 0.9, seed)


class _Gcn(Workload):
    def matrix(self, seed=0):
        return rmat(22, 62_000_000, nmax=2_400_000, seed=seed)


WORKLOADS = {
    "uniform": _Uniform("uniform", "uniform random CSR 1024x1024, 8 nnz/row, B U[-1,1) N=32",
                        [Product(32, False, "uniform", 1)]),
    "laplace": _Laplace("laplace", "3D 7-point Laplacian 64^3 (Dirichlet), B U[-1,1) N=64",
                        [Product(64, False, "uniform", 1)]),
    "rmat20": _Rmat20("rmat20", "R-MAT 2^20 vertices, 16Mi edges, GCN-normalised, B N(0,1) N=128",
                      [Product(128, False, "normal", 1)]),
    "block16": _Block16("block16", "131072^2 from 16x16 blocks, 32/block-row within +-512, 90% fill, B U[-1,1) N=64",
                        [Product(64, False, "uniform", 1)]),
    "gcn": _Gcn("gcn", "GCN SpMMs on R-MAT 2.4M vertices / 62M edges: A.X128, A.H64, A^T.G64, A^T.G128, N(0,1)",
                [Product(128, False, "normal", 1), Product(64, False, "normal", 2),
                 Product(64, True, "normal", 3), Product(128, True, "normal", 4)]),
}
