"""Pins of the CPU oracle against what the paper and mathematics fix.

Each test checks the oracle against something other than itself: exact
integer arithmetic, brute force on dense copies, closed forms (identity,
permutation, Laplacian, GCN normalisation), hand-worked fixtures and the
numbers printed in the paper (tests/golden/)."""
import collections
import json
import os

import numpy as np
import pytest

import gen
import oracle
from builders import from_rows, law_like, nemeth_like, shen_like

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def dense_of(A, dtype=np.float64):
    D = np.zeros((A.m, A.k), dtype)
    P = np.zeros((A.m, A.k), bool)
    for i in range(A.m):
        cols = A.colidx[A.rowptr[i]:A.rowptr[i + 1]]
        D[i, cols] = A.values[A.rowptr[i]:A.rowptr[i + 1]]
        P[i, cols] = True
    return D, P


def int_valued(A, seed):
    rng = np.random.default_rng(seed)
    A.values = rng.integers(-8, 9, A.nnz).astype(np.float32)
    return A


def ragged_lengths(m, k, seed):
    rng = np.random.default_rng(seed)
    r = rng.integers(0, min(k, 40), m)
    r[rng.random(m) < 0.2] = 0  # empty rows
    if m > 3:
        r[m // 3] = k  # one full row
    return r


SHAPES = [(1, 1, 1), (5, 7, 3), (33, 17, 4), (64, 129, 5), (100, 50, 1), (37, 300, 8), (0, 5, 3)]


# ------------------------------------------------------------------ SpMM ---

@pytest.mark.parametrize("m,k,n", SHAPES)
def test_spmm_integer_exact(m, k, n):
    """Integer-valued A and B: every partial sum is exact in fp64, so the
    oracle must equal the int64 matrix product exactly, and S = |A|.|B|."""
    A = int_valued(gen.random_rows(m, k, ragged_lengths(m, k, 1), seed=3), 4)
    Bi = np.random.default_rng(5).integers(-8, 9, (k, n))
    C, S = oracle.spmm(A, Bi.astype(np.float32))
    D, _ = dense_of(A, np.int64) if m else (np.zeros((0, k), np.int64), None)
    np.testing.assert_array_equal(C, (D @ Bi).astype(np.float64))
    np.testing.assert_array_equal(S, (np.abs(D) @ np.abs(Bi)).astype(np.float64))


@pytest.mark.parametrize("m,k,n", [(9, 13, 3), (31, 20, 5), (16, 64, 2)])
def test_spmm_dense_bruteforce_bitexact(m, k, n):
    """Dense triple loop in ascending k over the densified matrix: the zero
    entries add exact zeros, so the result is bit-identical to the CSR sum."""
    A = gen.random_rows(m, k, ragged_lengths(m, k, 2), seed=7)
    B = gen.dense_uniform(k, n, seed=9)
    C, S = oracle.spmm(A, B)
    D, _ = dense_of(A)
    for i in range(m):
        for j in range(n):
            acc = 0.0
            sacc = 0.0
            for kk in range(k):
                acc += D[i, kk] * float(B[kk, j])
                sacc += abs(D[i, kk]) * abs(float(B[kk, j]))
            assert C[i, j] == acc
            assert S[i, j] == sacc


def test_spmm_close_to_library_matmul():
    """Against numpy's fp64 GEMM (a different summation order): agreement
    within a few fp64 ulps of S."""
    A = gen.random_rows(200, 300, ragged_lengths(200, 300, 3), seed=11)
    B = gen.dense_normal(300, 16, seed=12)
    C, S = oracle.spmm(A, B)
    D, _ = dense_of(A)
    ref = D @ B.astype(np.float64)
    assert np.all(np.abs(C - ref) <= 1e-14 * (1 + S))


def test_spmm_identity_and_permutation():
    n = 24
    m = 50
    B = gen.dense_normal(m, n, seed=1)
    I = from_rows(m, m, [[i] for i in range(m)])
    C, _ = oracle.spmm(I, B)
    assert np.array_equal(C.astype(np.float32), B)
    perm = np.random.default_rng(0).permutation(m)
    P = from_rows(m, m, [[int(perm[i])] for i in range(m)])
    C, _ = oracle.spmm(P, B)
    assert np.array_equal(C.astype(np.float32), B[perm])


def test_spmm_laplacian_closed_forms():
    """7-point Laplacian: with B = 1, C_i = 6 - (#in-grid neighbours), exactly;
    with B = x coordinate, every interior row gives 0 exactly."""
    nx = 6
    A = gen.laplacian3d(nx)
    x, y, z = np.meshgrid(np.arange(nx), np.arange(nx), np.arange(nx), indexing="ij")
    # natural order idx = x + nx*(y + nx*z)
    xs = np.zeros(nx ** 3)
    nb = np.zeros(nx ** 3)
    for zz in range(nx):
        for yy in range(nx):
            for xx in range(nx):
                i = xx + nx * (yy + nx * zz)
                xs[i] = xx
                nb[i] = sum([xx > 0, xx < nx - 1, yy > 0, yy < nx - 1, zz > 0, zz < nx - 1])
    C, _ = oracle.spmm(A, np.ones((nx ** 3, 1), np.float32))
    np.testing.assert_array_equal(C[:, 0], 6 - nb)
    C, _ = oracle.spmm(A, xs.astype(np.float32)[:, None])
    interior = nb == 6
    assert np.all(C[interior, 0] == 0.0)


def test_spmm_gcn_sqrt_degree_identity():
    """GCN normalisation val = 1/sqrt(d_i d_j): with B_j = sqrt(d_j) the row
    sum is sum_j 1/sqrt(d_i) = sqrt(d_i)."""
    A = gen.rmat(10, 8000, seed=2)
    d = A.row_lengths().astype(np.float64)
    B = np.sqrt(d).astype(np.float32)[:, None]
    C, _ = oracle.spmm(A, B)
    np.testing.assert_allclose(C[:, 0], np.sqrt(d), rtol=2e-6)


def test_spmm_rows_and_transposed():
    A = gen.random_rows(70, 45, ragged_lengths(70, 45, 4), seed=5)
    B = gen.dense_uniform(45, 6, seed=1)
    C, S = oracle.spmm(A, B)
    rows = np.array([0, 69, 3, 3, 10], np.int32)
    Cr, Sr = oracle.spmm_rows(A, B, rows)
    assert np.array_equal(Cr, C[rows]) and np.array_equal(Sr, S[rows])
    # A^T B by scatter == CSR walk of the transposed copy, bit for bit
    Bt = gen.dense_uniform(70, 6, seed=2)
    Ct, St = oracle.spmm_transposed(A, Bt)
    tr, tc, tv = oracle.transpose(A)
    At = gen.CSR(A.k, A.m, tr, tc, tv)
    C2, S2 = oracle.spmm(At, Bt)
    assert np.array_equal(Ct, C2) and np.array_equal(St, S2)
    Ai = int_valued(gen.random_rows(30, 20, ragged_lengths(30, 20, 6), seed=8), 3)
    Bi = np.random.default_rng(1).integers(-8, 9, (30, 4))
    Ct, _ = oracle.spmm_transposed(Ai, Bi.astype(np.float32))
    D, _ = dense_of(Ai, np.int64)
    np.testing.assert_array_equal(Ct, (D.T @ Bi).astype(np.float64))


# ------------------------------------------------------- Representations ---

@pytest.mark.parametrize("m,k,b", [(33, 47, 4), (40, 40, 8), (50, 70, 16), (16, 16, 16), (1, 3, 16)])
def test_bsr_bell_conversion_bruteforce(m, k, b):
    """BSR and Blocked-ELL against a dense cut into b x b tiles."""
    A = gen.random_rows(m, k, ragged_lengths(m, k, 5), seed=13)
    D, P = dense_of(A, np.float32)
    mb, kb = -(-m // b), -(-k // b)
    Dp = np.zeros((mb * b, kb * b), np.float32)
    Pp = np.zeros((mb * b, kb * b), bool)
    Dp[:m, :k] = D
    Pp[:m, :k] = P
    tiles = Dp.reshape(mb, b, kb, b).transpose(0, 2, 1, 3)
    occ = Pp.reshape(mb, b, kb, b).any(axis=(1, 3))
    bptr, bcol, bval = oracle.to_bsr(A, b)
    assert np.array_equal(bptr, np.concatenate([[0], np.cumsum(occ.sum(1))]))
    exp_cols = np.concatenate([np.nonzero(occ[r])[0] for r in range(mb)]) if mb else np.zeros(0)
    assert np.array_equal(bcol, exp_cols)
    exp_vals = np.concatenate([tiles[r, np.nonzero(occ[r])[0]] for r in range(mb)])
    assert np.array_equal(bval.view(np.uint32), exp_vals.view(np.uint32))
    width, ecol, evals = oracle.to_bell(A, b)
    assert width == occ.sum(1).max()
    for r in range(mb):
        c = np.nonzero(occ[r])[0]
        assert np.array_equal(ecol[r, :c.size], c) and np.all(ecol[r, c.size:] == -1)
        assert np.array_equal(evals[r, :c.size].view(np.uint32), tiles[r, c].view(np.uint32))
        assert np.all(evals[r, c.size:].view(np.uint32) == 0)


@pytest.mark.parametrize("b", [4, 8, 16])
def test_csr_and_block_encodings_agree_bitwise(b):
    """The same A through CSR, BSR and Blocked-ELL gives bit-identical fp64
    C and S: the zero fill only adds exact zeros."""
    m, k = 77, 90
    A = gen.random_rows(m, k, ragged_lengths(m, k, 6), seed=17)
    B = gen.dense_normal(k, 7, seed=3)
    C, S = oracle.spmm(A, B)
    bptr, bcol, bval = oracle.to_bsr(A, b)
    Cb, Sb = oracle.spmm_bsr(m, k, b, bptr, bcol, bval, B)
    assert np.array_equal(C, Cb) and np.array_equal(S, Sb)
    width, ecol, evals = oracle.to_bell(A, b)
    Ce, Se = oracle.spmm_bell(m, k, b, width, ecol, evals, B)
    assert np.array_equal(C, Ce) and np.array_equal(S, Se)


@pytest.mark.parametrize("m,k", [(40, 30), (1, 5), (64, 64)])
def test_ell_conversion_bruteforce_and_agreement(m, k):
    """ELL against the dense rows (entries in column order, then padding), and
    ELL SpMM bit-identical to CSR SpMM (same terms, same order)."""
    A = gen.random_rows(m, k, ragged_lengths(m, k, 11), seed=31)
    width, ecol, evals = oracle.to_ell(A)
    D, P = dense_of(A, np.float32)
    assert width == P.sum(1).max()
    for i in range(m):
        cols = np.nonzero(P[i])[0]
        assert np.array_equal(ecol[i, :cols.size], cols) and np.all(ecol[i, cols.size:] == -1)
        assert np.array_equal(evals[i, :cols.size].view(np.uint32), D[i, cols].view(np.uint32))
        assert np.all(evals[i, cols.size:].view(np.uint32) == 0)
    B = gen.dense_normal(k, 5, seed=4)
    C, S = oracle.spmm(A, B)
    Ce, Se = oracle.spmm_ell(m, width, ecol, evals, B)
    assert np.array_equal(C, Ce) and np.array_equal(S, Se)


@pytest.mark.parametrize("m,k,C,sigma", [(40, 30, 4, 1), (70, 200, 4, 16), (70, 200, 8, 70), (5, 9, 16, 3),
                                          (64, 64, 1, 1), (33, 12, 2, 1000)])
def test_sell_bruteforce_and_agreement(m, k, C, sigma):
    """SELL-C-sigma against a brute force of its definition (stable sort by
    non-increasing length inside windows of sigma rows, slices of C padded to
    their longest row, row-major) and SpMM bit-identical to CSR."""
    A = gen.random_rows(m, k, ragged_lengths(m, k, 12), seed=43)
    perm, sp, col, val = oracle.to_sell(A, C, sigma)
    lens = np.diff(A.rowptr)
    want = []
    for b in range(0, m, sigma):
        want += sorted(range(b, min(m, b + sigma)), key=lambda r: (-lens[r], r))
    assert perm.tolist() == want
    total = 0
    for sl in range((m + C - 1) // C):
        rows = want[sl * C:(sl + 1) * C]
        w = max(lens[r] for r in rows)
        assert sp[sl] == total
        for j, r in enumerate(rows):
            base = total + j * w
            rc = A.colidx[A.rowptr[r]:A.rowptr[r + 1]]
            assert col[base:base + len(rc)].tolist() == rc.tolist()
            assert np.all(col[base + len(rc):base + w] == -1) and np.all(val[base + len(rc):base + w].view(np.uint32) == 0)
            assert np.array_equal(val[base:base + len(rc)].view(np.uint32), A.values[A.rowptr[r]:A.rowptr[r + 1]].view(np.uint32))
        total += len(rows) * w
    assert sp[-1] == total == col.size
    if sigma == 1:
        assert np.array_equal(perm, np.arange(m))
    if C == 1 and sigma == 1:  # no padding, no reordering: exactly the CSR arrays
        assert np.array_equal(col, A.colidx) and np.array_equal(val.view(np.uint32), A.values.view(np.uint32))
    B = gen.dense_normal(k, 5, seed=3)
    C64, S = oracle.spmm(A, B)
    Cs, Ss = oracle.spmm_sell(m, C, perm, sp, col, val, B)
    assert np.array_equal(C64, Cs) and np.array_equal(S, Ss)


def test_sell_padding_hand_count():
    """Row lengths 1, 5, 2, 7, 3, 3 with C = 2: unsorted slices (sigma = 1)
    hold 2*5 + 2*7 + 2*3 = 30 slots; one global sort (sigma = 6) gives slices
    (7, 5), (3, 3), (2, 1): 14 + 6 + 4 = 24 slots."""
    lengths = [1, 5, 2, 7, 3, 3]
    A = from_rows(6, 10, [list(range(r)) for r in lengths])
    assert oracle.to_sell(A, 2, 1)[1][-1] == 30
    perm, sp, _, _ = oracle.to_sell(A, 2, 6)
    assert perm.tolist() == [3, 1, 4, 5, 2, 0] and sp.tolist() == [0, 14, 20, 24]


def _split_for_windows(A, T, c):
    light, _ = oracle.heavy_split(A.rowptr, A.m, T, c)
    light = oracle.light_by_last_col(A, light)
    lptr, col, val, chunks = oracle.split_layout(A, T, c, light)
    return light, lptr, col, val, chunks


@pytest.mark.parametrize("m,k,R,cap,T", [(40, 30, 8, 1000, 25), (70, 200, 16, 3, 30), (5, 9, 64, 64, 1000),
                                         (64, 64, 64, 10, 20), (33, 12, 1, 64, 8), (120, 50, 7, 0, 35)])
def test_split_windows_bruteforce_and_agreement(m, k, R, cap, T):
    """Windows over the split layout against a brute force (per window of R
    light-list positions: the columns two or more of its rows use, the `cap`
    most used kept with ties to the smaller column, ascending; per light entry
    -2 - position or its column; heavy entries keep their columns), and the
    windowed SpMM bit-identical to the CSR oracle in fp64."""
    A = gen.random_rows(m, k, ragged_lengths(m, k, 12), seed=41)
    light, lptr, col, val, chunks = _split_for_windows(A, T, 4)
    wp, wc, code = oracle.split_windows(lptr, col, len(light), R, cap)
    assert wp[0] == 0 and np.all(np.diff(wp) >= 0)
    for w in range((len(light) + R - 1) // R):
        t0, t1 = w * R, min(len(light), (w + 1) * R)
        uses = collections.Counter(col[lptr[t0]:lptr[t1]].tolist())
        cand = sorted((c for c, u in uses.items() if u >= 2), key=lambda c: (-uses[c], c))[:cap]
        staged = sorted(cand)
        assert wc[wp[w]:wp[w + 1]].tolist() == staged
        for p in range(lptr[t0], lptr[t1]):
            assert code[p] == (-2 - staged.index(col[p]) if col[p] in staged else col[p])
    assert np.array_equal(code[lptr[-1]:], col[lptr[-1]:])  # heavy entries
    if R == 1 or cap == 0:  # nothing can be staged
        assert wp[-1] == 0 and np.array_equal(code, col)
    B = gen.dense_normal(k, 6, seed=2)
    C, S = oracle.spmm(A, B)
    Cw, Sw = oracle.spmm_split_windows(m, light, lptr, chunks, code, val, R, wp, wc, B)
    assert np.array_equal(C, Cw) and np.array_equal(S, Sw)


@pytest.mark.parametrize("R", [4, 16, 50])
def test_split_windows_tridiagonal_closed_form(R):
    """Tridiagonal rows, all light (the by-last-column list is then ascending):
    column j is used by rows j-1, j, j+1, so a window of rows [r0, r1) stages
    exactly its own columns r0 .. r1-1 (columns r0-1 and r1 have one user
    inside).  Interior columns have three users and the two end columns two,
    so a cap of R-2 keeps exactly r0+1 .. r1-2."""
    m = 300
    rows = [[j for j in (i - 1, i, i + 1) if 0 <= j < m] for i in range(m)]
    A = from_rows(m, m, rows)
    light, lptr, col, _, _ = _split_for_windows(A, m + 1, 4)
    assert light.tolist() == list(range(m))
    wp, wc, code = oracle.split_windows(lptr, col, m, R, R)
    for w in range((m + R - 1) // R):
        r0, r1 = w * R, min(m, (w + 1) * R)
        assert wc[wp[w]:wp[w + 1]].tolist() == (list(range(r0, r1)) if r1 - r0 >= 2 else [])
    nw = (m + R - 1) // R
    assert int((code >= 0).sum()) == 2 * (nw - 1) + (1 if m % R == 1 else 0)
    wp, wc, _ = oracle.split_windows(lptr, col, m, R, R - 2)
    for w in range(m // R):  # whole interior windows
        r0, r1 = w * R, (w + 1) * R
        if 0 < r0 and r1 < m:
            assert wc[wp[w]:wp[w + 1]].tolist() == list(range(r0 + 1, r1 - 1))


def test_transpose_bruteforce_and_involution():
    A = gen.random_rows(41, 29, ragged_lengths(41, 29, 7), seed=19)
    tr, tc, tv = oracle.transpose(A)
    At = gen.CSR(A.k, A.m, tr, tc, tv)
    D, P = dense_of(A, np.float32)
    Dt, Pt = dense_of(At, np.float32)
    assert np.array_equal(Pt, P.T) and np.array_equal(Dt.view(np.uint32), D.T.view(np.uint32))
    r2, c2, v2 = oracle.transpose(At)
    assert np.array_equal(r2, A.rowptr) and np.array_equal(c2, A.colidx)
    assert np.array_equal(v2.view(np.uint32), A.values.view(np.uint32))


# -------------------------------------------------------------- Schedules ---

def _read_fixture(name):
    rows = []
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            line = line.strip()
            if line and not line.startswith("#"):
                rows.append(line.split())
    return rows


def test_heavy_split_hand_worked():
    rowptr = np.array([0, 3, 3, 12, 16, 28, 29], np.int32)
    light, chunks = oracle.heavy_split(rowptr, 6, 4, 5)
    fx = _read_fixture("heavy_split_small.txt")
    exp_light = [int(x) for x in fx[0][1:]]
    exp_chunks = [[int(x) for x in r[1:]] for r in fx[1:]]
    assert light.tolist() == exp_light
    assert chunks.tolist() == exp_chunks


@pytest.mark.parametrize("T,c", [(1, 1), (4, 3), (16, 16), (64, 256), (1000, 7)])
def test_heavy_split_invariants(T, c):
    A = gen.random_rows(300, 400, ragged_lengths(300, 400, 8) * 3, seed=23)
    r = A.row_lengths()
    light, chunks = oracle.heavy_split(A.rowptr, A.m, T, c)
    assert light.tolist() == [i for i in range(A.m) if r[i] < T]
    heavy = [i for i in range(A.m) if r[i] >= T]
    pos = 0
    for i in heavy:
        begin = A.rowptr[i]
        while begin < A.rowptr[i + 1]:
            row, b0, b1 = chunks[pos]
            assert row == i and b0 == begin and b1 == min(begin + c, A.rowptr[i + 1]) and b1 > b0
            begin = b1
            pos += 1
    assert pos == len(chunks)


def test_light_by_last_col_hand_worked():
    """Rows 0..5 with last columns 7, -, 2, 9, 2, 5 (row 1 empty): by last
    column, ties by row, the empty row last -> 2, 4, 5, 0, 3, 1."""
    rows = [[1, 7], [], [0, 2], [3, 9], [2], [0, 1, 5]]
    rowptr = np.cumsum([0] + [len(r) for r in rows]).astype(np.int32)
    colidx = np.array([c for r in rows for c in r], np.int32)
    A = gen.CSR(6, 10, rowptr, colidx, np.ones(colidx.size, np.float32))
    assert oracle.light_by_last_col(A, np.arange(6)).tolist() == [2, 4, 5, 0, 3, 1]
    assert oracle.light_by_last_col(A, np.array([0, 3, 5])).tolist() == [5, 0, 3]
    assert oracle.light_by_last_col(A, np.array([], np.int32)).tolist() == []


def test_light_by_last_col_invariants():
    """A permutation of its input whose keys never decrease and whose ties
    keep ascending rows; a tridiagonal matrix (last column non-decreasing in
    the row) keeps its order."""
    A = gen.random_rows(500, 300, ragged_lengths(500, 300, 4), seed=31)
    light, _ = oracle.heavy_split(A.rowptr, A.m, 40, 16)
    out = oracle.light_by_last_col(A, light)
    assert sorted(out.tolist()) == sorted(light.tolist())
    keys = [A.colidx[A.rowptr[r + 1] - 1] if A.rowptr[r + 1] > A.rowptr[r] else A.k for r in out]
    for a, b, ra, rb in zip(keys, keys[1:], out, out[1:]):
        assert a < b or (a == b and ra < rb)
    m = 50
    rows = [[j for j in (i - 1, i, i + 1) if 0 <= j < m] for i in range(m)]
    rp = np.cumsum([0] + [len(r) for r in rows]).astype(np.int32)
    ci = np.array([c for r in rows for c in r], np.int32)
    tri = gen.CSR(m, m, rp, ci, np.ones(ci.size, np.float32))
    assert oracle.light_by_last_col(tri, np.arange(m)).tolist() == list(range(m))


def test_split_layout_hand_worked():
    """Rows 0..3 of lengths 2, 5, 1, 0 with T = 3, c = 2; light list (2, 0, 3):
    entries of row 2, then row 0, then (empty) row 3, then heavy row 1 cut into
    [3, 5), [5, 7), [7, 8)."""
    rows = [[4, 6], [0, 1, 2, 3, 5], [7], []]
    rowptr = np.cumsum([0] + [len(r) for r in rows]).astype(np.int32)
    colidx = np.array([c for r in rows for c in r], np.int32)
    vals = np.arange(1, colidx.size + 1, dtype=np.float32)
    A = gen.CSR(4, 8, rowptr, colidx, vals)
    lptr, col, val, chunks = oracle.split_layout(A, 3, 2, np.array([2, 0, 3], np.int32))
    assert lptr.tolist() == [0, 1, 3, 3]
    assert col.tolist() == [7, 4, 6, 0, 1, 2, 3, 5]
    assert val.tolist() == [8, 1, 2, 3, 4, 5, 6, 7]
    assert chunks.tolist() == [[1, 3, 5], [1, 5, 7], [1, 7, 8]]


def test_split_layout_invariants():
    """Every light row's entries and every heavy row's entries reappear, in
    order, where lptr and the chunks say; the chunks tile the heavy rows."""
    A = gen.random_rows(400, 500, ragged_lengths(400, 500, 9) * 3, seed=37)
    T, c = 30, 11
    light, _ = oracle.heavy_split(A.rowptr, A.m, T, c)
    order = oracle.light_by_last_col(A, light)
    lptr, col, val, chunks = oracle.split_layout(A, T, c, order)
    for i, r in enumerate(order):
        a, b = A.rowptr[r], A.rowptr[r + 1]
        assert np.array_equal(col[lptr[i]:lptr[i + 1]], A.colidx[a:b])
        assert np.array_equal(val[lptr[i]:lptr[i + 1]], A.values[a:b])
    pos = lptr[-1]
    k = 0
    for r in range(A.m):
        a, b = A.rowptr[r], A.rowptr[r + 1]
        if b - a < T:
            continue
        assert np.array_equal(col[pos:pos + b - a], A.colidx[a:b])
        q = pos
        while q < pos + b - a:
            assert chunks[k].tolist() == [r, q, min(q + c, pos + b - a)]
            q = chunks[k][2]
            k += 1
        pos += b - a
    assert pos == A.nnz and k == len(chunks)


def test_chunks_by_mid_col_hand_worked():
    """The hand-worked split layout above (T = 3, c = 2, light list 2, 0, 3):
    chunks [3, 5), [5, 7), [7, 8) of row 1 have middle entries 4, 6, 7, whose
    columns are 1, 3, 5 -> order 0, 1, 2.  Reversed middle columns give the
    reverse order, and equal ones keep the chunk order."""
    rows = [[4, 6], [0, 1, 2, 3, 5], [7], []]
    rowptr = np.cumsum([0] + [len(r) for r in rows]).astype(np.int32)
    colidx = np.array([c for r in rows for c in r], np.int32)
    A = gen.CSR(4, 8, rowptr, colidx, np.ones(colidx.size, np.float32))
    _, col, _, chunks = oracle.split_layout(A, 3, 2, np.array([2, 0, 3], np.int32))
    assert oracle.chunks_by_mid_col(col, chunks).tolist() == [0, 1, 2]
    col2 = np.array([7, 4, 6, 0, 9, 2, 5, 1], np.int32)  # middles 4 -> 9, 6 -> 5, 7 -> 1
    assert oracle.chunks_by_mid_col(col2, chunks).tolist() == [2, 1, 0]
    col3 = np.array([7, 4, 6, 0, 3, 2, 3, 3], np.int32)  # all middles 3
    assert oracle.chunks_by_mid_col(col3, chunks).tolist() == [0, 1, 2]
    assert oracle.chunks_by_mid_col(col, np.zeros((0, 3), np.int32)).tolist() == []


def test_chunks_by_mid_col_invariants():
    """A permutation of the chunk indices whose middle columns never
    decrease and whose ties keep ascending indices."""
    A = gen.random_rows(300, 2000, ragged_lengths(300, 2000, 5) * 9, seed=41)
    T, c = 60, 23
    light, _ = oracle.heavy_split(A.rowptr, A.m, T, c)
    _, col, _, chunks = oracle.split_layout(A, T, c, light)
    order = oracle.chunks_by_mid_col(col, chunks)
    assert len(chunks) > 50
    assert sorted(order.tolist()) == list(range(len(chunks)))
    keys = [col[(chunks[q][1] + chunks[q][2]) // 2] for q in order]
    for a, b, qa, qb in zip(keys, keys[1:], order, order[1:]):
        assert a < b or (a == b and qa < qb)


def test_merge_split_hand_worked():
    rowptr = np.array([0, 2, 2, 5, 6], np.int32)
    coords = oracle.merge_split(rowptr, 4, 3)
    fx = _read_fixture("merge_path_small.txt")
    assert coords.tolist() == [[int(r[1]), int(r[2])] for r in fx]


def _merge_bruteforce(rowptr, m, U):
    """Materialise the merged list of tokens, then read the coordinates."""
    nnz = int(rowptr[m])
    tokens = []  # ('e', row) or ('n', j)
    i, j = 0, 0
    ends = list(rowptr[1:])
    while i < m or j < nnz:
        if i < m and (j >= nnz or ends[i] <= j):
            tokens.append("e")
            i += 1
        else:
            tokens.append("n")
            j += 1
    total = m + nnz
    L = max(1, -(-total // U))
    out = []
    for u in range(U + 1):
        d = min(u * L, total)
        out.append([tokens[:d].count("e"), tokens[:d].count("n")])
    return out


@pytest.mark.parametrize("U", [1, 2, 3, 7, 50])
def test_merge_split_bruteforce(U):
    A = gen.random_rows(25, 30, ragged_lengths(25, 30, 9), seed=29)
    coords = oracle.merge_split(A.rowptr, A.m, U)
    assert coords.tolist() == _merge_bruteforce(A.rowptr, A.m, U)
    # invariants: monotone, first (0,0), last (m,nnz), each nonzero inside its row
    assert np.all(np.diff(coords, axis=0) >= 0)
    assert coords[0].tolist() == [0, 0] and coords[-1].tolist() == [A.m, A.nnz]
    for i, j in coords:
        if i < A.m:
            assert A.rowptr[i] <= j <= A.rowptr[i + 1]


def test_merge_split_empty_matrix():
    rowptr = np.zeros(6, np.int32)
    coords = oracle.merge_split(rowptr, 5, 4)
    assert coords.tolist() == _merge_bruteforce(rowptr, 5, 4)


# ------------------------------------------------------------- Statistics ---

def _padded_slots(lengths, height):
    """Stored slots of rows cut into slices of `height` consecutive rows, each
    slice padded to its longest row: the size of the padded arrays, counted
    by building them (ELL is one slice of all rows, SELL-C slices of C)."""
    total = 0
    for s in range(0, len(lengths), height):
        part = lengths[s:s + height]
        total += np.zeros((part.size, int(part.max()) if part.size else 0), np.int8).size
    return total


def _stats_bruteforce(A, dense_thr=128):
    """Every statistic except the shape class, from a dense boolean copy of the
    pattern: counts by scanning it, representation sizes by materialising the
    padded layouts of Eq. format-expansion and counting their slots, ratios as
    means over the objects they average (rows, columns, tiles, diagonal
    positions).  Independent of the oracle's row scans and formulas."""
    D, P = dense_of(A, np.float32)
    r = P.sum(1)
    m, k = A.m, A.k
    nnz = int(P.sum())
    out = {"m": m, "k": k, "nnz": nnz}
    s = np.sort(r)
    out.update(row_min=int(s[0]), row_max=int(s[-1]), row_q25=int(s[(m - 1) // 4]), row_q50=int(s[(m - 1) // 2]),
               row_q75=int(s[3 * (m - 1) // 4]), empty_rows=int((r == 0).sum()))
    deg = P.sum(0)
    out["col_deg_max"] = int(deg.max())
    spans, gaps = [], []
    for i in range(m):
        cols = np.nonzero(P[i])[0]
        if cols.size:
            spans.append(cols[-1] - cols[0] + 1)
        gaps.extend(np.diff(cols).tolist())
    spans = np.sort(np.asarray(spans, np.int64))
    out["row_span_median"] = int(spans[(len(spans) - 1) // 2]) if len(spans) else 0
    diag = np.diagonal(P[:min(m, k), :min(m, k)])
    out["diag_nnz"] = int(diag.sum())
    for b in (4, 8, 16):
        mb, kb = -(-m // b), -(-k // b)
        Pp = np.zeros((mb * b, kb * b), bool)
        Pp[:m, :k] = P
        cnt = Pp.reshape(mb, b, kb, b).sum(axis=(1, 3))
        occupied = cnt > 0
        out[f"nnzb{b}"] = int(occupied.sum())
        # BSR(b) stores every slot of every occupied block
        out[f"rho_bsr{b}"] = np.kron(occupied, np.ones((b, b), bool)).sum() / nnz if nnz else 0.0
        if b == 16:
            occ = cnt[occupied]
            dense = occupied & (cnt >= dense_thr)
            out["dense_tiles16"] = int(dense.sum())
            out["dense_tile_nnz16"] = int(occ[occ >= dense_thr].sum())
            width = int(occupied.sum(1).max())
            out["bell16_width"] = width
            out["fill16_hist"] = np.bincount((occ - 1) // 32, minlength=8)
            out["tile16_coverage"] = float(occupied.mean())
            out["dense_tile_frac"] = float((occ >= dense_thr).mean()) if occ.size else 0.0
            in_dense = np.kron(dense, np.ones((16, 16), bool))[:m, :k] & P
            out["dense_tile_nnz_frac"] = in_dense.sum() / nnz if nnz else 0.0
            out["nnz_per_tile16"] = float(occ.mean()) if occ.size else 0.0
            # Blocked-ELL(16): every block-row padded to the widest, 16 x 16 values per slot
            out["rho_bell16"] = np.zeros((mb, width, 16, 16), np.int8).size / nnz if nnz else 0.0
    for c in (16, 32, 512):
        out[f"sell{c}_slots"] = _padded_slots(r, c)
        out[f"rho_sell{c}"] = out[f"sell{c}_slots"] / nnz if nnz else 0.0
    out["rho_ell"] = _padded_slots(r, max(m, 1)) / nnz if nnz else 0.0
    hist = np.zeros(33, np.int64)
    for x in r:
        hist[int(x).bit_length()] += 1
    out["row_hist"] = hist
    out["density"] = float(P.mean())
    out["row_mean"] = float(r.mean())
    out["empty_row_frac"] = float((r == 0).mean())
    out["row_cv"] = float(r.std() / r.mean()) if nnz else 0.0
    out["col_deg_mean"] = float(deg.mean())
    out["col_deg_cv"] = float(deg.std() / deg.mean()) if nnz else 0.0
    out["col_gap_mean"] = float(np.mean(gaps)) if gaps else 0.0
    out["row_span_mean"] = float(np.mean(spans)) if len(spans) else 0.0
    out["row_span_norm"] = float(np.mean(spans / k)) if len(spans) else 0.0
    out["diag_frac"] = float(diag.mean()) if diag.size else 0.0
    return out


def _assert_stats_match(st, bf, what=""):
    for key, v in bf.items():
        if isinstance(v, np.ndarray):
            assert np.array_equal(st[key], v), (what, key)
        elif isinstance(v, float):
            assert st[key] == pytest.approx(v, rel=1e-12, abs=1e-15), (what, key, st[key], v)
        else:
            assert st[key] == v, (what, key, st[key], v)


def test_stats_bruteforce_covers_every_field():
    """The brute force pins every statistic but the shape class, which the
    hand-built row-length cases below pin."""
    A = gen.random_rows(20, 30, ragged_lengths(20, 30, 5), seed=5)
    bf = _stats_bruteforce(A)
    want = set(oracle.INT_FIELDS) | set(oracle.REAL_FIELDS) | {"row_hist", "fill16_hist"}
    assert set(bf) == want - {"shape_class"}


@pytest.mark.parametrize("seed,m,k", [(1, 64, 64), (2, 37, 91), (3, 100, 33), (4, 200, 260), (6, 1, 1),
                                      (7, 129, 17), (8, 17, 600)])
def test_stats_bruteforce(seed, m, k):
    A = gen.random_rows(m, k, ragged_lengths(m, k, seed), seed=seed)
    _assert_stats_match(oracle.stats(A), _stats_bruteforce(A), (seed, m, k))


@pytest.mark.parametrize("thr", [1, 64, 128, 200, 256])
@pytest.mark.parametrize("nbr,nbc", [(12, 12), (9, 21), (20, 7)])
def test_stats_bruteforce_blocky(nbr, nbc, thr):
    """Block-structured patterns (tiles from nearly empty to full) at several
    dense-tile thresholds, with m != k so that block-row and block-column
    counts cannot be swapped unnoticed; the last block-row and block-column
    are ragged."""
    Ab = gen.block(nbr, nbc, 16, min(4, nbc), 4, 0.8, seed=nbr + nbc)
    # drop the last 12 rows and 10 columns: ragged tiles (at most 4 x 16 and
    # 16 x 6 entries) along both edges
    m, k = Ab.m - 12, Ab.k - 10
    rows = [[c for c in Ab.colidx[Ab.rowptr[i]:Ab.rowptr[i + 1]] if c < k] for i in range(m)]
    A = from_rows(m, k, rows)
    st = oracle.stats(A, dense_threshold=thr)
    bf = _stats_bruteforce(A, dense_thr=thr)
    # the threshold splits the tiles: some dense unless it asks for full tiles
    assert 0 < bf["nnzb16"] and (thr == 256 or bf["dense_tiles16"] > 0)
    assert thr < 128 or bf["dense_tiles16"] < bf["nnzb16"]
    _assert_stats_match(st, bf, (nbr, nbc, thr))


def test_stats_hand_built_cases():
    # one dense 16x16 block inside a 64x64 matrix
    rows = [list(range(16, 32)) if 16 <= i < 32 else [] for i in range(64)]
    st = oracle.stats(from_rows(64, 64, rows))
    assert st["nnzb16"] == 1 and st["tile16_coverage"] == 1 / 16 and st["dense_tiles16"] == 1
    assert st["dense_tile_nnz_frac"] == 1.0 and st["fill16_hist"].tolist() == [0] * 7 + [1]
    assert st["nnzb4"] == 16 and st["rho_bsr16"] == 1.0 and st["empty_rows"] == 48
    assert st["diag_nnz"] == 16 and st["row_span_median"] == 16 and st["col_gap_mean"] == 1.0
    # by hand: 16 block-rows of 4 x 4 (all full), 4 of 8 x 8 (all full), one tile of 16 x 16
    assert st["rho_bsr4"] == 1.0 and st["rho_bsr8"] == 1.0 and st["rho_bell16"] == 4.0
    assert st["dense_tile_frac"] == 1.0 and st["nnz_per_tile16"] == 256.0
    assert st["rho_sell16"] == 1.0 and st["rho_sell32"] == 2.0 and st["rho_sell512"] == 4.0
    assert st["row_span_norm"] == 0.25 and st["col_deg_mean"] == 4.0
    # diagonal
    st = oracle.stats(from_rows(50, 50, [[i] for i in range(50)]))
    assert st["diag_frac"] == 1.0 and st["row_span_mean"] == 1.0 and st["row_cv"] == 0.0
    assert st["rho_ell"] == 1.0 and st["shape_class"] == 0
    # 50 diagonal entries: 13 occupied 4x4 blocks of which 12 hold 4 and the last 2
    assert st["rho_bsr4"] == 16 * 13 / 50 and st["rho_bsr8"] == 64 * 7 / 50 and st["rho_bsr16"] == 256 * 4 / 50
    # every block-row holds one tile; 4 block-rows, each padded to width 1
    assert st["rho_bell16"] == 256 * 4 / 50 and st["dense_tile_frac"] == 0.0
    # all-empty matrix: every ratio defined as 0
    st = oracle.stats(from_rows(8, 8, [[] for _ in range(8)]))
    assert st["nnz"] == 0 and st["rho_ell"] == 0.0 and st["empty_row_frac"] == 1.0 and st["nnzb16"] == 0
    assert st["shape_class"] == 0 and st["rho_sell16"] == 0.0 and st["rho_bell16"] == 0.0
    # a wide matrix (m != k): ceil(m/16) block-rows enter rho_BELL16, ceil(k/16) does not
    st = oracle.stats(from_rows(20, 100, [[0, 99] for _ in range(20)]))
    assert st["bell16_width"] == 2 and st["rho_bell16"] == 256 * 2 * 2 / 40
    assert st["tile16_coverage"] == 4 / (2 * 7) and st["col_deg_mean"] == 40 / 100


def _lengths_matrix(lengths):
    """Rows of the given lengths, columns 0 .. r-1 (k = longest row)."""
    lengths = list(lengths)
    k = max(max(lengths), 1)
    return from_rows(len(lengths), k, [list(range(r)) for r in lengths])


# Row-length vectors whose shape class and CV follow by hand from the reading:
# uniform if CV < 0.1; else bimodal if the log2 row-length histogram has two
# local maxima >= 2 bins apart, each holding >= 10 % of the rows; else
# moderate if CV < 0.5; else power-law if CV >= 1 and max >= 50 mean; else
# skewed.  Each threshold has a case on each side.
SHAPE_CASES = [
    # (name, lengths, class, CV worked by hand or None)
    ("constant rows", [8] * 40, "uniform", 0.0),
    ("19/21: CV 1/20 < 0.1", [19, 21] * 20, "uniform", 0.05),
    ("9/11: CV = 0.1 exactly", [9, 11] * 20, "moderate", 0.1),
    ("3/7: CV 0.4 < 0.5, bins 2 and 3 adjacent", [3, 7] * 20, "moderate", 0.4),
    ("2/4: peaks one bin apart", [2, 4] * 50, "moderate", 1 / 3),
    ("1/3: CV = 0.5 exactly", [1, 3] * 20, "skewed", 0.5),
    ("2/8: peaks two bins apart", [2, 8] * 50, "bimodal", 0.6),
    ("1/100 half and half", [1] * 50 + [100] * 50, "bimodal", 49.5 / 50.5),
    ("second peak at 10 % exactly", [1] * 90 + [100] * 10, "bimodal", None),
    ("second peak at 9 %", [1] * 91 + [100] * 9, "skewed", None),
    ("second peak at 5 %: CV >= 1, max < 50 mean", [1] * 95 + [100] * 5, "skewed", None),
    ("one long row: max = 50 mean exactly", [1] * 99 + [99], "power-law", None),
    ("one long row: max just under 50 mean", [1] * 99 + [98], "skewed", None),
    ("max >= 50 mean but CV 0.70 < 1", [1] * 4999 + [51], "skewed", None),
    ("one row of 1000 among 999 of 1", [1] * 999 + [1000], "power-law", None),
]


@pytest.mark.parametrize("name,lengths,cls,cv", SHAPE_CASES, ids=[c[0] for c in SHAPE_CASES])
def test_stats_shape_class_hand_built(name, lengths, cls, cv):
    st = oracle.stats(_lengths_matrix(lengths))
    assert oracle.SHAPE_CLASSES[st["shape_class"]] == cls, (name, st["row_cv"], st["row_max"], st["row_mean"])
    if cv is not None:
        assert st["row_cv"] == pytest.approx(cv, rel=1e-12)


def test_stats_shape_class_worked_numbers():
    """The numbers that put the boundary cases where they are, by hand."""
    st = oracle.stats(_lengths_matrix([1] * 99 + [99]))
    assert st["row_mean"] == 1.98 and st["row_max"] == 99  # 99 >= 50 * 1.98
    st = oracle.stats(_lengths_matrix([1] * 4999 + [51]))
    assert st["row_mean"] == 1.01 and st["row_cv"] == pytest.approx(np.sqrt(1.52 - 1.01 ** 2) / 1.01, rel=1e-12)
    st = oracle.stats(_lengths_matrix([1] * 90 + [100] * 10))
    assert st["row_hist"][1] == 90 and st["row_hist"][7] == 10


def _golden():
    with open(os.path.join(GOLDEN, "worked_examples.json")) as f:
        return json.load(f)


def _approx(entry):
    return pytest.approx(entry["approx"], abs=entry["tol"])


def test_stats_paper_worked_example_shen():
    """Shen/e40r0100 counts (m, nnz, max row, nnzb_16) reproduce the printed
    rho_ELL, rho_BSR(16), nonzeros per tile and tile coverage."""
    g = _golden()["shen_e40r0100"]
    A = shen_like()
    st = oracle.stats(A)
    assert (st["m"], st["nnz"], st["row_max"], st["nnzb16"]) == (g["m"], g["nnz"], g["row_max"], g["nnzb16"])
    for key in ("rho_ell", "rho_bsr16", "nnz_per_tile16", "tile16_coverage", "row_mean", "density"):
        assert st[key] == _approx(g[key]), key


@pytest.mark.parametrize("name,builder", [("nemeth26", nemeth_like), ("law_in_2004", law_like)])
def test_stats_paper_table_rows(name, builder):
    g = _golden()[name]
    A = builder()
    st = oracle.stats(A)
    assert (st["m"], st["k"], st["nnz"]) == (g["m"], g["k"], g["nnz"])
    assert st["row_mean"] == _approx(g["row_mean"])
    assert st["density"] == _approx(g["density"])
