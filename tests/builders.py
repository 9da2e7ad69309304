"""Deterministic matrices with prescribed structural counts, for the pins
that use numbers printed in the paper.  Input construction only."""
from __future__ import annotations

import numpy as np

from gen import CSR


def from_rows(m: int, k: int, rows: list, value: float = 1.0) -> CSR:
    lengths = np.array([len(r) for r in rows], np.int64)
    rowptr = np.zeros(m + 1, np.int64)
    np.cumsum(lengths, out=rowptr[1:])
    colidx = np.concatenate([np.sort(np.asarray(r, np.int64)) for r in rows]) if m else np.zeros(0, np.int64)
    vals = np.full(colidx.size, value, np.float32)
    return CSR(m, k, rowptr.astype(np.int32), colidx.astype(np.int32), vals)


def banded(m: int, k: int, lengths: np.ndarray, value: float = 1.0) -> CSR:
    """Row i holds lengths[i] consecutive columns centred on i (clamped)."""
    lengths = np.asarray(lengths, np.int64)
    start = np.clip(np.arange(m) - lengths // 2, 0, None)
    start = np.minimum(start, k - lengths)
    rowptr = np.zeros(m + 1, np.int64)
    np.cumsum(lengths, out=rowptr[1:])
    nnz = int(rowptr[-1])
    row_of = np.repeat(np.arange(m), lengths)
    colidx = start[row_of] + (np.arange(nnz) - rowptr[row_of])
    return CSR(m, k, rowptr.astype(np.int32), colidx.astype(np.int32), np.full(nnz, value, np.float32))


def shen_like() -> CSR:
    """m = k = 17,281, nnz = 553,562, max row 62, 20,130 occupied 16x16 tiles:
    the counts printed for Shen/e40r0100.  Block-row br < 1080 uses t = 19
    (br < 688) or 18 block-columns (br + 56 s) mod 1080; the last, one-row
    block-row uses 2.  Row lengths: 62 for row 0, 33 for rows 1..540, else 32;
    nonzero q of a row goes to block s = q mod t at in-block column q div t."""
    m = 17281
    rows = []
    for i in range(m):
        br = i // 16
        t = 2 if br == 1080 else (19 if br < 688 else 18)
        r = 62 if i == 0 else (33 if i <= 540 else 32)
        bcs = [(br + 56 * s) % 1080 for s in range(t)]
        rows.append([bcs[q % t] * 16 + q // t for q in range(r)])
    return from_rows(m, m, rows)


def nemeth_like() -> CSR:
    """m = k = 9,506 and nnz = 1,511,760 (the counts printed for nemeth26):
    rows 0..305 hold 160 nonzeros, the others 159, in a band."""
    m = 9506
    lengths = np.full(m, 159)
    lengths[:306] = 160
    return banded(m, m, lengths)


def law_like() -> CSR:
    """m = k = 1,382,908 and nnz = 16,917,053 (LAW_in-2004's size row)."""
    m = 1382908
    nnz = 16917053
    base = nnz // m
    lengths = np.full(m, base)
    lengths[: nnz - base * m] += 1
    return banded(m, m, lengths)
