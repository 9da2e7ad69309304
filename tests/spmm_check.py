"""Helpers for the GPU parity tests: run a plan through the C ABI on torch
device buffers and compare with the oracle."""
from __future__ import annotations

import numpy as np

TOL = 1e-5  # |C_gpu - C64| <= TOL * (1 + S) per element, S = |A|.|B|


def device_buffers(B: np.ndarray, rows_out: int, misalign: bool = False):
    """Copy B to the device and allocate C.  With misalign=True both start 4
    bytes past a 16-byte boundary, which forces the 32-bit access path."""
    import torch

    k, n = B.shape
    off = 1 if misalign else 0
    Bs = torch.empty(k * n + off, dtype=torch.float32, device="cuda")
    Bd = Bs[off:off + k * n].view(k, n) if k * n else Bs[off:off].view(k, n)
    Bd.copy_(torch.from_numpy(np.ascontiguousarray(B)))
    Cs = torch.full((rows_out * n + off,), float("nan"), dtype=torch.float32, device="cuda")
    Cd = Cs[off:off + rows_out * n].view(rows_out, n)
    return Bd, Cd


def run(sd, plan, B: np.ndarray, rows_out: int, misalign: bool = False, repeat: int = 1):
    import torch

    Bd, Cd = device_buffers(B, rows_out, misalign)
    outs = []
    for _ in range(repeat):
        Cd.fill_(float("nan"))
        sd.sd_spmm(plan, Bd, Cd, torch.cuda.current_stream())
        torch.cuda.synchronize()
        outs.append(Cd.cpu().numpy().copy())
    return outs if repeat > 1 else outs[0]


def max_err(C: np.ndarray, C64: np.ndarray, S: np.ndarray) -> float:
    if C.size == 0:
        return 0.0
    return float(np.max(np.abs(C.astype(np.float64) - C64) / (1.0 + S)))


def assert_close(C: np.ndarray, C64: np.ndarray, S: np.ndarray, what: str = ""):
    assert C.shape == C64.shape, (what, C.shape, C64.shape)
    finite = np.isfinite(C)
    assert finite.all(), f"{what}: {int((~finite).sum())} non-finite outputs"
    err = np.abs(C.astype(np.float64) - C64)
    bad = err > TOL * (1.0 + S)
    if bad.any():
        i, j = np.argwhere(bad)[0]
        raise AssertionError(f"{what}: {int(bad.sum())} elements out of tolerance; first ({i},{j}) "
                             f"gpu={C[i, j]!r} ref={C64[i, j]!r} S={S[i, j]!r}")


def expected_csr_arrays(A, info: dict):
    """The CSR arrays a plan holds for operand A (already transposed for a
    transpose plan): A itself, or for a heavy-split plan the oracle's split
    layout (light rows in the plan's order, then heavy rows), whose row
    pointers run over the light rows by list position."""
    import oracle

    if info["family"] != 2:  # SD_FMT_CSR_SPLIT
        return A.rowptr, A.colidx, A.values
    T, c = info["heavy_threshold"], info["chunk_nnz"]
    light, _ = oracle.heavy_split(A.rowptr, A.m, T, c)
    if info["light_order"] == 2:
        light = oracle.light_by_last_col(A, light)
    lptr, col, val, _ = oracle.split_layout(A, T, c, light)
    return lptr, col, val


def expected_split_chunks(A, info: dict):
    """For a heavy-split plan on operand A: the oracle's chunk triples (in the
    split layout's coordinates) and the chunk processing order the plan's
    chunk_order names."""
    import oracle

    T, c = info["heavy_threshold"], info["chunk_nnz"]
    light, _ = oracle.heavy_split(A.rowptr, A.m, T, c)
    if info["light_order"] == 2:
        light = oracle.light_by_last_col(A, light)
    _, col, _, chunks = oracle.split_layout(A, T, c, light)
    order = oracle.chunks_by_mid_col(col, chunks) if info["chunk_order"] == 2 else \
        np.arange(len(chunks), dtype=np.int32)
    return chunks, order


def assert_close_all_rows(src, B: np.ndarray, Cd, what: str = "", chunk_elems: int = 1 << 25):
    """Every row of the device result Cd (a torch tensor, src.m x n) against
    the oracle, in row chunks of about chunk_elems outputs so host memory
    stays bounded at full size."""
    import oracle

    n = B.shape[1]
    rows_per = max(1, chunk_elems // max(1, n))
    bufs = (np.empty(rows_per * n), np.empty(rows_per * n))
    for r0 in range(0, src.m, rows_per):
        r1 = min(src.m, r0 + rows_per)
        C64, S = oracle.spmm_rows(src, B, np.arange(r0, r1, dtype=np.int32), out=bufs)
        assert_close(Cd[r0:r1].cpu().numpy(), C64, S, f"{what} rows [{r0}, {r1})")
