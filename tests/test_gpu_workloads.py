"""Full-size parity: the five synthetic workloads at their real sizes, each
product planned exactly as bench.py plans it (default options) and checked
against the oracle on every row (in row chunks), plus the other families on
the workloads they are measured on, and the device copies of the plan's
conversions and partitions against the oracle bit for bit."""
import numpy as np
import pytest

import gen
import oracle
from spmm_check import assert_close, assert_close_all_rows, expected_csr_arrays, expected_split_chunks

pytestmark = [pytest.mark.gpu, pytest.mark.slow]

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():  # pragma: no cover - CPU container
    pytest.skip("needs a GPU", allow_module_level=True)

import paper_2608_05033_amd as sd  # noqa: E402

_cache = {}


def workload(name):
    if name not in _cache:
        _cache.clear()  # keep one large workload in host memory at a time
        A = gen.WORKLOADS[name].matrix(seed=0)
        At = None
        if any(p.transpose for p in gen.WORKLOADS[name].products):
            tr, tc, tv = oracle.transpose(A)
            At = gen.CSR(A.k, A.m, tr, tc, tv)
        _cache[name] = (A, At)
    return _cache[name]


def run_product(A, At, prod, **opts):
    src = At if prod.transpose else A
    B = prod.dense(src.k, seed=0)
    print(f"case m={src.m} nnz={src.nnz} n={prod.n} transpose={prod.transpose} opts={opts}", flush=True)
    plan = sd.sd_plan_ex(A, prod.n, transpose=prod.transpose, **opts)
    Bd = torch.from_numpy(B).cuda()
    Cd = torch.full((src.m, prod.n), float("nan"), device="cuda")
    sd.sd_spmm(plan, Bd, Cd, torch.cuda.current_stream())
    torch.cuda.synchronize()
    return plan, src, B, Cd


def check(src, B, Cd, what=""):
    """Every row against the oracle, then the properties that hold at any
    size: finite everywhere, and empty rows give exactly 0."""
    assert_close_all_rows(src, B, Cd, what)
    empty = np.nonzero(np.diff(src.rowptr) == 0)[0]
    if empty.size:
        assert bool((Cd[torch.from_numpy(empty).long().cuda()] == 0).all())


@pytest.mark.parametrize("name", ["laplace", "rmat20", "block16"])
@pytest.mark.parametrize("n", [1, 8, 16, 32])
def test_workload_narrow_widths(name, n):
    """Planner defaults at narrow widths on the full-size workloads: sliced
    rows and whole-wave heavy chunks (power-law), sliced CSR rows or ELL
    (Laplacian), MFMA with one or two n-tiles (blocks)."""
    import dataclasses

    A, At = workload(name)
    prod = dataclasses.replace(gen.WORKLOADS[name].products[0], n=n)
    plan, src, B, Cd = run_product(A, At, prod)
    check(src, B, Cd, what=f"{name}/{plan.family}/n={n}")
    plan.destroy()


@pytest.mark.parametrize("name", list(gen.WORKLOADS))
def test_workload_default_plan(name):
    """The bench's launch configuration (planner defaults) on every product."""
    A, At = workload(name)
    for prod in gen.WORKLOADS[name].products:
        plan, src, B, Cd = run_product(A, At, prod)
        check(src, B, Cd, what=f"{name}/{plan.family}/{prod.n}")
        plan.destroy()


@pytest.mark.parametrize("name,opts", [
    ("laplace", {"force": "csr_row"}),
    ("laplace", {"force": "csr_split"}),
    ("laplace", {"force": "csr_merge"}),
    ("rmat20", {"force": "csr_row"}),
    ("rmat20", {"force": "csr_split", "heavy_threshold": 64, "chunk_nnz": 64}),
    ("rmat20", {"force": "win"}),
    ("gcn", {"force": "win"}),
    ("block16", {"force": "bsr", "engine": "mfma"}),
    ("block16", {"force": "bell", "engine": "mfma"}),
    ("block16", {"force": "bsr", "engine": "valu"}),
    ("block16", {"force": "csr_row"}),
])
def test_workload_other_families(name, opts):
    A, At = workload(name)
    prod = gen.WORKLOADS[name].products[0]
    plan, src, B, Cd = run_product(A, At, prod, **opts)
    check(src, B, Cd, what=f"{name}/{opts}")
    plan.destroy()


def test_full_size_conversions_bitexact():
    """Device copies of the full-size conversions and partitions equal the
    oracle's, bit for bit."""
    A, _ = workload("rmat20")
    with sd.sd_plan_ex(A, 128, force="csr_merge") as p:
        assert np.array_equal(sd.sd_plan_export(p, sd.SD_EXPORT_MERGE_COORDS).reshape(-1, 2),
                              oracle.merge_split(A.rowptr, A.m, p.info["units"]))
    with sd.sd_plan_ex(A, 128, force="csr_split") as p:
        T, c = p.info["heavy_threshold"], p.info["chunk_nnz"]
        light, _ = oracle.heavy_split(A.rowptr, A.m, T, c)
        light = oracle.light_by_last_col(A, light)
        lptr, col, val, chunks = oracle.split_layout(A, T, c, light)
        assert np.array_equal(sd.sd_plan_export(p, sd.SD_EXPORT_LIGHT_ROWS), light)
        assert np.array_equal(sd.sd_plan_export(p, sd.SD_EXPORT_CHUNKS).reshape(-1, 3), chunks)
        assert np.array_equal(sd.sd_plan_export(p, sd.SD_EXPORT_ROWPTR), lptr)
        assert np.array_equal(sd.sd_plan_export(p, sd.SD_EXPORT_COLIDX), col)
        assert np.array_equal(sd.sd_plan_export(p, sd.SD_EXPORT_VALUES).view(np.uint32), val.view(np.uint32))
        assert np.array_equal(sd.sd_plan_export(p, sd.SD_EXPORT_CHUNK_ORDER), oracle.chunks_by_mid_col(col, chunks))
    L, _ = workload("laplace")
    with sd.sd_plan_ex(L, 64, force="ell") as p:
        w, ec, ev = oracle.to_ell(L)
        assert np.array_equal(sd.sd_plan_export(p, sd.SD_EXPORT_ELL_COL), ec.ravel())
        assert np.array_equal(sd.sd_plan_export(p, sd.SD_EXPORT_ELL_VAL).view(np.uint32), ev.ravel().view(np.uint32))
    Bm, _ = workload("block16")
    with sd.sd_plan_ex(Bm, 64, force="bsr") as p:
        bp, bc, bv = oracle.to_bsr(Bm, 16)
        assert np.array_equal(sd.sd_plan_export(p, sd.SD_EXPORT_BLOCK_PTR), bp)
        assert np.array_equal(sd.sd_plan_export(p, sd.SD_EXPORT_BLOCK_COL), bc)
        assert np.array_equal(sd.sd_plan_export(p, sd.SD_EXPORT_BLOCK_VAL).view(np.uint32),
                              bv.ravel().view(np.uint32))


def test_gcn_transpose_conversion_bitexact():
    A, At = workload("gcn")
    with sd.sd_plan_ex(A, 64, transpose=True) as p:
        if p.family.startswith("csr"):
            er, ec, ev = expected_csr_arrays(At, p.info)
            assert np.array_equal(sd.sd_plan_export(p, sd.SD_EXPORT_ROWPTR), er)
            assert np.array_equal(sd.sd_plan_export(p, sd.SD_EXPORT_COLIDX), ec)
            assert np.array_equal(sd.sd_plan_export(p, sd.SD_EXPORT_VALUES).view(np.uint32), ev.view(np.uint32))
        if p.family == "csr_split":
            chunks, order = expected_split_chunks(At, p.info)
            assert np.array_equal(sd.sd_plan_export(p, sd.SD_EXPORT_CHUNKS).reshape(-1, 3), chunks)
            assert np.array_equal(sd.sd_plan_export(p, sd.SD_EXPORT_CHUNK_ORDER), order)


@pytest.mark.parametrize("name", list(gen.WORKLOADS))
def test_workload_device_plan(name):
    """sd_plan_device on the device copy of each full-size workload gives the
    host plan's info and exported arrays, and the same C bit for bit."""
    A, At = workload(name)
    dev = [torch.from_numpy(np.ascontiguousarray(x)).cuda() for x in (A.rowptr, A.colidx, A.values)]
    for prod in gen.WORKLOADS[name].products:
        src = At if prod.transpose else A
        print(f"case device plan {name} n={prod.n} transpose={prod.transpose}", flush=True)
        with sd.sd_plan_ex(A, prod.n, transpose=prod.transpose) as hp, \
                sd.sd_plan_device(*dev, A.m, A.k, A.nnz, prod.n, stream=torch.cuda.current_stream(),
                                  transpose=prod.transpose) as dp:
            assert dp.info["device_built"] == 1
            hi = {k: v for k, v in hp.info.items() if k != "device_built"}
            di = {k: v for k, v in dp.info.items() if k != "device_built"}
            assert hi == di, {k: (hi[k], di[k]) for k in hi if hi[k] != di[k]}
            for what in range(1, 21):
                try:
                    he = sd.sd_plan_export(hp, what)
                except sd.SparseDittoError:
                    continue
                assert he.tobytes() == sd.sd_plan_export(dp, what).tobytes(), (name, prod.n, what)
            B = torch.from_numpy(prod.dense(src.k, seed=1)).cuda()
            Ch = torch.full((src.m, prod.n), float("nan"), device="cuda")
            Cd = torch.full((src.m, prod.n), float("nan"), device="cuda")
            sd.sd_spmm(hp, B, Ch, torch.cuda.current_stream())
            sd.sd_spmm(dp, B, Cd, torch.cuda.current_stream())
            torch.cuda.synchronize()
            assert torch.equal(Ch.view(torch.int32), Cd.view(torch.int32))


@pytest.fixture(scope="module")
def big_case():
    """20 M x 20 M with 2 nonzeros per row and N = 128: C holds 2.56e9 elements,
    so rows past 2^31 / 128 are reached only through 64-bit offsets.  B (10 GB)
    is freed when the module's tests end."""
    m = 20_000_000
    A = gen.random_rows(m, m, np.full(m, 2, np.int32), seed=12)
    g = torch.Generator(device="cuda").manual_seed(5)
    B = torch.randn((m, 128), generator=g, device="cuda", dtype=torch.float32)
    yield A, B
    del B
    torch.cuda.empty_cache()


@pytest.mark.parametrize("fam", ["csr_row", "csr_split", "csr_merge", "ell", "sell"])
def test_index_range_beyond_int32(fam, big_case):
    A, B = big_case
    n = B.shape[1]
    print(f"case int64 offsets {fam} m={A.m} n={n}", flush=True)
    C = torch.full((A.m, n), float("nan"), device="cuda")
    with sd.sd_plan_ex(A, n, force=fam, heavy_threshold=2, chunk_nnz=2) as plan:  # split: every row heavy
        sd.sd_spmm(plan, B, C, torch.cuda.current_stream())
        torch.cuda.synchronize()
    rng = np.random.default_rng(3)
    rows = np.unique(np.concatenate([rng.choice(A.m, 1500, replace=False),
                                     np.arange(A.m - 500, A.m)])).astype(np.int64)
    # the sampled rows as a small CSR over the columns they use
    starts, ends = A.rowptr[rows].astype(np.int64), A.rowptr[rows + 1].astype(np.int64)
    idx = np.concatenate([np.arange(s, e) for s, e in zip(starts, ends)])
    cols = A.colidx[idx]
    used = np.unique(cols)
    sub = gen.CSR(len(rows), len(used), np.concatenate([[0], np.cumsum(ends - starts)]).astype(np.int32),
                  np.searchsorted(used, cols).astype(np.int32), A.values[idx])
    Bsub = B[torch.from_numpy(used).long().cuda()].cpu().numpy()
    C64, S = oracle.spmm(sub, Bsub)
    got = C[torch.from_numpy(rows).cuda()].cpu().numpy()
    assert_close(got, C64, S, f"int64 offsets {fam}")
    assert bool(torch.isfinite(C).all())
    del C
    torch.cuda.empty_cache()


@pytest.mark.parametrize("fam,engine", [("bsr", "mfma"), ("bsr", "valu"), ("bell", "mfma")])
def test_block_index_range_beyond_int32(fam, engine, big_case):
    """The block kernels on a 20 M-row diagonal (one 16 x 16 block per
    block-row), N = 128: C = diag(a) B, rows past 2^31 / 128 included."""
    _, B = big_case
    m, n = B.shape
    rng = np.random.default_rng(8)
    a = rng.uniform(-1.0, 1.0, m).astype(np.float32)
    D = gen.CSR(m, m, np.arange(m + 1, dtype=np.int32), np.arange(m, dtype=np.int32), a)
    print(f"case int64 offsets {fam}/{engine} m={m} n={n}", flush=True)
    C = torch.full((m, n), float("nan"), device="cuda")
    rp, ci, vv = (torch.from_numpy(x).cuda() for x in (D.rowptr, D.colidx, D.values))
    with sd.sd_plan_device(rp, ci, vv, m, m, m, n, force=fam, engine=engine) as plan:
        del rp, ci, vv
        sd.sd_spmm(plan, B, C, torch.cuda.current_stream())
        torch.cuda.synchronize()
    rows = np.unique(np.concatenate([rng.choice(m, 1500, replace=False), np.arange(m - 500, m)]))
    r = torch.from_numpy(rows).long().cuda()
    got = C[r].cpu().numpy().astype(np.float64)
    want = a[rows].astype(np.float64)[:, None] * B[r].cpu().numpy().astype(np.float64)
    assert np.max(np.abs(got - want) / (1.0 + np.abs(want))) <= 1e-5
    assert bool(torch.isfinite(C).all())
    del C
    torch.cuda.empty_cache()
