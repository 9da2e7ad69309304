"""Plans built from a matrix in device memory (sd_plan_device): the info
record, every exported array and the SpMM output equal those of sd_plan_ex on
the host copy of the same matrix, bit for bit, for every family and policy
converted on the device; outputs also meet the oracle's tolerance.  Searches from device memory share the choice
cache with host searches.  Malformed matrices are rejected as on the host."""
import numpy as np
import pytest

import gen
import oracle
from spmm_check import assert_close, run

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():  # pragma: no cover - CPU container
    pytest.skip("needs a GPU", allow_module_level=True)

import paper_2608_05033_amd as sd  # noqa: E402


def ragged(m, k, seed):
    rng = np.random.default_rng(seed)
    r = rng.integers(0, 60, m)
    r[rng.random(m) < 0.15] = 0
    if m > 10:
        r[m // 2] = min(k, 3000)
        r[m - 1] = min(k, 700)
    return np.minimum(r, k)


MATS = {
    "ragged": lambda: gen.random_rows(2000, 3001, ragged(2000, 3001, 1), seed=1),
    "uniform": lambda: gen.uniform_rows(1024, 1024, 8, 0),
    "rmat": lambda: gen.rmat(13, 120000, seed=3),
    "laplace": lambda: gen.laplacian3d(16, 16, 16),
    "block": lambda: gen.block(70, 75, 16, 12, 20, 0.9, 5),
    "empty_rows": lambda: gen.random_rows(50, 30, np.zeros(50, np.int32), seed=5),
    "onerow": lambda: gen.random_rows(1, 4000, np.array([4000], np.int32), seed=6),
    "odd": lambda: gen.random_rows(37, 19, np.arange(37, dtype=np.int32) % 19, seed=7),
}
_cache = {}


def matrix(name):
    if name not in _cache:
        _cache[name] = MATS[name]()
    return _cache[name]


# (options, built on the device?)
CASES = [
    ({}, None),  # the planner's own choice: device-built iff it is a device family
    ({"transpose": True}, None),
    ({"force": "csr_row"}, True),
    ({"force": "csr_row", "rows_per_group": 4, "gather_unroll": 8}, True),
    ({"force": "csr_split", "heavy_threshold": 40, "chunk_nnz": 17}, True),
    ({"force": "csr_split", "heavy_threshold": 1, "chunk_nnz": 256}, True),
    ({"force": "csr_split", "heavy_threshold": 40, "chunk_nnz": 17, "light_order": "ascending"}, True),
    ({"force": "csr_split", "heavy_threshold": 600, "chunk_nnz": 2048, "light_order": "last_col"}, True),
    ({"force": "csr_merge", "units": 97}, True),
    ({"force": "csr_merge", "units": 5000, "cache_policy": "nontemporal"}, True),
    ({"force": "csr_merge", "units": 300, "cache_policy": "tiered"}, True),
    ({"force": "csr_merge", "units": 300, "cache_policy": "tiered", "hot_budget_kib": 1}, True),
    ({"force": "ell"}, True),
    ({"force": "ell", "wg_order": "round_robin"}, True),
    ({"force": "bsr", "engine": "valu"}, True),
    ({"force": "bsr"}, True),
    ({"force": "bell", "engine": "valu"}, True),
    ({"force": "sell"}, True),
    ({"force": "sell", "sell_sigma": 1}, True),
    ({"force": "sell", "sell_sigma": 50}, True),
    ({"force": "win"}, True),
    ({"force": "win", "window_rows": 16, "heavy_threshold": 40, "chunk_nnz": 17}, True),
    ({"force": "win", "window_rows": 1}, True),
    ({"force": "win", "window_rows": 512, "heavy_threshold": 100, "chunk_nnz": 33}, True),
    ({"force": "csr_split", "transpose": True, "heavy_threshold": 30, "chunk_nnz": 30}, True),
    ({"force": "ell", "transpose": True}, True),
    ({"force": "bsr", "transpose": True, "engine": "valu"}, True),
    ({"force": "sell", "transpose": True}, True),
    ({"force": "win", "transpose": True}, True),
]
DEVICE_FAMILIES = tuple(sd.FAMILIES[f] for f in ("csr_row", "csr_split", "csr_merge", "ell", "bsr", "bell", "win",
                                                  "sell"))
EXPORT_KINDS = range(1, 21)


def device_csr(A, stream=None):
    dev = [torch.from_numpy(np.ascontiguousarray(x)).cuda() for x in
           (A.rowptr.astype(np.int32), A.colidx.astype(np.int32), A.values.astype(np.float32))]
    return dev


def exports(plan):
    out = {}
    for what in EXPORT_KINDS:
        try:
            out[what] = sd.sd_plan_export(plan, what)
        except sd.SparseDittoError as e:
            assert e.status == sd.SD_ERR_INVALID_VALUE
    return out


def compare_plans(host, devp, what):
    hi, di = dict(host.info), dict(devp.info)
    built = di.pop("device_built")
    assert hi.pop("device_built") == 0
    diff = {f: (hi[f], di[f]) for f in hi if hi[f] != di[f]}
    assert not diff, f"{what}: info differs {diff}"
    he, de = exports(host), exports(devp)
    assert he.keys() == de.keys(), what
    for kind in he:
        assert he[kind].dtype == de[kind].dtype and he[kind].shape == de[kind].shape, (what, kind)
        assert he[kind].tobytes() == de[kind].tobytes(), f"{what}: export {kind} differs"
    return built


@pytest.mark.parametrize("name", list(MATS))
@pytest.mark.parametrize("ci", range(len(CASES)))
@pytest.mark.parametrize("n", [8, 64])
def test_device_plan_matches_host_plan(name, ci, n):
    opts, expect_dev = CASES[ci]
    A = matrix(name)
    print(f"case plan_device {name} m={A.m} nnz={A.nnz} n={n} opts={opts}", flush=True)
    try:
        host = sd.sd_plan_ex(A, n, **opts)
    except sd.SparseDittoError as e:  # infeasible for this matrix: the device path must say the same
        rp, cidx, vv = device_csr(A)
        with pytest.raises(sd.SparseDittoError) as e2:
            sd.sd_plan_device(rp, cidx, vv, A.m, A.k, A.nnz, n, stream=torch.cuda.current_stream(), **opts)
        assert e2.value.status == e.status
        return
    rp, cidx, vv = device_csr(A)
    with host, sd.sd_plan_device(rp, cidx, vv, A.m, A.k, A.nnz, n, stream=torch.cuda.current_stream(),
                                 **opts) as devp:
        del rp, cidx, vv  # the plan keeps no reference to the caller's arrays
        built = compare_plans(host, devp, f"{name} {opts}")
        if expect_dev is None:
            expect_dev = devp.info["family"] in DEVICE_FAMILIES
        assert built == (1 if expect_dev else 0), (name, opts, devp.info["family"])
        rows = A.k if opts.get("transpose") else A.m
        cols = A.m if opts.get("transpose") else A.k
        B = gen.dense_normal(cols, n, seed=n + 3)
        Ch = run(sd, host, B, rows)
        Cd = run(sd, devp, B, rows)
        assert Ch.tobytes() == Cd.tobytes(), f"{name} {opts}: outputs differ"
        if opts.get("transpose"):
            C64, S = oracle.spmm_transposed(A, B)
        else:
            C64, S = oracle.spmm(A, B)
        assert_close(Cd, C64, S, f"device plan {name} {opts} n={n}")


def test_device_plan_orders_after_caller_stream():
    """The matrix is written on a side stream; the plan reads it on that stream."""
    A = matrix("ragged")
    side = torch.cuda.Stream()
    with torch.cuda.stream(side):
        rp = torch.empty(A.m + 1, dtype=torch.int32, device="cuda")
        ci = torch.empty(A.nnz, dtype=torch.int32, device="cuda")
        vv = torch.empty(A.nnz, dtype=torch.float32, device="cuda")
        for d, h in ((rp, A.rowptr), (ci, A.colidx), (vv, A.values)):
            d.copy_(torch.from_numpy(np.ascontiguousarray(h)).pin_memory(), non_blocking=True)
        plan = sd.sd_plan_device(rp, ci, vv, A.m, A.k, A.nnz, 32, stream=side, force="csr_split",
                                 heavy_threshold=40, chunk_nnz=17)
    with plan, sd.sd_plan_ex(A, 32, force="csr_split", heavy_threshold=40, chunk_nnz=17) as host:
        compare_plans(host, plan, "side stream")


@pytest.mark.parametrize("name", ["uniform", "ragged", "block"])
@pytest.mark.parametrize("transpose", [False, True])
def test_device_plan_search(name, transpose):
    """A search from device memory: candidates built on the device, a correct
    plan, and one choice cache with the host search (same key)."""
    A = matrix(name)
    n = 64
    rp, ci, vv = device_csr(A)
    sd.sd_plan_cache_clear()
    try:
        with sd.sd_plan_device(rp, ci, vv, A.m, A.k, A.nnz, n, search=True, transpose=transpose) as p:
            assert p.info["device_built"] == 1 and p.info["search_candidates"] >= 2
            assert p.info["search_cache_hit"] == 0
            rows, cols = (A.k, A.m) if transpose else (A.m, A.k)
            B = gen.dense_normal(cols, n, seed=1)
            C64, S = oracle.spmm_transposed(A, B) if transpose else oracle.spmm(A, B)
            assert_close(run(sd, p, B, rows), C64, S, f"device search {name} T={transpose}")
            family = p.info["family"]
        assert sd.sd_plan_cache_size() == 1
        # the host search finds the device search's choice, and the other way round
        with sd.sd_plan_ex(A, n, search=True, transpose=transpose) as h:
            assert h.info["search_cache_hit"] == 1 and h.info["family"] == family
        with sd.sd_plan_device(rp, ci, vv, A.m, A.k, A.nnz, n, search=True, transpose=transpose) as p2:
            assert p2.info["search_cache_hit"] == 1 and p2.info["device_built"] == 1
            assert p2.info["family"] == family
    finally:
        sd.sd_plan_cache_clear()


@pytest.mark.parametrize("m,k", [(0, 0), (0, 7), (5, 0), (6, 9)])
@pytest.mark.parametrize("fam", ["csr_row", "csr_split", "csr_merge", "ell", "bsr", "bell", "win", "sell"])
@pytest.mark.parametrize("transpose", [False, True])
def test_device_plan_empty(m, k, fam, transpose):
    rp = torch.zeros(m + 1, dtype=torch.int32, device="cuda")
    hrp = np.zeros(m + 1, np.int32)
    empty_i, empty_f = np.zeros(0, np.int32), np.zeros(0, np.float32)
    opts = dict(force=fam, engine="valu", transpose=transpose) if fam in ("bsr", "bell") else \
        dict(force=fam, transpose=transpose)
    with sd.sd_plan_ex(rowptr=hrp, colidx=empty_i, values=empty_f, m=m, k=k, n=8, **opts) as host, \
            sd.sd_plan_device(rp, 0, 0, m, k, 0, 8, **opts) as devp:
        assert compare_plans(host, devp, f"empty {m}x{k} {opts}") == 1
        rows, cols = (k, m) if transpose else (m, k)
        if rows:
            C = run(sd, devp, np.zeros((cols, 8), np.float32), rows)
            assert (C == 0).all()


@pytest.mark.parametrize("bad", ["unsorted", "duplicate", "col_range", "neg_col", "rowptr_dec", "rowptr_end",
                                 "rowptr_start"])
@pytest.mark.parametrize("fam", ["auto", "bsr"])
def test_device_plan_rejects_malformed(bad, fam):
    A = gen.random_rows(40, 30, np.full(40, 6, np.int32), seed=9)
    rowptr, colidx = A.rowptr.copy(), A.colidx.copy()
    if bad == "unsorted":
        colidx[[60, 61]] = colidx[[61, 60]]
    elif bad == "duplicate":
        colidx[61] = colidx[60]
    elif bad == "col_range":
        colidx[100] = 30
    elif bad == "neg_col":
        colidx[7] = -3
    elif bad == "rowptr_dec":
        rowptr[20] = rowptr[19] - 1
    elif bad == "rowptr_end":
        rowptr[-1] = A.nnz - 1
    elif bad == "rowptr_start":
        rowptr[0] = 1
    rp = torch.from_numpy(rowptr).cuda()
    ci = torch.from_numpy(colidx).cuda()
    vv = torch.from_numpy(A.values).cuda()
    print(f"case plan_device malformed {bad} {fam}", flush=True)
    with pytest.raises(sd.SparseDittoError) as e:
        sd.sd_plan_device(rp, ci, vv, A.m, A.k, A.nnz, 8, force=fam)
    assert e.value.status == sd.SD_ERR_INVALID_CSR
