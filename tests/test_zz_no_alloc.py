"""sd_spmm_merge_noalloc (no plan, no allocation, the library's fixed device
scratch) against sd_spmm on a CSR_MERGE plan with the same pieces: the same
kernels in the same order give the same bits, and both meet the oracle's
tolerance.  Two calls in a row on the shared scratch, the second with a
smaller input, then the rejections that need no kernel."""
import numpy as np
import pytest

import gen
import oracle
from spmm_check import assert_close

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():  # pragma: no cover - CPU container
    pytest.skip("needs a GPU", allow_module_level=True)

import paper_2608_05033_amd as sd  # noqa: E402


def ragged(m, k, seed):
    rng = np.random.default_rng(seed)
    r = rng.integers(0, 50, m)
    r[rng.random(m) < 0.2] = 0
    r[m // 2] = min(k, 2500)  # a row that spans many pieces
    return np.minimum(r, k)


def device_csr(A):
    return [torch.from_numpy(np.ascontiguousarray(x)).cuda() for x in (A.rowptr, A.colidx, A.values)]


def both(A, n, units, stream):
    """(plan result, no-alloc result) for the same A, B and pieces."""
    rp, ci, vv = device_csr(A)
    B = torch.from_numpy(gen.dense_uniform(A.k, n, seed=n)).cuda()
    Cp = torch.full((A.m, n), float("nan"), device="cuda")
    Cn = torch.full((A.m, n), float("nan"), device="cuda")
    with sd.sd_plan_device(rp, ci, vv, A.m, A.k, A.nnz, n, stream=stream, force="csr_merge",
                           units=units) as plan:
        sd.sd_spmm(plan, B, Cp, stream)
    sd.sd_spmm_merge_noalloc(rp, ci, vv, A.m, A.k, A.nnz, n, B, Cn, units=units, stream=stream)
    torch.cuda.synchronize()
    return B.cpu().numpy(), Cp.cpu().numpy(), Cn.cpu().numpy()


@pytest.mark.parametrize("n", [1, 3, 64, 128])
def test_noalloc_matches_plan_two_calls(n):
    stream = torch.cuda.current_stream()
    cases = [gen.random_rows(3000, 3500, ragged(3000, 3500, 1), seed=1),  # the larger input first
             gen.random_rows(500, 700, ragged(500, 700, 2), seed=2)]
    for A, units in zip(cases, (777, 61)):
        print(f"case noalloc m={A.m} nnz={A.nnz} n={n} units={units}", flush=True)
        B, Cp, Cn = both(A, n, units, stream)
        assert Cn.tobytes() == Cp.tobytes()
        C64, S = oracle.spmm(A, B)
        assert_close(Cn, C64, S, f"noalloc n={n} m={A.m}")


def test_noalloc_default_units():
    """units = 0 takes the planner's rule (halved until the scratch holds it):
    checked against the oracle, on an R-MAT graph with heavy rows."""
    A = gen.rmat(13, 120000, seed=3)
    rp, ci, vv = device_csr(A)
    for n in (128, 8):
        B = gen.dense_uniform(A.k, n, seed=5)
        Bd = torch.from_numpy(B).cuda()
        C = torch.full((A.m, n), float("nan"), device="cuda")
        print(f"case noalloc default units rmat n={n}", flush=True)
        sd.sd_spmm_merge_noalloc(rp, ci, vv, A.m, A.k, A.nnz, n, Bd, C, stream=torch.cuda.current_stream())
        torch.cuda.synchronize()
        C64, S = oracle.spmm(A, B)
        assert_close(C.cpu().numpy(), C64, S, f"noalloc default n={n}")


def test_noalloc_rejects_without_launching():
    A = gen.uniform_rows(64, 64, 4, 0)
    rp, ci, vv = device_csr(A)
    B = torch.zeros((64, 8), device="cuda")
    C = torch.zeros((64, 8), device="cuda")
    Bw = torch.zeros((64, 4096), device="cuda")
    Cw = torch.zeros((64, 4096), device="cuda")
    with pytest.raises(sd.SparseDittoError) as e:  # scratch too small for these pieces at this width
        sd.sd_spmm_merge_noalloc(rp, ci, vv, A.m, A.k, A.nnz, 4096, Bw, Cw, units=1 << 20)
    assert e.value.status == sd.SD_ERR_UNSUPPORTED
    with pytest.raises(sd.SparseDittoError) as e:  # overlapping operands
        sd.sd_spmm_merge_noalloc(rp, ci, vv, A.m, A.k, A.nnz, 8, B, B, units=4)
    assert e.value.status == sd.SD_ERR_INVALID_VALUE
    with pytest.raises(sd.SparseDittoError) as e:
        sd.sd_spmm_merge_noalloc(rp, ci, vv, A.m, A.k, A.nnz, 0, B, C)
    assert e.value.status == sd.SD_ERR_INVALID_VALUE
    # an empty output is a no-op
    sd.sd_spmm_merge_noalloc(rp, ci, vv, 0, A.k, 0, 8, B, C)


def test_noalloc_misaligned_operands():
    """B and C one float past a 16-byte boundary: both paths take the 32-bit
    lane geometry, and give the same bits as each other."""
    A = gen.random_rows(700, 900, ragged(700, 900, 4), seed=4)
    rp, ci, vv = device_csr(A)
    stream = torch.cuda.current_stream()
    for n in (8, 64):
        Bh = gen.dense_uniform(A.k, n, seed=7)
        Bbuf = torch.empty(A.k * n + 1, device="cuda")
        Bd = Bbuf[1:].view(A.k, n)
        Bd.copy_(torch.from_numpy(Bh))
        Cp = torch.full((A.m * n + 1,), float("nan"), device="cuda")[1:].view(A.m, n)
        Cn = torch.full((A.m * n + 1,), float("nan"), device="cuda")[1:].view(A.m, n)
        print(f"case noalloc misaligned n={n}", flush=True)
        with sd.sd_plan_device(rp, ci, vv, A.m, A.k, A.nnz, n, stream=stream, force="csr_merge", units=97) as plan:
            sd.sd_spmm(plan, Bd, Cp, stream)
        sd.sd_spmm_merge_noalloc(rp, ci, vv, A.m, A.k, A.nnz, n, Bd, Cn, units=97, stream=stream)
        torch.cuda.synchronize()
        assert Cn.cpu().numpy().tobytes() == Cp.cpu().numpy().tobytes()
        C64, S = oracle.spmm(A, Bh)
        assert_close(Cn.cpu().numpy(), C64, S, f"noalloc misaligned n={n}")
