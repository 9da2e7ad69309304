"""sd_spmm inside a captured HIP graph: it allocates nothing and does not
synchronise, so a caller can capture it.  Each family is captured once and
replayed several times with B changed by eager work between replays; every
replay must equal the eager call on the same B bitwise (the kernels' order
of summation does not depend on the launch path)."""
import numpy as np
import pytest

import gen

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():  # pragma: no cover - CPU container
    pytest.skip("needs a GPU", allow_module_level=True)

import paper_2608_05033_amd as sd  # noqa: E402

CASES = [
    ("csr_row", 64, {}),
    ("csr_row", 1, {}),
    ("csr_split", 64, {"heavy_threshold": 40, "chunk_nnz": 17}),
    ("csr_split", 8, {"heavy_threshold": 40, "chunk_nnz": 17}),
    ("csr_merge", 32, {"units": 97}),
    ("ell", 64, {}),
    ("sell", 16, {}),
    ("win", 16, {}),
    ("bsr", 64, {"engine": "mfma"}),
    ("bsr", 32, {"engine": "mfma"}),
    ("bell", 48, {"engine": "valu"}),
]


def _matrix(fam):
    if fam in ("bsr", "bell"):
        return gen.block(40, 45, 16, 9, 12, 0.9, 3)
    if fam in ("ell", "sell", "win"):
        return gen.laplacian3d(12, 10, 9)
    lengths = np.random.default_rng(1).integers(0, 60, 2000)
    lengths[1000] = 2500
    return gen.random_rows(2000, 3001, lengths, seed=1)


@pytest.mark.parametrize("fam,n,opts", CASES, ids=[f"{f}-{n}" for f, n, _ in CASES])
def test_captured_graph_replays(fam, n, opts):
    A = _matrix(fam)
    print(f"case graph {fam} n={n} m={A.m} nnz={A.nnz}", flush=True)
    with sd.sd_plan_ex(A, n, force=fam, **opts) as plan:
        B = torch.from_numpy(gen.dense_uniform(A.k, n, seed=3)).cuda()
        C = torch.full((A.m, n), float("nan"), device="cuda")
        ref = torch.empty_like(C)
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):  # warm-up launch outside the capture
            sd.sd_spmm(plan, B, C, side)
        torch.cuda.current_stream().wait_stream(side)
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            sd.sd_spmm(plan, B, C, torch.cuda.current_stream())
        for rep in range(4):
            B.mul_(-0.5).add_(0.25 * rep)  # eager work between replays
            torch.cuda.synchronize()
            C.fill_(float("nan"))
            g.replay()
            torch.cuda.synchronize()
            sd.sd_spmm(plan, B, ref, torch.cuda.current_stream())
            torch.cuda.synchronize()
            assert torch.equal(C, ref), f"replay {rep} differs from the eager call"
        del g
