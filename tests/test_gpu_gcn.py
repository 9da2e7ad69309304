"""The two-layer GCN built on sd_spmm: the autograd wrapper against the
oracle (C = Â·B and dB = Âᵀ·dC), one training step against an fp64 CPU
reference of the whole forward and backward pass, and a short training run."""
import numpy as np
import pytest

import gen
import oracle
from spmm_check import assert_close

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():  # pragma: no cover - CPU container
    pytest.skip("needs a GPU", allow_module_level=True)

import scipy.sparse  # noqa: E402

import paper_2608_05033_amd as sd  # noqa: E402
from paper_2608_05033_amd import gcn  # noqa: E402


def graph(scale=11, edges=30000, nmax=None, seed=3):
    return gen.rmat(scale, edges, nmax=nmax, seed=seed)


@pytest.mark.parametrize("n", [8, 64, 128])
def test_spmm_autograd_matches_oracle(n):
    A = graph(nmax=1900)
    print(f"case gcn autograd m={A.m} nnz={A.nnz} n={n}", flush=True)
    B = gen.dense_normal(A.k, n, seed=n)
    R = gen.dense_normal(A.m, n, seed=n, stream=2)
    plans = gcn.AggregationPlans(A, [n])
    try:
        Bd = torch.from_numpy(B).cuda().requires_grad_(True)
        C = plans(Bd)
        (C * torch.from_numpy(R).cuda()).sum().backward()
        torch.cuda.synchronize()
        C64, S = oracle.spmm(A, B)
        assert_close(C.detach().cpu().numpy(), C64, S, f"gcn forward n={n}")
        G64, GS = oracle.spmm_transposed(A, R)
        assert_close(Bd.grad.cpu().numpy(), G64, GS, f"gcn backward n={n}")
    finally:
        plans.destroy()


def reference_step(A, X, labels, W1, W2):
    """fp64 forward and hand-derived backward of the same model."""
    Ah = scipy.sparse.csr_matrix((A.values.astype(np.float64), A.colidx, A.rowptr), shape=(A.m, A.k))
    X, W1, W2 = X.astype(np.float64), W1.astype(np.float64), W2.astype(np.float64)
    P1 = Ah @ (X @ W1)
    H1 = np.maximum(P1, 0.0)
    P2 = Ah @ (H1 @ W2)
    z = P2 - P2.max(axis=1, keepdims=True)
    prob = np.exp(z) / np.exp(z).sum(axis=1, keepdims=True)
    m = A.m
    loss = -np.mean(np.log(prob[np.arange(m), labels]))
    dP2 = prob.copy()
    dP2[np.arange(m), labels] -= 1.0
    dP2 /= m
    dZ2 = Ah.T @ dP2
    dW2 = H1.T @ dZ2
    dP1 = (dZ2 @ W2.T) * (P1 > 0)
    dZ1 = Ah.T @ dP1
    dW1 = X.T @ dZ1
    return loss, dW1, dW2


def rel(a, b):
    return float(np.linalg.norm(a - b) / max(np.linalg.norm(b), 1e-30))


def test_gcn_step_matches_fp64_reference():
    A = graph(scale=11, edges=25000, nmax=2000, seed=7)
    in_feats, hidden, classes = 48, 32, 8
    X = gen.dense_normal(A.m, in_feats, seed=1)
    labels = (np.arange(A.m) * 7919 % classes).astype(np.int64)
    print(f"case gcn step m={A.m} nnz={A.nnz}", flush=True)
    model = gcn.GCN2(A, in_feats, hidden, classes, device="cuda", seed=5)
    try:
        W1 = model.W1.detach().cpu().numpy().copy()
        W2 = model.W2.detach().cpu().numpy().copy()
        out = model(torch.from_numpy(X).cuda())
        loss = torch.nn.functional.cross_entropy(out, torch.from_numpy(labels).cuda())
        loss.backward()
        torch.cuda.synchronize()
        ref_loss, ref_dW1, ref_dW2 = reference_step(A, X, labels, W1, W2)
        assert abs(loss.item() - ref_loss) <= 1e-5 * max(1.0, abs(ref_loss))
        assert rel(model.W2.grad.cpu().numpy(), ref_dW2) <= 1e-4
        assert rel(model.W1.grad.cpu().numpy(), ref_dW1) <= 1e-4
    finally:
        model.agg.destroy()


def test_gcn_training_reduces_loss():
    """Labels a fixed random GCN can produce; 40 Adam epochs must cut the loss."""
    A = graph(scale=11, edges=25000, nmax=2000, seed=11)
    in_feats, hidden, classes = 32, 16, 4
    X = torch.from_numpy(gen.dense_normal(A.m, in_feats, seed=2)).cuda()
    teacher = gcn.GCN2(A, in_feats, hidden, classes, device="cuda", seed=99)
    student = gcn.GCN2(A, in_feats, hidden, classes, device="cuda", seed=1)
    try:
        with torch.no_grad():
            labels = teacher(X).argmax(dim=1)
        opt = torch.optim.Adam(student.parameters(), lr=0.02)
        losses = [gcn.train_epoch(student, X, labels, opt).item() for _ in range(40)]
        print(f"gcn training loss {losses[0]:.4f} -> {losses[-1]:.4f}", flush=True)
        assert all(np.isfinite(losses))
        assert losses[-1] < 0.7 * losses[0]
    finally:
        teacher.agg.destroy()
        student.agg.destroy()


def test_plans_from_torch_sparse_csr():
    """Aggregation plans from a CUDA sparse CSR tensor (planned on the device)
    equal those from the host CSR, and give the same forward and backward bits."""
    A = graph(nmax=1900)
    n = 64
    adj = torch.sparse_csr_tensor(torch.from_numpy(A.rowptr.astype(np.int64)),
                                  torch.from_numpy(A.colidx.astype(np.int64)),
                                  torch.from_numpy(A.values), size=(A.m, A.k)).cuda()
    dev_plans = gcn.AggregationPlans(adj, [n])
    host_plans = gcn.AggregationPlans(A, [n])
    try:
        for (df, db), (hf, hb) in zip(dev_plans.plans.values(), host_plans.plans.values()):
            assert df.info["device_built"] == 1 and db.info["device_built"] == 1
            for d, h in ((df, hf), (db, hb)):
                assert {k: v for k, v in d.info.items() if k != "device_built"} == \
                    {k: v for k, v in h.info.items() if k != "device_built"}
        B = torch.from_numpy(gen.dense_normal(A.k, n, seed=2)).cuda()
        outs = []
        for plans in (dev_plans, host_plans):
            Bd = B.clone().requires_grad_(True)
            C = plans(Bd)
            C.sum().backward()
            outs.append((C.detach(), Bd.grad))
        torch.cuda.synchronize()
        assert torch.equal(outs[0][0], outs[1][0]) and torch.equal(outs[0][1], outs[1][1])
    finally:
        dev_plans.destroy()
        host_plans.destroy()
