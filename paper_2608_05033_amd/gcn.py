"""Two-layer full-batch GCN whose sparse aggregations run through sd_spmm.

The paper's application study (Sec. "Evaluation", GCN paragraph) trains a
two-layer GCN on a normalised adjacency Â with four sparse aggregations per
epoch: Â·(X W1) and Â·(H1 W2) forward, Âᵀ·G at both widths backward. Only the
aggregation is replaced; the dense transforms, activation, loss and optimiser
are ordinary torch operations.

Each aggregation is `spmm(B, fwd, bwd)`: C = Â·B with plan `fwd`, and in the
backward pass dB = Âᵀ·dC with the transpose plan `bwd` (A is not assumed
symmetric).  Plans are built once per (graph, width) and reused every epoch.
"""
from __future__ import annotations

import torch

from . import Plan, sd_plan_device, sd_plan_ex, sd_spmm


class _SpMM(torch.autograd.Function):
    @staticmethod
    def forward(ctx, B, fwd: Plan, bwd: Plan):
        info = fwd.info
        if B.dim() != 2 or B.shape[0] != info["k"] or B.shape[1] != info["n"] or B.dtype != torch.float32:
            raise ValueError(f"spmm: B must be float32 [{info['k']}, {info['n']}], got {tuple(B.shape)} {B.dtype}")
        B = B.contiguous()
        C = torch.empty((info["m"], info["n"]), dtype=torch.float32, device=B.device)
        sd_spmm(fwd, B, C, torch.cuda.current_stream(B.device))
        ctx.bwd = bwd
        return C

    @staticmethod
    def backward(ctx, dC):
        bwd = ctx.bwd
        info = bwd.info
        dC = dC.contiguous()
        dB = torch.empty((info["m"], info["n"]), dtype=torch.float32, device=dC.device)
        sd_spmm(bwd, dC, dB, torch.cuda.current_stream(dC.device))
        return dB, None, None


def spmm(B: torch.Tensor, fwd: Plan, bwd: Plan) -> torch.Tensor:
    """C = Â·B; its gradient with respect to B is Âᵀ·dC (plan `bwd`)."""
    return _SpMM.apply(B, fwd, bwd)


class AggregationPlans:
    """Forward and transpose plans of one adjacency for each width used.

    A is a host CSR (an object with m, k, rowptr, colidx, values) or a
    torch sparse CSR tensor on the GPU; the latter is planned from device
    memory (sd_plan_device), its int64 indices narrowed to int32."""

    def __init__(self, A, widths, **plan_opts):
        self.plans = {}
        if isinstance(A, torch.Tensor):
            if A.layout != torch.sparse_csr or not A.is_cuda or A.dtype != torch.float32:
                raise ValueError("adjacency tensor must be a float32 sparse CSR tensor on the GPU")
            m, k = A.shape
            rowptr = A.crow_indices().to(torch.int32).contiguous()
            colidx = A.col_indices().to(torch.int32).contiguous()
            values = A.values().contiguous()
            stream = torch.cuda.current_stream(A.device)
            nnz = int(values.numel())

            def plan(n, **kw):
                return sd_plan_device(rowptr, colidx, values, m, k, nnz, n, stream=stream, **plan_opts, **kw)
        else:
            def plan(n, **kw):
                return sd_plan_ex(A, n, **plan_opts, **kw)
        for n in widths:
            self.plans[n] = (plan(n), plan(n, transpose=True))

    def __call__(self, B: torch.Tensor) -> torch.Tensor:
        fwd, bwd = self.plans[B.shape[1]]
        return spmm(B, fwd, bwd)

    def destroy(self):
        for fwd, bwd in self.plans.values():
            fwd.destroy()
            bwd.destroy()
        self.plans = {}


class GCN2(torch.nn.Module):
    """H1 = relu(Â X W1), logits = Â H1 W2 (transform, then aggregate)."""

    def __init__(self, A, in_feats: int, hidden: int, classes: int, device, seed: int = 0, **plan_opts):
        super().__init__()
        g = torch.Generator(device="cpu").manual_seed(seed)

        def glorot(fan_in, fan_out):
            bound = (6.0 / (fan_in + fan_out)) ** 0.5
            return (torch.rand((fan_in, fan_out), generator=g, dtype=torch.float32) * 2 - 1) * bound

        self.W1 = torch.nn.Parameter(glorot(in_feats, hidden).to(device))
        self.W2 = torch.nn.Parameter(glorot(hidden, classes).to(device))
        self.agg = AggregationPlans(A, sorted({hidden, classes}), **plan_opts)

    def forward(self, X: torch.Tensor) -> torch.Tensor:
        H1 = torch.relu(self.agg(X @ self.W1))
        return self.agg(H1 @ self.W2)


def train_epoch(model: GCN2, X, labels, opt) -> torch.Tensor:
    """One full-batch epoch: forward, cross-entropy, backward, optimiser step."""
    opt.zero_grad(set_to_none=True)
    loss = torch.nn.functional.cross_entropy(model(X), labels)
    loss.backward()
    opt.step()
    return loss.detach()
