"""Helpers shared by the GPU tests: run the HIP path and the fp64 oracle on identical inputs."""
from __future__ import annotations

import numpy as np
import torch

from oracle import dense_step
from workloads import Stream, Workload

DEV = torch.device("cuda:0")


def rel(a, b) -> float:
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    return float(np.linalg.norm(a - b) / max(np.linalg.norm(b), 1e-300))


def to_dev(*arrs):
    return [torch.from_numpy(np.ascontiguousarray(a)).to(DEV) for a in arrs]


def make_factored(w: Workload, V0: np.ndarray, m_max=None, K_max=None, U0=None):
    import paper_1606_08061_amd as lst

    f = lst.Factored(w.D, w.d, m_max or w.m, w.K if K_max is None else K_max, w.loss,
                     float(np.float32(w.eps)), device=DEV)
    f.init(to_dev(V0)[0], None if U0 is None else to_dev(U0)[0])
    f.check("init")
    return f


def make_naive(w: Workload, W0: np.ndarray, m_max=None, K_max=None):
    import paper_1606_08061_amd as lst

    n = lst.Naive(w.D, w.d, m_max or w.m, w.K if K_max is None else K_max, w.loss,
                  float(np.float32(w.eps)), device=DEV)
    n.init(to_dev(W0)[0])
    return n


def oracle_step(W, H, idx, val, w: Workload):
    # the oracle takes the float64 values of the exact float32 inputs, lr and eps included
    return dense_step(W, H, idx, val, np.float32(w.lr), w.loss, np.float32(w.eps))


class Compare:
    """Runs n steps of a workload on a GPU context and on the oracle, step by step."""

    def __init__(self, w: Workload, path: str = "factored", seed=None, U0=None):
        self.w = w
        self.s = Stream(w, seed=seed)
        self.W = self.s.V0.astype(np.float64)
        if U0 is not None:  # float32 U0 on the GPU, its float64 value in the oracle
            self.W = self.W @ np.asarray(U0, dtype=np.float32).astype(np.float64)
        if path == "factored":
            self.ctx = make_factored(w, self.s.V0, U0=U0)
        else:
            self.ctx = make_naive(w, self.s.V0)
        self.steps = 0

    def step(self, batch=None):
        H, idx, val = batch if batch is not None else self.s.batch()
        ref = oracle_step(self.W, H, idx, val, self.w)
        loss, grad = self.ctx.step(*to_dev(H, idx, val), self.w.lr)
        st = self.ctx.sync_status()
        self.W = ref.W_new
        self.steps += 1
        return st, float(loss.item()), grad.cpu().numpy(), ref

    def W_gpu(self) -> np.ndarray:
        return self.ctx.materialize_W().cpu().numpy()

    def close(self):
        self.ctx.close()
