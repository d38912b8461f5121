"""Parity at the full workload sizes (D = 200k / 800k), in the launch configuration the
benchmark times: one step of the factored and of the naive path against the fp64 oracle
(loss, grad_H and the whole updated W), rows of V outside the targets bit-identical, and
ten steps of the D = 200k squared-error workload."""
import numpy as np
import pytest
import torch

from gpu_common import DEV, make_factored, make_naive, oracle_step, rel, to_dev
from workloads import WORKLOADS, Stream

pytestmark = pytest.mark.gpu

FULL = ["sq_D200k_d500_m128_K5", "sphsm_D200k_d500_m128_zipf", "sq_D800k_d512_m256_K10_zipf"]


@pytest.mark.parametrize("name", FULL)
def test_full_size_single_step(name):
    w = WORKLOADS[name]
    s = Stream(w)
    H, idx, val = s.batch()
    print(f"[{name}] oracle step", flush=True)
    ref = oracle_step(s.V0, H, idx, val, w)
    b = to_dev(H, idx, val)

    f = make_factored(w, s.V0)
    V_before = f.V.clone()
    loss, grad = f.step(*b, w.lr)
    assert f.sync_status() == 0
    assert abs(loss.item() - ref.loss) <= 1e-4 * abs(ref.loss)
    assert rel(grad.cpu().numpy(), ref.grad_H) <= 1e-4
    touched = torch.zeros(w.D, dtype=torch.bool, device=DEV)
    touched[torch.from_numpy(idx.reshape(-1).astype(np.int64)).to(DEV)] = True
    assert torch.equal(f.V[~touched], V_before[~touched])
    del V_before
    Wf = f.materialize_W().cpu().numpy()
    assert rel(Wf, ref.W_new) <= 1e-4
    f.close()
    del Wf

    n = make_naive(w, s.V0)
    loss_n, grad_n = n.step(*b, w.lr)
    assert n.sync_status() == 0
    assert abs(loss_n.item() - ref.loss) <= 1e-4 * abs(ref.loss)
    assert rel(grad_n.cpu().numpy(), ref.grad_H) <= 1e-4
    assert rel(n.W.cpu().numpy(), ref.W_new) <= 1e-4
    n.close()


def test_full_size_ten_steps():
    w = WORKLOADS["sq_D200k_d500_m128_K5"]
    s = Stream(w)
    W = s.V0.astype(np.float64)
    f = make_factored(w, s.V0)
    for t in range(10):
        H, idx, val = s.batch()
        ref = oracle_step(W, H, idx, val, w)
        loss, grad = f.step(*to_dev(H, idx, val), w.lr)
        assert f.sync_status() == 0
        tol = 1e-4 if t == 0 else 1e-3
        assert abs(loss.item() - ref.loss) <= tol * abs(ref.loss)
        assert rel(grad.cpu().numpy(), ref.grad_H) <= tol
        W = ref.W_new
        print(f"step {t} ok", flush=True)
    assert rel(f.materialize_W().cpu().numpy(), W) <= 1e-3
    f.close()
