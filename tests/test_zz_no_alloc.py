"""The allocation-free step (lst_step_noalloc, its intermediates in the library's fixed
device array) against lst_step on a context, from the same state: consecutive calls, the
later ones with a smaller minibatch and fewer slots (another layout in the same array,
whose arrival counters must start at zero again), then the first shape again."""
import numpy as np
import pytest
import torch

import paper_1606_08061_amd as lst
from gpu_common import DEV, make_factored, rel, to_dev
from workloads import LOSS_SPHERICAL_SOFTMAX, LOSS_SQUARED, LOSS_TAYLOR_SOFTMAX, Stream, Workload

pytestmark = pytest.mark.gpu

TOL = 1e-4


@pytest.mark.parametrize("loss", [LOSS_SQUARED, LOSS_SPHERICAL_SOFTMAX, LOSS_TAYLOR_SOFTMAX,
                                  "squared_frequent_rows", "squared_m512"])
def test_noalloc_step_matches_lst_step(loss):
    shapes = None
    if loss == "squared_frequent_rows":
        # six rows targeted by every example: every row is summed in chunks, whose arrival
        # counters sit in the array at another place for each layout
        w = Workload("t", LOSS_SQUARED, 6, 64, 128, 6, lr=1e-3)
        loss = LOSS_SQUARED
    elif loss == "squared_m512":
        # m = 512 (the 64 x 64 tiles of launches 1 and 3), then m = 300 (32 x 32 tiles: the
        # plan and the carve change in the same array), then m = 512 again
        w = Workload("t", LOSS_SQUARED, 20000, 320, 512, 5)
        loss = LOSS_SQUARED
        shapes = [(512, 5), (300, 4), (512, 5)]
    else:
        sq = loss == LOSS_SQUARED
        w = Workload("t", loss, 20000, 256, 128, 5 if sq else 3,
                     index_dist="uniform" if sq else "zipf",
                     value_dist="normal" if sq else "ones")
    s = Stream(w)
    f = make_factored(w, s.V0)
    V, U, UinvT, Q, WO = (t.clone() for t in (f.V, f.U, f.UinvT, f.Q, f.WO))
    loss_dev = torch.zeros(1, dtype=torch.float32, device=DEV)
    status = torch.full((1,), 99, dtype=torch.int32, device=DEV)
    stream = torch.cuda.current_stream(DEV).cuda_stream
    for m, K in shapes or [(128, w.K), (40, w.K - 1), (128, w.K)]:
        print(f"noalloc step: loss {loss}, m {m}, K {K}", flush=True)
        H, idx, val = s.batch(m)
        idx, val = np.ascontiguousarray(idx[:, :K]), np.ascontiguousarray(val[:, :K])
        Hd, idxd, vald = to_dev(H, idx, val)
        l_ref, g_ref = f.step(Hd, idxd, vald, w.lr)
        assert f.sync_status() == 0
        grad = torch.empty((m, w.d), dtype=torch.float32, device=DEV)
        st = lst.lst_step_noalloc(w.D, w.d, lst.LOSSES[loss], float(np.float32(w.eps)),
                                  V.data_ptr(), w.d, U.data_ptr(), UinvT.data_ptr(),
                                  Q.data_ptr(), WO.data_ptr(), w.d, Hd.data_ptr(), m,
                                  idxd.data_ptr(),
                                  vald.data_ptr(), K, w.lr, loss_dev.data_ptr(),
                                  grad.data_ptr(), status.data_ptr(), stream)
        assert st == lst.LST_OK
        torch.cuda.synchronize(DEV)
        assert int(status.item()) == 0
        assert abs(loss_dev.item() - l_ref.item()) <= TOL * abs(l_ref.item())
        assert rel(grad.cpu().numpy(), g_ref.cpu().numpy()) <= TOL
        for mine, theirs in ((V, f.V), (U, f.U), (UinvT, f.UinvT), (Q, f.Q), (WO, f.WO)):
            assert rel(mine.cpu().numpy(), theirs.cpu().numpy()) <= TOL
    f.close()
