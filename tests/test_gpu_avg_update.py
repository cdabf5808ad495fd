"""GPU parity of mtx_average_grads / mtx_sgd_update (average of R gradient buffers fused with
the momentum update) against the CPU oracle, through the C ABI."""
import numpy as np
import pytest
import torch

from oracle import oracle as orc
from paper_1704_04560_amd import mtx
from paper_1704_04560_amd import workloads as wl
from tests import parity

pytestmark = pytest.mark.gpu


def _dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


@pytest.mark.parametrize("R", [1, 2, 3, 4, 8, 16])
@pytest.mark.parametrize("n,pad", [(1, 0), (7, 0), (1000, 0), (1000003, 0), (4099, 5), (4096, 64)])
@pytest.mark.parametrize("mu", [0.0, 0.9])
def test_sgd_update_matches_oracle(R, n, pad, mu):
    print(f"[case] sgd_update R={R} n={n} ld={n + pad} mu={mu}", flush=True)
    ld = n + pad
    grads, w, v = wl.make_avg_update_inputs(R, n, seed=R * 7 + n, ld=ld)
    ref_avg, ref_w, ref_v = orc.average_update(grads, w, v if mu else None, 0.01, mu, n=n)
    gd, wd, vd = _dev(grads), _dev(w), _dev(v)
    avg = torch.empty(n, device="cuda")
    mtx.mtx_sgd_update(wd, vd if mu else None, gd, R, n, ld, 0.01, mu, avg)
    torch.cuda.synchronize()
    parity.assert_tensor_close(avg.cpu().numpy(), ref_avg, 1e-6, "average")
    parity.assert_update_close(wd.cpu().numpy(), ref_w, w, 1e-4)
    if mu:
        parity.assert_tensor_close(vd.cpu().numpy(), ref_v, 1e-6, "velocity")
    else:
        assert np.array_equal(vd.cpu().numpy(), v)


@pytest.mark.parametrize("R,n,ld", [(16, 100003, 100003), (5, 64, 64), (2, 3, 9)])
def test_average_grads_matches_oracle(R, n, ld):
    print(f"[case] average_grads R={R} n={n} ld={ld}", flush=True)
    grads, _, _ = wl.make_avg_update_inputs(R, n, seed=1, ld=ld)
    ref_avg, _, _ = orc.average_update(grads, np.zeros(n, np.float32), None, 0.0, 0.0, n=n)
    avg = torch.empty(n, device="cuda")
    mtx.mtx_average_grads(_dev(grads), R, n, ld, avg)
    torch.cuda.synchronize()
    parity.assert_tensor_close(avg.cpu().numpy(), ref_avg, 1e-6, "average")


def test_sgd_update_without_avg_output():
    R, n = 4, 12345
    grads, w, v = wl.make_avg_update_inputs(R, n, seed=3)
    _, ref_w, ref_v = orc.average_update(grads, w, v, 0.01, 0.9)
    wd, vd = _dev(w), _dev(v)
    mtx.mtx_sgd_update(wd, vd, _dev(grads), R, n, n, 0.01, 0.9, None)
    torch.cuda.synchronize()
    parity.assert_update_close(wd.cpu().numpy(), ref_w, w, 1e-4)
    parity.assert_tensor_close(vd.cpu().numpy(), ref_v, 1e-6, "velocity")


def test_microbench_size_sampled():
    """R = 16 buffers of 61,000,000 elements (the full microbenchmark size): the whole update on
    the GPU, checked against the oracle at 20,000 sampled elements plus the tail."""
    R, n = 16, 61_000_000
    print(f"[case] sgd_update full size R={R} n={n}", flush=True)
    grads, w, v = wl.make_avg_update_inputs(R, n, seed=0)
    idx = np.unique(np.concatenate([np.random.default_rng(0).choice(n, 20000, replace=False),
                                    np.arange(n - 7, n)]))
    ref_avg, ref_w, ref_v = orc.average_update(grads[:, idx], w[idx], v[idx], 0.01, 0.9)
    gd = _dev(grads)
    del grads
    wd, vd = _dev(w), _dev(v)
    avg = torch.empty(n, device="cuda")
    mtx.mtx_sgd_update(wd, vd, gd, R, n, n, 0.01, 0.9, avg)
    torch.cuda.synchronize()
    it = torch.from_numpy(idx).cuda()
    parity.assert_tensor_close(avg[it].cpu().numpy(), ref_avg, 1e-6, "average")
    parity.assert_tensor_close(vd[it].cpu().numpy(), ref_v, 1e-6, "velocity")
    parity.assert_update_close(wd[it].cpu().numpy(), ref_w, w[idx], 1e-4)
