"""GPU: the Winograd F(2x2, 3x3) comparison path against the oracle -- within
the acceptance tolerance and within its own worst-case rounding bound -- on
the 3x3 / stride-1 workloads and ragged shapes (odd output sizes leave
partial 2x2 tiles)."""
import numpy as np
import pytest

import oracle
import workloads
from gpu_common import dev, note, random_case, torch_cuda
from winograd_math import G, error_bound

pytestmark = pytest.mark.gpu

CASES = [c for c in workloads.ALL_CASES if c.k == 3 and c.stride == 1]


@pytest.fixture(scope="module")
def ilpm():
    torch_cuda()
    import paper_1909_02765_amd as m
    oracle.set_threads(16)
    return m


def run_and_check(ilpm, name, x, w, b, pad):
    torch = torch_cuda()
    c_in = x.shape[1]
    ref, sab = oracle.conv2d_f64(x, w, b, 1, pad)
    note(f"[winograd] {name}")
    u = ilpm.winograd_transform_filter(dev(w))
    got = ilpm.conv2d_winograd(dev(x), u, dev(b), pad)
    again = ilpm.conv2d_winograd(dev(x), u, dev(b), pad)
    torch.cuda.synchronize()
    g = got.cpu().numpy().astype(np.float64)
    np.testing.assert_array_equal(got.cpu().numpy(), again.cpu().numpy())
    err = np.abs(g - ref)
    tol = oracle.tolerance(sab, c_in, 3)
    assert (err <= tol).all(), f"{name}: tolerance ratio {np.max(err / tol)}"
    assert (err <= error_bound(x, w, pad) + 1e-30).all(), f"{name}: outside the rounding bound"
    return u


@pytest.mark.parametrize("case", CASES, ids=lambda c: c.name)
def test_winograd_workloads(ilpm, case):
    x, w, b = case.inputs()
    run_and_check(ilpm, case.name, x, w, b, case.pad)


def test_winograd_ragged_and_filter_layout(ilpm):
    for seed, (c_in, h, w_, c_out, pad) in enumerate([(5, 9, 11, 7, 1), (3, 6, 5, 4, 0), (17, 13, 8, 33, 2),
                                                      (1, 3, 3, 1, 1)]):
        x, w, b = random_case(9500 + 10 * seed, c_in, h, w_, c_out, 3)
        u = run_and_check(ilpm, f"ragged{seed}", x, w, b, pad)
        # U[4*xi + nu][co][ci] = (G g G^T)[xi][nu], to fp32 rounding of the transform
        want = np.einsum("ij,ocjk,lk->iloc", G, w.astype(np.float64), G).reshape(16, c_out, c_in)
        mag = np.einsum("ij,ocjk,lk->iloc", np.abs(G), np.abs(w.astype(np.float64)), np.abs(G)).reshape(16, c_out, c_in)
        got = u.cpu().numpy().astype(np.float64)
        assert (np.abs(got - want) <= 6 * 2.0 ** -24 * mag + 1e-30).all()
