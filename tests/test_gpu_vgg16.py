"""GPU parity on the batch-1 VGG-16 conv stack (13 3x3/pad-1 convs, ReLU after
each, 2x2 max-pool after stages 1-4), checked layer by layer and element by
element: the oracle recomputes each conv in full from the exact fp32 tensor
the GPU layer consumed.

* Unfused: conv (default plan) -> ReLU kernel -> pool kernel; every conv
  output within the tolerance, the ReLU and max-pool outputs bit for bit.
* Fused: the stack exactly as the benchmark times it -- one
  ilpm_conv2d_fwd_epilogue call per conv with ReLU (and the 2x2 max-pool
  after stages 1-4), default plans -- each layer's output against the
  oracle's conv -> ReLU (-> pool) of that layer's GPU input, within the
  tolerance of the window element the maximum comes from (ReLU and max are
  1-Lipschitz, so the largest tolerance in a window bounds the difference).
* Fused on prepacked weights: the same with ilpm_conv2d_plan_for's plans
  (prepacked, per epilogue) and ilpm_conv2d_fwd_prepacked_epilogue, as the
  benchmark's prepacked stack runs it."""
import numpy as np
import pytest

import oracle
import workloads
from gpu_common import assert_matches, dev, note, torch_cuda

pytestmark = pytest.mark.gpu


def _pool_max(a):
    """2x2 / stride-2 maximum (floor) of [1, C, H, W] float64, exactly."""
    _, c, h, w = a.shape
    return a[:, :, : h // 2 * 2, : w // 2 * 2].reshape(1, c, h // 2, 2, w // 2, 2).max(axis=(3, 5))


def test_vgg16_stack_layerwise():
    torch = torch_cuda()
    import paper_1909_02765_amd as ilpm
    oracle.set_threads(16)
    x = dev(workloads.vgg16_input())
    for name, ci, co, hw, pool, seed in workloads.vgg16_layers():
        w_np = workloads.vgg16_weights(ci, co, seed)
        plan = ilpm.plan(ci, hw, hw, co, 3, 1, 1)
        note(f"[vgg16] {name} {ci}->{co} @{hw} path={plan.path} v={plan.variant} splits={plan.splits}")
        y = ilpm.conv2d(x, dev(w_np), None, 1, 1)
        torch.cuda.synchronize()
        x_np = x.cpu().numpy()
        y_np = y.cpu().numpy()
        ref, sab = oracle.conv2d_f64(x_np, w_np, None, 1, 1)
        assert_matches(y_np, ref, sab, ci, 3, name)
        ilpm.relu_(y)
        torch.cuda.synchronize()
        r_np = y.cpu().numpy()
        np.testing.assert_array_equal(r_np, oracle.relu(y_np))
        if pool:
            x = ilpm.maxpool2x2(y)
            torch.cuda.synchronize()
            np.testing.assert_array_equal(x.cpu().numpy(), oracle.maxpool2x2(r_np))
        else:
            x = y
    assert tuple(x.shape) == (1, 512, 14, 14)


def test_vgg16_fused_stack_against_oracle():
    torch = torch_cuda()
    import paper_1909_02765_amd as ilpm
    oracle.set_threads(16)
    x = dev(workloads.vgg16_input())
    for name, ci, co, hw, pool, seed in workloads.vgg16_layers():
        w_np = workloads.vgg16_weights(ci, co, seed)
        epi = ilpm.EPI_RELU | (ilpm.EPI_MAXPOOL2 if pool else 0)
        plan = ilpm.plan_for(ci, hw, hw, co, 3, 1, 1, epi)
        note(f"[vgg16 fused] {name} {ci}->{co} @{hw} epi={epi} path={plan.path} "
             f"v={ilpm.variant_name(plan.path, plan.variant)} splits={plan.splits}")
        y = torch.empty(ilpm.epilogue_out_shape(co, hw, hw, 3, 1, 1, epi), device="cuda", dtype=torch.float32)
        ilpm.conv2d_epilogue_launcher(x, dev(w_np), None, 1, 1, epi, y)()
        torch.cuda.synchronize()
        ref, sab = oracle.conv2d_f64(x.cpu().numpy(), w_np, None, 1, 1)
        tol = oracle.tolerance(sab, ci, 3)
        want = np.maximum(ref, 0.0)
        if pool:
            want, tol = _pool_max(want), _pool_max(tol)
        got = y.cpu().numpy().astype(np.float64)
        assert got.shape == want.shape, (name, got.shape, want.shape)
        assert np.isfinite(got).all(), name
        err = np.abs(got - want)
        assert (err <= tol).all(), f"{name}: worst |gpu-ref|/tol {np.max(err / tol):.3g}"
        x = y
    assert tuple(x.shape) == (1, 512, 14, 14)


def _check_fused_layer(name, x_gpu, w_np, ci, pool, y):
    ref, sab = oracle.conv2d_f64(x_gpu.cpu().numpy(), w_np, None, 1, 1)
    tol = oracle.tolerance(sab, ci, 3)
    want = np.maximum(ref, 0.0)
    if pool:
        want, tol = _pool_max(want), _pool_max(tol)
    got = y.cpu().numpy().astype(np.float64)
    assert got.shape == want.shape, (name, got.shape, want.shape)
    assert np.isfinite(got).all(), name
    err = np.abs(got - want)
    assert (err <= tol).all(), f"{name}: worst |gpu-ref|/tol {np.max(err / tol):.3g}"


def test_vgg16_fused_prepacked_stack_against_oracle():
    torch = torch_cuda()
    import paper_1909_02765_amd as ilpm
    oracle.set_threads(16)
    x = dev(workloads.vgg16_input())
    for name, ci, co, hw, pool, seed in workloads.vgg16_layers():
        w_np = workloads.vgg16_weights(ci, co, seed)
        epi = ilpm.EPI_RELU | (ilpm.EPI_MAXPOOL2 if pool else 0)
        plan = ilpm.plan_for(ci, hw, hw, co, 3, 1, 1, epi, prepacked=True)
        packed = ilpm.prepack_weights(dev(w_np), plan)
        note(f"[vgg16 fused prepacked] {name} {ci}->{co} @{hw} epi={epi} path={plan.path} "
             f"v={ilpm.variant_name(plan.path, plan.variant)} splits={plan.splits}")
        y = ilpm.conv2d_prepacked_epilogue(x, packed, co, 3, None, 1, 1, epi, plan=plan)
        torch.cuda.synchronize()
        _check_fused_layer(name, x, w_np, ci, pool, y)
        x = y
    assert tuple(x.shape) == (1, 512, 14, 14)


def test_relu_and_maxpool_odd_sizes():
    torch = torch_cuda()
    import paper_1909_02765_amd as ilpm
    a = workloads.uniform(77, (1, 5, 9, 13), -1.0, 1.0)
    t = dev(a)
    note("[stack ops] maxpool 9x13")
    p = ilpm.maxpool2x2(t)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(p.cpu().numpy(), oracle.maxpool2x2(a))
    ilpm.relu_(t)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(t.cpu().numpy(), oracle.relu(a))
