"""GPU parity on the batch-1 VGG-16 conv stack (13 3x3/pad-1 convs, ReLU after
each, 2x2 max-pool after stages 1-4), checked layer by layer: the oracle
recomputes each conv from the exact fp32 tensor the GPU layer consumed (at
sampled output points plus the whole first and last output channel), and the
ReLU and max-pool outputs must equal the oracle's bit for bit."""
import numpy as np
import pytest

import oracle
import workloads
from gpu_common import assert_matches, dev, note, torch_cuda

pytestmark = pytest.mark.gpu


def sample_indices(c_out, ho, wo, n, seed):
    rng = np.random.default_rng(seed)
    plane = ho * wo
    idx = set(rng.integers(0, c_out * plane, size=n).tolist())
    idx.update(range(plane))                              # first output channel
    idx.update(range((c_out - 1) * plane, c_out * plane))  # last output channel
    return np.array(sorted(idx), dtype=np.int64)


def test_vgg16_stack_layerwise():
    torch = torch_cuda()
    import paper_1909_02765_amd as ilpm
    oracle.set_threads(16)
    x = dev(workloads.vgg16_input())
    for li, (name, ci, co, hw, pool, seed) in enumerate(workloads.vgg16_layers()):
        w_np = workloads.vgg16_weights(ci, co, seed)
        plan = ilpm.plan(ci, hw, hw, co, 3, 1, 1)
        note(f"[vgg16] {name} {ci}->{co} @{hw} path={plan.path} v={plan.variant} splits={plan.splits}")
        y = ilpm.conv2d(x, dev(w_np), None, 1, 1)
        torch.cuda.synchronize()
        x_np = x.cpu().numpy()
        y_np = y.cpu().numpy()
        idx = sample_indices(co, hw, hw, 4096, seed)
        ref, sab = oracle.conv2d_f64_points(x_np, w_np, None, 1, 1, idx)
        assert_matches(y_np.reshape(-1)[idx], ref, sab, ci, 3, name)
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
