"""GPU: ilpm_conv2d_fwd_noalloc (split plans keep their partial sums in the
library's fixed per-device array instead of an allocated workspace) gives
exactly the bits of ilpm_conv2d_fwd, and agrees with the oracle, on two calls
in a row -- the second with a smaller input -- and then on the first shape
again (the array keeps the previous call's contents; nothing may depend on
them)."""
import numpy as np
import pytest

import oracle
import workloads
from gpu_common import GUARD, assert_matches, dev, note, torch_cuda


# (C_in, H, W, C_out, K, stride, pad): a 512-channel 14x14 layer whose plan
# splits the input channels 8 ways (3 MiB of partial sums), then a smaller
# 256-channel 7x7 one (4 splits), then a one-split layer, then the first again.
SHAPES = [(512, 14, 14, 512, 3, 1, 1), (256, 7, 7, 256, 3, 1, 1), (32, 20, 24, 40, 3, 1, 1),
          (512, 14, 14, 512, 3, 1, 1)]


def _case(i, c_in, h, w, c_out, k):
    x = workloads.uniform(9100 + 10 * i, (1, c_in, h, w), 0.0, 1.0)
    wt = workloads.normal(9101 + 10 * i, (c_out, c_in, k, k), 0.0, workloads.he_std(c_in, k))
    b = workloads.normal(9102 + 10 * i, (c_out,), 0.0, 0.1)
    return x, wt, b


@pytest.mark.gpu
def test_noalloc_matches_fwd_on_consecutive_calls():
    torch = torch_cuda()
    import paper_1909_02765_amd as ilpm
    oracle.set_threads(16)
    for i, (c_in, h, w, c_out, k, s, p) in enumerate(SHAPES):
        x, wt, b = _case(i % 3, c_in, h, w, c_out, k)
        plan = ilpm.plan(c_in, h, w, c_out, k, s, p)
        assert plan.workspace_bytes <= ilpm.NOALLOC_SCRATCH_BYTES
        xd, wd, bd = dev(x), dev(wt), dev(b)
        ho, wo = ilpm.out_size(h, k, s, p), ilpm.out_size(w, k, s, p)
        n = c_out * ho * wo
        note(f"[noalloc] call {i}: shape {(c_in, h, w, c_out, k, s, p)} splits={plan.splits} "
             f"workspace={plan.workspace_bytes}")
        buf = torch.full((n + 2 * GUARD,), float("nan"), device="cuda", dtype=torch.float32)
        out = buf[GUARD:GUARD + n].view(1, c_out, ho, wo)
        ilpm.conv2d_noalloc(xd, wd, bd, s, p, out=out)
        torch.cuda.synchronize()
        assert torch.isnan(buf[:GUARD]).all() and torch.isnan(buf[GUARD + n:]).all(), "write outside out"
        got = out.cpu().numpy()
        want = ilpm.conv2d(xd, wd, bd, s, p)
        torch.cuda.synchronize()
        np.testing.assert_array_equal(got, want.cpu().numpy(), err_msg=f"call {i}: noalloc != fwd")
        ref, sab = oracle.conv2d_f64(x, wt, b, s, p)
        assert_matches(got, ref, sab, c_in, k, f"noalloc call {i}")


_CHILD = r"""
import ctypes, sys
sys.path.insert(0, {root!r})
import paper_1909_02765_amd as ilpm
# Host pointers that are never dereferenced: the size check comes first.
print(ilpm.lib.ilpm_conv2d_fwd_noalloc(0x1000, 0x10000000, None, 512, 28, 28, 512, 3, 1, 1, 0x40000000, None))
"""


@pytest.mark.parametrize("splits,want", [("64", -3)])
def test_noalloc_rejects_a_plan_beyond_the_array(splits, want):
    """With 64 forced splits the 512->512 @28 plan needs 64 x 1.6 MB of partial
    sums, beyond the fixed array: ILPM_ERR_WORKSPACE, before any device
    access (this runs without a GPU)."""
    import os
    import subprocess
    import sys
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    env = {k: v for k, v in os.environ.items() if not k.startswith("ILPM_")}
    env.update(ILPM_SPLIT=splits, ILPM_TILE="7x7")
    r = subprocess.run([sys.executable, "-c", _CHILD.format(root=root)], capture_output=True, text=True,
                       env=env, timeout=300)
    assert r.returncode == 0, r.stderr
    assert int(r.stdout.strip().splitlines()[-1]) == want
