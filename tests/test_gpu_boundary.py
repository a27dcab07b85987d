"""GPU: the boundary's workspace rules.  A call that would have to grow the
library-owned workspace while its stream is being captured returns
ILPM_ERR_WORKSPACE (nothing is allocated during capture); once sized, the
same call captures and every replay equals the eager result; and growing the
workspace later leaves an earlier graph valid, since the smaller buffer is
kept rather than freed."""
import numpy as np
import pytest

import workloads
from gpu_common import dev, note, torch_cuda

pytestmark = pytest.mark.gpu


def _split_plan(ilpm, c_in, h, w, c_out, splits):
    """An explicit matrix-core plan with `splits` input-channel splits on
    7x7-tile variant k3s1_t7x7_co64 (a workspace of splits full-size slices,
    summed by the second kernel)."""
    v = [i for i in range(ilpm.num_variants(ilpm.PATH_IGEMM))
         if ilpm.variant_name(ilpm.PATH_IGEMM, i) == "k3s1_t7x7_co64"][0]
    p = ilpm.plan_variant(c_in, h, w, c_out, 3, 1, 1, ilpm.PATH_IGEMM, v, splits)
    assert p.splits == splits and p.workspace_bytes == 4 * splits * c_out * h * w
    return p


def _inputs(seed, c_in, h, w, c_out):
    x = workloads.uniform(seed, (1, c_in, h, w), 0.0, 1.0)
    wt = workloads.normal(seed + 1, (c_out, c_in, 3, 3), 0.0, workloads.he_std(c_in, 3))
    return dev(x), dev(wt)


def test_capture_needs_a_sized_workspace_and_replays_exactly():
    torch = torch_cuda()
    import paper_1909_02765_amd as ilpm
    ilpm.set_workspace(None)
    # One small eager call first, so that the library's one-time device
    # queries are behind us before any capture.
    xs, ws_ = _inputs(7000, 4, 8, 8, 4)
    ilpm.conv2d(xs, ws_, None, 1, 1)
    torch.cuda.synchronize()
    # 512 input channels in 64 splits of 8: a 102 MB workspace, larger than
    # any other test's, so the library's own buffer is too small here.
    c_in, h, w, c_out = 512, 28, 28, 512
    plan = _split_plan(ilpm, c_in, h, w, c_out, 64)
    x, wt = _inputs(7100, c_in, h, w, c_out)
    out = torch.empty((1, c_out, h, w), device="cuda", dtype=torch.float32)
    stream = torch.cuda.Stream()
    stream.wait_stream(torch.cuda.current_stream())
    torch.cuda.synchronize()
    note("[boundary] capture before the workspace is sized")
    g = torch.cuda.CUDAGraph()
    status = None
    with torch.cuda.graph(g, stream=stream):
        try:
            ilpm.conv2d(x, wt, None, 1, 1, out=out, plan=plan)
        except ilpm.IlpmError as e:
            status = e.status
    torch.cuda.synchronize()
    assert status == ilpm.ERR_WORKSPACE, status
    del g

    note("[boundary] eager call sizes it; capture and replay")
    want = ilpm.conv2d(x, wt, None, 1, 1, plan=plan)
    torch.cuda.synchronize()
    want = want.cpu().numpy()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=stream):
        ilpm.conv2d(x, wt, None, 1, 1, out=out, plan=plan)
    torch.cuda.synchronize()
    for i in range(3):
        out.fill_(float("nan"))
        g.replay()
        torch.cuda.synchronize()
        np.testing.assert_array_equal(out.cpu().numpy(), want, err_msg=f"replay {i}")
        # eager work of the program's own between replays
        ilpm.conv2d(x, wt, None, 1, 1, plan=plan)
        torch.cuda.synchronize()


def test_growth_keeps_earlier_graphs_valid():
    torch = torch_cuda()
    import paper_1909_02765_amd as ilpm
    ilpm.set_workspace(None)
    # Graph A on a split plan, captured with the workspace sized for it; then
    # an eager call that needs a workspace larger than every other test's
    # (the library allocates a new one and keeps the old); then A again.
    ca, ha, coa = 256, 14, 256
    plan_a = _split_plan(ilpm, ca, ha, ha, coa, 8)
    xa, wa = _inputs(7200, ca, ha, ha, coa)
    want = ilpm.conv2d(xa, wa, None, 1, 1, plan=plan_a)
    torch.cuda.synchronize()
    want = want.cpu().numpy()
    out = torch.empty((1, coa, ha, ha), device="cuda", dtype=torch.float32)
    stream = torch.cuda.Stream()
    stream.wait_stream(torch.cuda.current_stream())
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    note("[boundary] capture graph A")
    with torch.cuda.graph(g, stream=stream):
        ilpm.conv2d(xa, wa, None, 1, 1, out=out, plan=plan_a)
    torch.cuda.synchronize()
    note("[boundary] grow the workspace (1024 channels in 128 splits)")
    cb, hb, cob = 1024, 28, 512
    plan_b = _split_plan(ilpm, cb, hb, hb, cob, 128)
    xb, wb = _inputs(7300, cb, hb, hb, cob)
    ilpm.conv2d(xb, wb, None, 1, 1, plan=plan_b)
    torch.cuda.synchronize()
    note("[boundary] replay graph A after the growth")
    for i in range(2):
        out.fill_(float("nan"))
        g.replay()
        torch.cuda.synchronize()
        np.testing.assert_array_equal(out.cpu().numpy(), want, err_msg=f"replay {i}")
