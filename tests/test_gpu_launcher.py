"""GPU: a launcher keeps the tensors it marshalled alive.  The launchers hold
raw device addresses; if the tensors behind them could be freed, emptying
torch's cache (as every graph capture does first) would return their memory
to the driver and the next launch would read unmapped memory.  The test
checks that the tensors survive before it launches anything."""
import gc
import weakref

import numpy as np
import pytest

import workloads
from gpu_common import dev, note, torch_cuda

pytestmark = pytest.mark.gpu


def test_launchers_keep_their_tensors_alive():
    torch = torch_cuda()
    import paper_1909_02765_amd as ilpm
    c_in, h, c_out = 16, 20, 32
    x = dev(workloads.uniform(9100, (1, c_in, h, h), 0.0, 1.0))
    w = dev(workloads.normal(9101, (c_out, c_in, 3, 3), 0.0, workloads.he_std(c_in, 3)))
    want = ilpm.conv2d(x, w, None, 1, 1)
    want_epi = ilpm.conv2d_epilogue(x, w, None, 1, 1, ilpm.EPI_RELU | ilpm.EPI_MAXPOOL2)
    torch.cuda.synchronize()
    want, want_epi = want.cpu().numpy(), want_epi.cpu().numpy()
    out = torch.empty((1, c_out, h, h), device="cuda", dtype=torch.float32)
    out_epi = torch.empty((1, c_out, h // 2, h // 2), device="cuda", dtype=torch.float32)
    launch = ilpm.conv2d_launcher(x, w, None, 1, 1, out)
    launch_epi = ilpm.conv2d_epilogue_launcher(x, w, None, 1, 1, ilpm.EPI_RELU | ilpm.EPI_MAXPOOL2, out_epi)
    refs = [weakref.ref(t) for t in (x, w, out, out_epi)]
    del x, w, out, out_epi
    gc.collect()
    torch.cuda.empty_cache()
    assert all(r() is not None for r in refs), "a launcher let go of a tensor it points at"
    note("[launcher] launch after the caller dropped its tensors")
    launch()
    launch_epi()
    torch.cuda.synchronize()
    np.testing.assert_array_equal(refs[2]().cpu().numpy(), want)
    np.testing.assert_array_equal(refs[3]().cpu().numpy(), want_epi)
