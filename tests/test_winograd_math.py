"""The Winograd F(2x2, 3x3) transforms, in fp64, reproduce the convolution of
the oracle exactly (to fp64 rounding) -- the matrices the comparison path
uses are the right ones -- and the error-bound sum dominates the direct one."""
import numpy as np
import pytest

import oracle
import workloads
from winograd_math import error_bound, winograd_conv


@pytest.mark.parametrize("shape", [(1, 4, 4, 1, 0), (3, 7, 9, 5, 1), (8, 11, 6, 4, 1), (2, 5, 5, 3, 2)])
def test_winograd_fp64_equals_definition(shape):
    c_in, h, w, c_out, pad = shape
    x = workloads.uniform(9100 + c_in, (1, c_in, h, w), -1.0, 1.0)
    wt = workloads.uniform(9200 + c_out, (c_out, c_in, 3, 3), -1.0, 1.0)
    b = workloads.uniform(9300, (c_out,), -1.0, 1.0)
    ref, sab = oracle.conv2d_f64(x, wt, b, 1, pad)
    got = winograd_conv(x, wt, b, pad)
    assert got.shape == ref.shape
    np.testing.assert_allclose(got, ref, rtol=0, atol=1e-12 * (1 + sab.max()))
    # The absolute-value Winograd sum bounds the direct product sum from above.
    wabs = winograd_conv(x, wt, None, pad, absolute=True)
    assert (wabs >= sab - 1e-12 * (1 + sab)).all()


def test_winograd_fp32_within_bound_and_tolerance():
    """The same transforms carried out in fp32 (numpy's summation order, not
    the GPU's) stay within the worst-case rounding bound and within the
    acceptance tolerance 1e-4 (1 + S / (C_in K^2)) on the 3x3 workloads --
    the worst-case bound itself is far looser than the tolerance for wide
    layers, as is the direct sum's; realistic rounding is what the tolerance
    measures."""
    from winograd_math import error_bound
    for case in (workloads.TINY, workloads.RESNET_CONV4, workloads.RESNET_CONV5):
        x, w, b = case.inputs()
        ref, sab = oracle.conv2d_f64(x, w, b, 1, case.pad)
        got = winograd_conv(x, w, b, case.pad, dtype=np.float32).astype(np.float64)
        err = np.abs(got - ref)
        assert (err <= error_bound(x, w, case.pad) + 1e-30).all(), case.name
        tol = oracle.tolerance(sab, case.c_in, 3)
        assert (err <= tol).all(), f"{case.name}: worst {np.max(err / tol)}"
