"""Helpers for the GPU parity tests: run the HIP path through the C ABI on
seeded inputs and compare with the CPU oracle element by element."""
from __future__ import annotations

import sys

import numpy as np

import oracle
import workloads

GUARD = 4096  # floats of NaN canary on each side of an output buffer


def torch_cuda():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    return torch


def dev(a):
    torch = torch_cuda()
    if a is None:
        return None
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).cuda()


def note(msg: str):
    """Name the case before a GPU step, flushed, so a failure is attributable."""
    print(msg, flush=True)
    sys.stdout.flush()


def run_conv(x, w, b, stride, pad, plan=None, guard=True, stream=None):
    """The GPU path's output as numpy (float32), with canaries around it checked."""
    import paper_1909_02765_amd as ilpm
    torch = torch_cuda()
    c_out, c_in, k, _ = w.shape
    ho = ilpm.out_size(x.shape[2], k, stride, pad)
    wo = ilpm.out_size(x.shape[3], k, stride, pad)
    n = c_out * ho * wo
    xd, wd, bd = dev(x), dev(w), dev(b)
    if guard:
        buf = torch.full((n + 2 * GUARD,), float("nan"), device="cuda", dtype=torch.float32)
        out = buf[GUARD:GUARD + n].view(1, c_out, ho, wo)
    else:
        buf = None
        out = torch.empty((1, c_out, ho, wo), device="cuda", dtype=torch.float32)
    ilpm.conv2d(xd, wd, bd, stride, pad, out=out, plan=plan, stream=stream)
    torch.cuda.synchronize()
    if guard:
        head = buf[:GUARD].cpu().numpy()
        tail = buf[GUARD + n:].cpu().numpy()
        assert np.isnan(head).all() and np.isnan(tail).all(), "write outside the output tensor"
    return out.cpu().numpy()


def assert_matches(got, ref, sab, c_in, k, what):
    ok, ratio, i = oracle.check(got, ref, sab, c_in, k)
    if not ok:
        g = np.asarray(got).reshape(-1)
        r = np.asarray(ref).reshape(-1)
        raise AssertionError(f"{what}: worst |gpu-ref|/tol = {ratio:.3g} at flat index {i} "
                             f"(gpu {g[i]!r}, ref {r[i]!r}), shape {np.shape(got)}")
    return ratio


def random_case(seed, c_in, h, w, c_out, k, bias=True):
    x = workloads.uniform(seed, (1, c_in, h, w), -1.0, 1.0)
    wt = workloads.uniform(seed + 1, (c_out, c_in, k, k), -0.5, 0.5)
    b = workloads.uniform(seed + 2, (c_out,), -1.0, 1.0) if bias else None
    return x, wt, b


def small_int_case(seed, c_in, h, w, c_out, k, bias=True):
    x = workloads.small_ints(seed, (1, c_in, h, w))
    wt = workloads.small_ints(seed + 1, (c_out, c_in, k, k))
    b = workloads.small_ints(seed + 2, (c_out,)) if bias else None
    return x, wt, b
