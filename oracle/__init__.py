"""CPU oracle for the batch-1 conv2d forward pass (ctypes wrapper of oracle_conv.c).

TEST INFRASTRUCTURE ONLY: the tests, the smoke check and the benchmark's
CPU-baseline leg may use this package; the GPU library never does, and this
package never imports the GPU library.

It computes the plain definition of the convolution that the ILP-M method
(Section 4, Algorithm 2) reorders, in float64 with exact products: see the
header of oracle_conv.c.  The acceptance rule for a float32 result r of the
GPU path is, element by element,

    |r - out| <= 1e-4 * (1 + S / (C_in * K * K))

with out the float64 value and S the sum of the absolute values of the
C_in*K*K products (the bias excluded; padding taps add 0 to S but still count
in the divisor).
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from typing import Optional

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
SOURCE = os.path.join(_HERE, "oracle_conv.c")
LIBRARY = os.path.join(_HERE, "liboracle.so")

_lib = None


def compile_oracle(source: str = SOURCE, output: str = LIBRARY, openmp: bool = True) -> str:
    """Build the oracle's shared library with gcc (-O2, OpenMP over output channels)."""
    cmd = ["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-Wall", "-Wextra"]
    if openmp:
        cmd.append("-fopenmp")
    tmp = output + ".tmp"
    cmd += [source, "-o", tmp, "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(tmp, output)
    return output


def _bind(lib):
    f32p = ctypes.POINTER(ctypes.c_float)
    f64p = ctypes.POINTER(ctypes.c_double)
    i64p = ctypes.POINTER(ctypes.c_int64)
    c_int = ctypes.c_int
    lib.oracle_out_size.argtypes = [c_int, c_int, c_int, c_int]
    lib.oracle_out_size.restype = c_int
    lib.oracle_set_threads.argtypes = [c_int]
    lib.oracle_set_threads.restype = c_int
    lib.oracle_conv2d_f64.argtypes = [f32p, f32p, f32p] + [c_int] * 7 + [f64p, f64p]
    lib.oracle_conv2d_f64.restype = c_int
    lib.oracle_conv2d_f64_points.argtypes = ([f32p, f32p, f32p] + [c_int] * 7 +
                                             [i64p, ctypes.c_int64, f64p, f64p])
    lib.oracle_conv2d_f64_points.restype = c_int
    lib.oracle_relu_f32.argtypes = [f32p, f32p, ctypes.c_int64]
    lib.oracle_relu_f32.restype = None
    lib.oracle_maxpool2x2_f32.argtypes = [f32p, c_int, c_int, c_int, f32p]
    lib.oracle_maxpool2x2_f32.restype = None
    return lib


def load(path: Optional[str] = None):
    """The bound oracle library at ``path`` (default: the in-tree build, built if absent)."""
    global _lib
    if path is not None:
        return _bind(ctypes.CDLL(path))
    if _lib is None:
        if not os.path.exists(LIBRARY):
            compile_oracle()
        _lib = _bind(ctypes.CDLL(LIBRARY))
    return _lib


def _f32(a):
    return np.ascontiguousarray(a, dtype=np.float32)


def _ptr(a, t):
    return a.ctypes.data_as(ctypes.POINTER(t)) if a is not None else None


def set_threads(n: int, lib=None) -> int:
    return (lib or load()).oracle_set_threads(int(n))


def out_size(n: int, k: int, stride: int, pad: int, lib=None) -> int:
    return (lib or load()).oracle_out_size(n, k, stride, pad)


def conv2d_f64(x, w, b=None, stride: int = 1, pad: int = 0, lib=None):
    """(out, S): float64 arrays of shape [1, C_out, H_out, W_out].

    x: [1, C_in, H, W], w: [C_out, C_in, K, K], b: [C_out] or None (float32)."""
    lib = lib or load()
    x, w = _f32(x), _f32(w)
    b = _f32(b) if b is not None else None
    _, c_in, h, wd = x.shape
    c_out, c_in2, k, k2 = w.shape
    assert c_in == c_in2 and k == k2, "weight shape does not match the input"
    ho, wo = lib.oracle_out_size(h, k, stride, pad), lib.oracle_out_size(wd, k, stride, pad)
    out = np.empty((1, c_out, max(ho, 0), max(wo, 0)), dtype=np.float64)
    sab = np.empty_like(out)
    rc = lib.oracle_conv2d_f64(_ptr(x, ctypes.c_float), _ptr(w, ctypes.c_float),
                               _ptr(b, ctypes.c_float), c_in, h, wd, c_out, k, stride, pad,
                               _ptr(out, ctypes.c_double), _ptr(sab, ctypes.c_double))
    if rc != 0:
        raise ValueError("oracle: no output for this shape")
    return out, sab


def conv2d_f64_points(x, w, b, stride: int, pad: int, flat_idx, lib=None):
    """(out, S) at the flat indices ``flat_idx`` into [C_out, H_out, W_out]."""
    lib = lib or load()
    x, w = _f32(x), _f32(w)
    b = _f32(b) if b is not None else None
    _, c_in, h, wd = x.shape
    c_out, _, k, _ = w.shape
    idx = np.ascontiguousarray(flat_idx, dtype=np.int64)
    out = np.empty(idx.shape[0], dtype=np.float64)
    sab = np.empty_like(out)
    rc = lib.oracle_conv2d_f64_points(_ptr(x, ctypes.c_float), _ptr(w, ctypes.c_float),
                                      _ptr(b, ctypes.c_float), c_in, h, wd, c_out, k, stride,
                                      pad, _ptr(idx, ctypes.c_int64), idx.shape[0],
                                      _ptr(out, ctypes.c_double), _ptr(sab, ctypes.c_double))
    if rc != 0:
        raise ValueError("oracle: bad shape or index")
    return out, sab


def relu(x, lib=None):
    lib = lib or load()
    x = _f32(x)
    y = np.empty_like(x)
    lib.oracle_relu_f32(_ptr(x, ctypes.c_float), _ptr(y, ctypes.c_float), x.size)
    return y


def maxpool2x2(x, lib=None):
    """x: [1, C, H, W] -> [1, C, H//2, W//2]."""
    lib = lib or load()
    x = _f32(x)
    _, c, h, w = x.shape
    y = np.empty((1, c, h // 2, w // 2), dtype=np.float32)
    lib.oracle_maxpool2x2_f32(_ptr(x, ctypes.c_float), c, h, w, _ptr(y, ctypes.c_float))
    return y


def tolerance(sumabs, c_in: int, k: int):
    """Per-element bound 1e-4 * (1 + S / (C_in*K*K))."""
    return 1e-4 * (1.0 + np.asarray(sumabs, dtype=np.float64) / float(c_in * k * k))


def check(result, ref, sumabs, c_in: int, k: int):
    """(ok, worst ratio |result-ref|/bound, index of the worst element)."""
    r = np.asarray(result, dtype=np.float64).reshape(-1)
    ref = np.asarray(ref, dtype=np.float64).reshape(-1)
    tol = tolerance(sumabs, c_in, k).reshape(-1)
    if r.shape != ref.shape:
        raise ValueError(f"shape mismatch {r.shape} vs {ref.shape}")
    if r.size == 0:
        return True, 0.0, -1
    ratio = np.abs(r - ref) / tol
    bad = ~np.isfinite(ratio)
    if bad.any():
        i = int(np.argmax(bad))
        return False, float("inf"), i
    i = int(np.argmax(ratio))
    return bool(ratio[i] <= 1.0), float(ratio[i]), i
