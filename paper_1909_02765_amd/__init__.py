"""Batch-1 fp32 conv2d forward for AMD MI355X: Python binding of libilpm.so.

Argument marshalling only: every step of the convolution runs in the HIP
kernels behind the C ABI declared in include/ilpm.h.  PyTorch supplies device
memory and the current stream.  There is no fallback: if the library is not
built, importing the binding raises.

    import paper_1909_02765_amd as ilpm
    y = ilpm.conv2d(x, w, bias, stride=1, pad=1)   # x [1,C_in,H,W], w [C_out,C_in,K,K]
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass
from typing import Optional

PKG = os.path.dirname(os.path.abspath(__file__))
LIBRARY = os.path.join(PKG, "libilpm.so")

OK = 0
ERR_INVALID_ARG = -1
ERR_UNSUPPORTED = -2
ERR_WORKSPACE = -3
ERR_HIP = -4
ERR_ARCH = -5
SPLIT_SUM_FUSED = 0
SPLIT_SUM_KERNEL = 1
PATH_DIRECT = 0
PATH_IGEMM = 1
VARIANT_WEIGHTS_LDS = 1   # ilpm_variant_pipeline flags
VARIANT_PROGRESSIVE_FIRST = 2
VARIANT_CONSECUTIVE_CHANNELS = 4


class IlpmError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        msg = f"{where}: {status_str(status)} ({status})"
        if status == ERR_HIP:
            msg += f", hipError_t {lib.ilpm_last_hip_error()}"
        super().__init__(msg)


class ilpm_plan(ctypes.Structure):
    _fields_ = [("path", ctypes.c_int), ("variant", ctypes.c_int),
                ("tile_h", ctypes.c_int), ("tile_w", ctypes.c_int),
                ("co_tile", ctypes.c_int), ("ci_chunk", ctypes.c_int),
                ("splits", ctypes.c_int), ("grid", ctypes.c_int), ("block", ctypes.c_int),
                ("lds_bytes", ctypes.c_int), ("h_out", ctypes.c_int), ("w_out", ctypes.c_int),
                ("workspace_bytes", ctypes.c_size_t)]

    def as_dict(self):
        return {name: getattr(self, name) for name, _ in self._fields_}


if not os.path.exists(LIBRARY):
    raise ImportError(f"{LIBRARY} is not built: run `python paper_1909_02765_amd/build.py` "
                      "(or __graft_entry__.build()) first")

# PyTorch ships its own HIP runtime.  Load it first so that the library's
# dependency on libamdhip64.so.7 resolves to that same, already loaded runtime:
# one process must hold one HIP runtime, or the streams and device pointers
# torch hands over would belong to another runtime instance.
import torch  # noqa: E402,F401

lib = ctypes.CDLL(LIBRARY)


def _hip_runtimes_mapped():
    paths = set()
    try:
        with open("/proc/self/maps") as f:
            for line in f:
                if "libamdhip64" in line:
                    paths.add(os.path.realpath(line.split()[-1]))
    except OSError:
        pass
    return paths


if len(_hip_runtimes_mapped()) > 1:
    raise ImportError(f"two HIP runtimes are loaded in this process: {sorted(_hip_runtimes_mapped())}")

_vp = ctypes.c_void_p
_i = ctypes.c_int
_plan_p = ctypes.POINTER(ilpm_plan)
_SIGS = {
    "ilpm_conv2d_fwd": ([_vp, _vp, _vp] + [_i] * 7 + [_vp, _vp], _i),
    "ilpm_conv2d_fwd_plan": ([_vp, _vp, _vp] + [_i] * 7 + [_vp, _plan_p, _vp], _i),
    "ilpm_conv2d_fwd_noalloc": ([_vp, _vp, _vp] + [_i] * 7 + [_vp, _vp], _i),
    "ilpm_conv2d_workspace_size": ([_i] * 7 + [ctypes.POINTER(ctypes.c_size_t)], _i),
    "ilpm_set_workspace": ([_vp, ctypes.c_size_t, _vp], _i),
    "ilpm_set_split_sum": ([_i], _i),
    "ilpm_status_str": ([_i], ctypes.c_char_p),
    "ilpm_arch_supported": ([ctypes.c_char_p], _i),
    "ilpm_last_hip_error": ([], _i),
    "ilpm_conv2d_validate": ([_vp, _vp, _vp] + [_i] * 7 + [_vp], _i),
    "ilpm_conv2d_plan": ([_i] * 7 + [_plan_p], _i),
    "ilpm_conv2d_plan_prepacked": ([_i] * 7 + [_plan_p], _i),
    "ilpm_conv2d_plan_for": ([_i] * 9 + [_plan_p], _i),
    "ilpm_conv2d_plan_variant": ([_i] * 10 + [_plan_p], _i),
    "ilpm_num_variants": ([_i], _i),
    "ilpm_variant_name": ([_i, _i], ctypes.c_char_p),
    "ilpm_variant_info": ([_i, _i] + [ctypes.POINTER(_i)] * 5, _i),
    "ilpm_variant_pipeline": ([_i, _i] + [ctypes.POINTER(_i)] * 4, _i),
    "ilpm_conv2d_prepacked_size": ([_plan_p, _i, _i, _i, ctypes.POINTER(ctypes.c_size_t)], _i),
    "ilpm_conv2d_prepack_weights": ([_vp, _i, _i, _i, _plan_p, _vp, _vp], _i),
    "ilpm_conv2d_fwd_prepacked": ([_vp, _vp, _vp] + [_i] * 7 + [_plan_p, _vp, _vp], _i),
    "ilpm_conv2d_fwd_epilogue": ([_vp, _vp, _vp] + [_i] * 8 + [_plan_p, _vp, _vp], _i),
    "ilpm_conv2d_fwd_prepacked_epilogue": ([_vp, _vp, _vp] + [_i] * 8 + [_plan_p, _vp, _vp], _i),
    "ilpm_conv2d_epilogue_workspace_size": ([_i] * 8 + [_plan_p, ctypes.POINTER(ctypes.c_size_t)], _i),
    "ilpm_winograd_filter_size": ([_i, _i, ctypes.POINTER(ctypes.c_size_t)], _i),
    "ilpm_winograd_transform_filter": ([_vp, _i, _i, _vp, _vp], _i),
    "ilpm_conv2d_winograd_workspace_size": ([_i] * 5 + [ctypes.POINTER(ctypes.c_size_t)], _i),
    "ilpm_conv2d_fwd_winograd": ([_vp, _vp, _vp] + [_i] * 5 + [_vp, _vp], _i),
    "ilpm_relu_inplace": ([_vp, ctypes.c_int64, _vp], _i),
    "ilpm_maxpool2x2": ([_vp, _i, _i, _i, _vp, _vp], _i),
}
for _name, (_args, _res) in _SIGS.items():
    _f = getattr(lib, _name)
    _f.argtypes = _args
    _f.restype = _res


def status_str(status: int) -> str:
    return lib.ilpm_status_str(int(status)).decode()


def _check(rc: int, where: str):
    if rc != OK:
        raise IlpmError(rc, where)


def _torch():
    import torch
    return torch


def _stream_handle(stream=None):
    torch = _torch()
    s = stream if stream is not None else torch.cuda.current_stream()
    return ctypes.c_void_p(s.cuda_stream)


def _stream_obj(stream=None):
    return stream if stream is not None else _torch().cuda.current_stream()


def _dev_f32(t, name):
    torch = _torch()
    if not isinstance(t, torch.Tensor) or not t.is_cuda or t.dtype != torch.float32 or not t.is_contiguous():
        raise TypeError(f"{name} must be a contiguous float32 CUDA tensor")
    return ctypes.c_void_p(t.data_ptr())


def out_size(n: int, k: int, stride: int, pad: int) -> int:
    span = n + 2 * pad - k
    return span // stride + 1 if span >= 0 else 0


def plan(c_in, h, w, c_out, k, stride=1, pad=0) -> ilpm_plan:
    """The plan the library picks for this shape."""
    p = ilpm_plan()
    _check(lib.ilpm_conv2d_plan(c_in, h, w, c_out, k, stride, pad, ctypes.byref(p)), "ilpm_conv2d_plan")
    return p


def plan_prepacked(c_in, h, w, c_out, k, stride=1, pad=0) -> ilpm_plan:
    """The plan the library picks for this shape when the weights will be prepacked."""
    p = ilpm_plan()
    _check(lib.ilpm_conv2d_plan_prepacked(c_in, h, w, c_out, k, stride, pad, ctypes.byref(p)),
           "ilpm_conv2d_plan_prepacked")
    return p


def plan_for(c_in, h, w, c_out, k, stride=1, pad=0, epilogue=0, prepacked=False) -> ilpm_plan:
    """The plan the library picks for this shape, epilogue and weight layout."""
    p = ilpm_plan()
    _check(lib.ilpm_conv2d_plan_for(c_in, h, w, c_out, k, stride, pad, epilogue, 1 if prepacked else 0,
                                    ctypes.byref(p)), "ilpm_conv2d_plan_for")
    return p


def plan_variant(c_in, h, w, c_out, k, stride, pad, path, variant, splits=0) -> ilpm_plan:
    p = ilpm_plan()
    _check(lib.ilpm_conv2d_plan_variant(c_in, h, w, c_out, k, stride, pad, path, variant, splits,
                                        ctypes.byref(p)), "ilpm_conv2d_plan_variant")
    return p


def num_variants(path: int) -> int:
    return lib.ilpm_num_variants(path)


def variant_name(path: int, variant: int) -> str:
    n = lib.ilpm_variant_name(path, variant)
    if n is None:
        raise IlpmError(ERR_INVALID_ARG, "ilpm_variant_name")
    return n.decode()


def variant_info(path: int, variant: int):
    vals = [ctypes.c_int() for _ in range(5)]
    _check(lib.ilpm_variant_info(path, variant, *[ctypes.byref(v) for v in vals]), "ilpm_variant_info")
    k, s, th, tw, co = (v.value for v in vals)
    cc, ns, nb, fl = (ctypes.c_int() for _ in range(4))
    _check(lib.ilpm_variant_pipeline(path, variant, *(ctypes.byref(v) for v in (cc, ns, nb, fl))),
           "ilpm_variant_pipeline")
    return dict(k=k, stride=s, tile_h=th, tile_w=tw, co_tile=co, ci_chunk=cc.value, stages=ns.value,
                buffers=nb.value, weights_lds=bool(fl.value & VARIANT_WEIGHTS_LDS),
                progressive_first=bool(fl.value & VARIANT_PROGRESSIVE_FIRST),
                consecutive_channels=bool(fl.value & VARIANT_CONSECUTIVE_CHANNELS))


def workspace_size(c_in, h, w, c_out, k, stride=1, pad=0) -> int:
    n = ctypes.c_size_t()
    _check(lib.ilpm_conv2d_workspace_size(c_in, h, w, c_out, k, stride, pad, ctypes.byref(n)),
           "ilpm_conv2d_workspace_size")
    return n.value


def set_workspace(buf=None, stream=None):
    """Register a caller-owned device buffer (a CUDA tensor, 256-byte aligned) as
    the current device's workspace, or unregister it with None."""
    if buf is None:
        _check(lib.ilpm_set_workspace(None, 0, _stream_handle(stream)), "ilpm_set_workspace")
        return
    nbytes = buf.numel() * buf.element_size()
    _check(lib.ilpm_set_workspace(ctypes.c_void_p(buf.data_ptr()), nbytes, _stream_handle(stream)),
           "ilpm_set_workspace")


def set_split_sum(mode: int):
    """How split plans sum their partial outputs from now on: SPLIT_SUM_FUSED (the
    last workgroup of each output tile, the default) or SPLIT_SUM_KERNEL (a second
    kernel).  Both give bit-identical outputs."""
    _check(lib.ilpm_set_split_sum(int(mode)), "ilpm_set_split_sum")


def conv2d(x, w, bias=None, stride: int = 1, pad: int = 0, out=None, plan: Optional[ilpm_plan] = None,
           stream=None):
    """out[1, C_out, H_out, W_out] = conv2d(x, w) + bias on the current CUDA stream."""
    torch = _torch()
    if x.dim() != 4 or x.shape[0] != 1:
        raise ValueError("x must be [1, C_in, H, W]")
    if w.dim() != 4 or w.shape[2] != w.shape[3] or w.shape[1] != x.shape[1]:
        raise ValueError("w must be [C_out, C_in, K, K] with C_in matching x")
    _, c_in, h, wd = x.shape
    c_out, _, k, _ = w.shape
    if bias is not None and (bias.dim() != 1 or bias.shape[0] != c_out):
        raise ValueError("bias must be [C_out]")
    ho, wo = out_size(h, k, stride, pad), out_size(wd, k, stride, pad)
    if out is None:
        out = torch.empty((1, c_out, max(ho, 1), max(wo, 1)), device=x.device, dtype=torch.float32)
    elif tuple(out.shape) != (1, c_out, ho, wo):
        raise ValueError(f"out must be [1, {c_out}, {ho}, {wo}]")
    args = (_dev_f32(x, "x"), _dev_f32(w, "w"),
            _dev_f32(bias, "bias") if bias is not None else None,
            c_in, h, wd, c_out, k, stride, pad, _dev_f32(out, "out"))
    if plan is None:
        rc = lib.ilpm_conv2d_fwd(*args, _stream_handle(stream))
        _check(rc, "ilpm_conv2d_fwd")
    else:
        rc = lib.ilpm_conv2d_fwd_plan(*args, ctypes.byref(plan), _stream_handle(stream))
        _check(rc, "ilpm_conv2d_fwd_plan")
    return out


NOALLOC_SCRATCH_BYTES = 16 << 20  # ILPM_NOALLOC_SCRATCH_BYTES


def conv2d_noalloc(x, w, bias=None, stride: int = 1, pad: int = 0, *, out, stream=None):
    """conv2d through ilpm_conv2d_fwd_noalloc (no device allocation: split
    plans use the library's fixed per-device array).  `out` must be given."""
    if x.dim() != 4 or x.shape[0] != 1 or w.dim() != 4 or w.shape[2] != w.shape[3] or w.shape[1] != x.shape[1]:
        raise ValueError("x must be [1, C_in, H, W] and w [C_out, C_in, K, K]")
    _, c_in, h, wd = x.shape
    c_out, _, k, _ = w.shape
    if tuple(out.shape) != (1, c_out, out_size(h, k, stride, pad), out_size(wd, k, stride, pad)):
        raise ValueError("out has the wrong shape")
    _check(lib.ilpm_conv2d_fwd_noalloc(_dev_f32(x, "x"), _dev_f32(w, "w"),
                                       _dev_f32(bias, "bias") if bias is not None else None,
                                       c_in, h, wd, c_out, k, stride, pad, _dev_f32(out, "out"),
                                       _stream_handle(stream)), "ilpm_conv2d_fwd_noalloc")
    return out


class _Launcher:
    """A library entry point with its arguments marshalled once; `keep` holds
    the objects behind the raw addresses in `args` for the launcher's life."""

    __slots__ = ("fn", "args", "keep", "name")

    def __init__(self, fn, args, keep, name):
        self.fn, self.args, self.keep, self.name = fn, args, keep, name

    def __call__(self):
        rc = self.fn(*self.args)
        if rc != OK:
            raise IlpmError(rc, self.name)


def conv2d_launcher(x, w, bias, stride, pad, out, stream=None, plan: Optional[ilpm_plan] = None):
    """A zero-argument callable that enqueues the same conv2d again, with the
    arguments marshalled once (for timing loops and graph capture).

    The callable holds raw device addresses, so it keeps the tensors (and
    stream) they come from alive: a tensor freed while a launcher still
    points at it could be returned to the driver -- torch empties its cache
    when a graph capture begins -- and the next launch would then read
    unmapped memory.  The stream is the one current when the launcher is made.
    With `plan`, the calls run that plan (ilpm_conv2d_fwd_plan)."""
    _, c_in, h, wd = x.shape
    c_out, _, k, _ = w.shape
    if tuple(out.shape) != (1, c_out, out_size(h, k, stride, pad), out_size(wd, k, stride, pad)):
        raise ValueError("out has the wrong shape")
    if plan is not None:
        args = (_dev_f32(x, "x"), _dev_f32(w, "w"), _dev_f32(bias, "bias") if bias is not None else None,
                c_in, h, wd, c_out, k, stride, pad, _dev_f32(out, "out"), ctypes.byref(plan), _stream_handle(stream))
        return _Launcher(lib.ilpm_conv2d_fwd_plan, args, (x, w, bias, out, plan, _stream_obj(stream)),
                         "ilpm_conv2d_fwd_plan")
    args = (_dev_f32(x, "x"), _dev_f32(w, "w"), _dev_f32(bias, "bias") if bias is not None else None,
            c_in, h, wd, c_out, k, stride, pad, _dev_f32(out, "out"), _stream_handle(stream))
    return _Launcher(lib.ilpm_conv2d_fwd, args, (x, w, bias, out, _stream_obj(stream)), "ilpm_conv2d_fwd")


def prepacked_size(plan_: ilpm_plan, c_in: int, c_out: int, k: int) -> int:
    n = ctypes.c_size_t()
    _check(lib.ilpm_conv2d_prepacked_size(ctypes.byref(plan_), c_in, c_out, k, ctypes.byref(n)),
           "ilpm_conv2d_prepacked_size")
    return n.value


def prepack_weights(w, plan_: ilpm_plan, stream=None):
    """w [C_out, C_in, K, K] re-laid out for plan_'s kernel (a new flat CUDA
    tensor); pass it to conv2d_prepacked with the same plan."""
    torch = _torch()
    if w.dim() != 4 or w.shape[2] != w.shape[3]:
        raise ValueError("w must be [C_out, C_in, K, K]")
    c_out, c_in, k, _ = w.shape
    n = prepacked_size(plan_, c_in, c_out, k)
    packed = torch.empty(n // 4, device=w.device, dtype=torch.float32)
    _check(lib.ilpm_conv2d_prepack_weights(_dev_f32(w, "w"), c_in, c_out, k, ctypes.byref(plan_),
                                           _dev_f32(packed, "packed"), _stream_handle(stream)),
           "ilpm_conv2d_prepack_weights")
    return packed


def conv2d_prepacked(x, packed, c_out: int, k: int, bias=None, stride: int = 1, pad: int = 0, *,
                     plan: ilpm_plan, out=None, stream=None):
    """conv2d with weights from prepack_weights(w, plan)."""
    torch = _torch()
    if x.dim() != 4 or x.shape[0] != 1:
        raise ValueError("x must be [1, C_in, H, W]")
    _, c_in, h, wd = x.shape
    ho, wo = out_size(h, k, stride, pad), out_size(wd, k, stride, pad)
    if out is None:
        out = torch.empty((1, c_out, max(ho, 1), max(wo, 1)), device=x.device, dtype=torch.float32)
    elif tuple(out.shape) != (1, c_out, ho, wo):
        raise ValueError(f"out must be [1, {c_out}, {ho}, {wo}]")
    _check(lib.ilpm_conv2d_fwd_prepacked(_dev_f32(x, "x"), _dev_f32(packed, "packed"),
                                         _dev_f32(bias, "bias") if bias is not None else None,
                                         c_in, h, wd, c_out, k, stride, pad, ctypes.byref(plan),
                                         _dev_f32(out, "out"), _stream_handle(stream)),
           "ilpm_conv2d_fwd_prepacked")
    return out


def conv2d_prepacked_launcher(x, packed, c_out, k, bias, stride, pad, out, plan, stream=None):
    """conv2d_launcher for prepacked weights (it keeps the plan object alive too)."""
    _, c_in, h, wd = x.shape
    if tuple(out.shape) != (1, c_out, out_size(h, k, stride, pad), out_size(wd, k, stride, pad)):
        raise ValueError("out has the wrong shape")
    args = (_dev_f32(x, "x"), _dev_f32(packed, "packed"), _dev_f32(bias, "bias") if bias is not None else None,
            c_in, h, wd, c_out, k, stride, pad, ctypes.byref(plan), _dev_f32(out, "out"), _stream_handle(stream))
    return _Launcher(lib.ilpm_conv2d_fwd_prepacked, args, (x, packed, bias, out, plan, _stream_obj(stream)),
                     "ilpm_conv2d_fwd_prepacked")


EPI_RELU = 1
EPI_MAXPOOL2 = 2


def epilogue_out_shape(c_out, h, w, k, stride, pad, epilogue):
    ho, wo = out_size(h, k, stride, pad), out_size(w, k, stride, pad)
    if epilogue & EPI_MAXPOOL2:
        ho, wo = ho // 2, wo // 2
    return (1, c_out, ho, wo)


def epilogue_workspace_size(c_in, h, w, c_out, k, stride, pad, epilogue, plan_=None) -> int:
    n = ctypes.c_size_t()
    _check(lib.ilpm_conv2d_epilogue_workspace_size(c_in, h, w, c_out, k, stride, pad, epilogue,
                                                   ctypes.byref(plan_) if plan_ is not None else None,
                                                   ctypes.byref(n)), "ilpm_conv2d_epilogue_workspace_size")
    return n.value


def conv2d_epilogue(x, w, bias=None, stride: int = 1, pad: int = 0, epilogue: int = EPI_RELU, *,
                    plan: Optional[ilpm_plan] = None, out=None, stream=None):
    """conv2d (+ bias) followed by ReLU and/or a 2x2 max-pool (EPI_* bits)."""
    torch = _torch()
    _, c_in, h, wd = x.shape
    c_out, _, k, _ = w.shape
    shape = epilogue_out_shape(c_out, h, wd, k, stride, pad, epilogue)
    if out is None:
        out = torch.empty(tuple(max(d, 1) for d in shape), device=x.device, dtype=torch.float32)
    elif tuple(out.shape) != shape:
        raise ValueError(f"out must be {list(shape)}")
    _check(lib.ilpm_conv2d_fwd_epilogue(_dev_f32(x, "x"), _dev_f32(w, "w"),
                                        _dev_f32(bias, "bias") if bias is not None else None,
                                        c_in, h, wd, c_out, k, stride, pad, epilogue,
                                        ctypes.byref(plan) if plan is not None else None,
                                        _dev_f32(out, "out"), _stream_handle(stream)), "ilpm_conv2d_fwd_epilogue")
    return out


def conv2d_epilogue_launcher(x, w, bias, stride, pad, epilogue, out, stream=None):
    """conv2d_launcher for ilpm_conv2d_fwd_epilogue with the default plan."""
    _, c_in, h, wd = x.shape
    c_out, _, k, _ = w.shape
    if tuple(out.shape) != epilogue_out_shape(c_out, h, wd, k, stride, pad, epilogue):
        raise ValueError("out has the wrong shape")
    args = (_dev_f32(x, "x"), _dev_f32(w, "w"), _dev_f32(bias, "bias") if bias is not None else None,
            c_in, h, wd, c_out, k, stride, pad, epilogue, None, _dev_f32(out, "out"), _stream_handle(stream))
    return _Launcher(lib.ilpm_conv2d_fwd_epilogue, args, (x, w, bias, out, _stream_obj(stream)),
                     "ilpm_conv2d_fwd_epilogue")


def conv2d_prepacked_epilogue(x, packed, c_out: int, k: int, bias=None, stride: int = 1, pad: int = 0,
                              epilogue: int = EPI_RELU, *, plan: ilpm_plan, out=None, stream=None):
    """conv2d_epilogue with weights from prepack_weights(w, plan)."""
    torch = _torch()
    _, c_in, h, wd = x.shape
    shape = epilogue_out_shape(c_out, h, wd, k, stride, pad, epilogue)
    if out is None:
        out = torch.empty(tuple(max(d, 1) for d in shape), device=x.device, dtype=torch.float32)
    elif tuple(out.shape) != shape:
        raise ValueError(f"out must be {list(shape)}")
    _check(lib.ilpm_conv2d_fwd_prepacked_epilogue(_dev_f32(x, "x"), _dev_f32(packed, "packed"),
                                                  _dev_f32(bias, "bias") if bias is not None else None,
                                                  c_in, h, wd, c_out, k, stride, pad, epilogue, ctypes.byref(plan),
                                                  _dev_f32(out, "out"), _stream_handle(stream)),
           "ilpm_conv2d_fwd_prepacked_epilogue")
    return out


def conv2d_prepacked_epilogue_launcher(x, packed, c_out, k, bias, stride, pad, epilogue, out, plan, stream=None):
    """conv2d_launcher for ilpm_conv2d_fwd_prepacked_epilogue (it keeps the plan object alive too)."""
    _, c_in, h, wd = x.shape
    if tuple(out.shape) != epilogue_out_shape(c_out, h, wd, k, stride, pad, epilogue):
        raise ValueError("out has the wrong shape")
    args = (_dev_f32(x, "x"), _dev_f32(packed, "packed"), _dev_f32(bias, "bias") if bias is not None else None,
            c_in, h, wd, c_out, k, stride, pad, epilogue, ctypes.byref(plan), _dev_f32(out, "out"),
            _stream_handle(stream))
    return _Launcher(lib.ilpm_conv2d_fwd_prepacked_epilogue, args,
                     (x, packed, bias, out, plan, _stream_obj(stream)), "ilpm_conv2d_fwd_prepacked_epilogue")


def winograd_transform_filter(w, stream=None):
    """U = G g G^T of 3x3 weights [C_out, C_in, 3, 3] as a [16, C_out, C_in] CUDA tensor."""
    torch = _torch()
    if w.dim() != 4 or w.shape[2] != 3 or w.shape[3] != 3:
        raise ValueError("w must be [C_out, C_in, 3, 3]")
    c_out, c_in = w.shape[0], w.shape[1]
    u = torch.empty((16, c_out, c_in), device=w.device, dtype=torch.float32)
    _check(lib.ilpm_winograd_transform_filter(_dev_f32(w, "w"), c_in, c_out, _dev_f32(u, "u"),
                                              _stream_handle(stream)), "ilpm_winograd_transform_filter")
    return u


def conv2d_winograd(x, u, bias=None, pad: int = 1, out=None, stream=None):
    """3x3 / stride-1 conv2d by Winograd F(2x2,3x3) from transformed weights u [16, C_out, C_in]."""
    torch = _torch()
    _, c_in, h, wd = x.shape
    c_out = u.shape[1]
    ho, wo = out_size(h, 3, 1, pad), out_size(wd, 3, 1, pad)
    if out is None:
        out = torch.empty((1, c_out, max(ho, 1), max(wo, 1)), device=x.device, dtype=torch.float32)
    _check(lib.ilpm_conv2d_fwd_winograd(_dev_f32(x, "x"), _dev_f32(u, "u"),
                                        _dev_f32(bias, "bias") if bias is not None else None,
                                        c_in, h, wd, c_out, pad, _dev_f32(out, "out"), _stream_handle(stream)),
           "ilpm_conv2d_fwd_winograd")
    return out


def conv2d_winograd_launcher(x, u, bias, pad, out, stream=None):
    _, c_in, h, wd = x.shape
    c_out = u.shape[1]
    args = (_dev_f32(x, "x"), _dev_f32(u, "u"), _dev_f32(bias, "bias") if bias is not None else None,
            c_in, h, wd, c_out, pad, _dev_f32(out, "out"), _stream_handle(stream))
    return _Launcher(lib.ilpm_conv2d_fwd_winograd, args, (x, u, bias, out, _stream_obj(stream)),
                     "ilpm_conv2d_fwd_winograd")


def relu_(x, stream=None):
    _check(lib.ilpm_relu_inplace(_dev_f32(x, "x"), x.numel(), _stream_handle(stream)), "ilpm_relu_inplace")
    return x


def maxpool2x2(x, stream=None):
    torch = _torch()
    if x.dim() != 4 or x.shape[0] != 1:
        raise ValueError("x must be [1, C, H, W]")
    _, c, h, w = x.shape
    out = torch.empty((1, c, h // 2, w // 2), device=x.device, dtype=torch.float32)
    _check(lib.ilpm_maxpool2x2(_dev_f32(x, "x"), c, h, w, _dev_f32(out, "out"), _stream_handle(stream)),
           "ilpm_maxpool2x2")
    return out
