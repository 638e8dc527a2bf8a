"""Thin Python binding of the C ABI in ``include/numbat_conv.h`` (argument marshalling only).

Every function here has the name of the C entry point it calls and does nothing but
turn Python arguments into C arguments: tensors become device pointers (their
``data_ptr()``), ``None`` becomes NULL, the stream defaults to PyTorch's current
stream.  All computation happens in the gfx950 kernels of ``libnumbat_conv.so``;
there is no fallback: if the library is missing, importing it raises.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

HERE = os.path.dirname(os.path.abspath(__file__))
# the in-tree build; NUMBAT_LIB names another build of the same library (a tuning build)
LIB_PATH = os.environ.get("NUMBAT_LIB") or os.path.join(HERE, "libnumbat_conv.so")

NUMBAT_ABI_VERSION = 1

OK, ERR_NULL, ERR_BAD_DESC, ERR_UNSUPPORTED, ERR_ALIGN, ERR_WORKSPACE, ERR_DEVICE, ERR_VERSION = range(8)
(OP_CONV_FWD, OP_CONV_BWD_DATA, OP_CONV_BWD_WEIGHT, OP_BN_SILU_FWD, OP_BN_SILU_BWD, OP_CLIP_SGD_NESTEROV,
 OP_CONV_BWD_DATA_BN_SILU) = range(7)

EXPORTED = (
    "numbat_abi_version", "numbat_last_error", "numbat_status_string", "numbat_conv_output_shape",
    "numbat_workspace_size", "numbat_conv_fwd", "numbat_conv_bwd_data", "numbat_conv_bwd_weight",
    "numbat_bn_silu_fwd", "numbat_bn_silu_bwd", "numbat_kernel_class_count", "numbat_kernel_class_name",
    "numbat_timing_enable", "numbat_timing_read", "numbat_conv_fwd_noalloc", "numbat_clip_sgd_nesterov",
    "numbat_conv_fwd_bias", "numbat_conv_bn_silu_infer", "numbat_bn_silu_infer",
    "numbat_maxpool5_fwd", "numbat_maxpool5_bwd", "numbat_upsample2x_fwd", "numbat_upsample2x_bwd",
    "numbat_conv_fwd_bn_silu_prologue", "numbat_conv_bwd_data_bn_silu_prologue",
)


class numbat_conv_problem(ctypes.Structure):
    _fields_ = [("struct_size", ctypes.c_uint32)] + [
        (f, ctypes.c_int32)
        for f in ("n", "h", "w", "c_in", "c_out", "kh", "kw", "stride_h", "stride_w", "pad_h", "pad_w")
    ] + [("x_pixel_stride", ctypes.c_int64), ("y_pixel_stride", ctypes.c_int64)]


class numbat_bn_problem(ctypes.Structure):
    _fields_ = [
        ("struct_size", ctypes.c_uint32), ("c", ctypes.c_int32), ("m", ctypes.c_int64), ("eps", ctypes.c_float),
        ("momentum", ctypes.c_float), ("y_pixel_stride", ctypes.c_int64), ("a_pixel_stride", ctypes.c_int64),
        ("r_pixel_stride", ctypes.c_int64), ("dy_pixel_stride", ctypes.c_int64),
    ]


class numbat_pool_problem(ctypes.Structure):
    _fields_ = [("struct_size", ctypes.c_uint32), ("n", ctypes.c_int32), ("h", ctypes.c_int32),
                ("w", ctypes.c_int32), ("c", ctypes.c_int32), ("x_pixel_stride", ctypes.c_int64),
                ("y_pixel_stride", ctypes.c_int64)]


class numbat_param_tensor(ctypes.Structure):
    _fields_ = [("w", ctypes.c_void_p), ("grad", ctypes.c_void_p), ("momentum", ctypes.c_void_p),
                ("n", ctypes.c_int64), ("group", ctypes.c_int32), ("reserved", ctypes.c_int32)]


class numbat_sgd_group(ctypes.Structure):
    _fields_ = [("lr", ctypes.c_float), ("weight_decay", ctypes.c_float)]


class NumbatError(RuntimeError):
    def __init__(self, status: int, name: str, detail: str, call: str):
        super().__init__(f"{call}: {name}: {detail}")
        self.status = status
        self.detail = detail


_lib = None


def load() -> ctypes.CDLL:
    """Load the HIP library.  Raises if it has not been built (no fallback path exists)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is missing: build it with __graft_entry__.build() "
                              "(python -m paper_2609_10632_amd.build); there is no non-HIP fallback")
        lib = ctypes.CDLL(LIB_PATH)
        P, S = ctypes.c_void_p, ctypes.c_size_t
        CP, BP = ctypes.POINTER(numbat_conv_problem), ctypes.POINTER(numbat_bn_problem)
        PP = ctypes.POINTER(numbat_pool_problem)
        sig = {
            "numbat_abi_version": (ctypes.c_uint32, []),
            "numbat_last_error": (ctypes.c_char_p, []),
            "numbat_status_string": (ctypes.c_char_p, [ctypes.c_int]),
            "numbat_conv_output_shape": (ctypes.c_int, [CP, ctypes.POINTER(ctypes.c_int32),
                                                         ctypes.POINTER(ctypes.c_int32)]),
            "numbat_workspace_size": (ctypes.c_int, [ctypes.c_int, P, ctypes.POINTER(S)]),
            "numbat_conv_fwd": (ctypes.c_int, [CP, P, P, P, P, P, S, P]),
            "numbat_conv_fwd_bn_silu_prologue": (ctypes.c_int, [CP, P, P, P, P, ctypes.c_float, P, P, P, P, S, P]),
            "numbat_conv_fwd_noalloc": (ctypes.c_int, [CP, P, P, P, P, P]),
            "numbat_conv_fwd_bias": (ctypes.c_int, [CP, P, P, P, P, P]),
            "numbat_conv_bn_silu_infer": (ctypes.c_int, [CP, P, P, P, P, P, P, ctypes.c_float, P, P]),
            "numbat_bn_silu_infer": (ctypes.c_int, [BP, P, P, P, P, P, P, P, P]),
            "numbat_maxpool5_fwd": (ctypes.c_int, [PP, P, P, P, P]),
            "numbat_maxpool5_bwd": (ctypes.c_int, [PP, P, P, P, ctypes.c_int, P]),
            "numbat_upsample2x_fwd": (ctypes.c_int, [PP, P, P, P]),
            "numbat_upsample2x_bwd": (ctypes.c_int, [PP, P, P, ctypes.c_int, P]),
            "numbat_clip_sgd_nesterov": (ctypes.c_int, [P, ctypes.c_int32, ctypes.POINTER(numbat_sgd_group),
                                                         ctypes.c_int32, ctypes.c_float, ctypes.c_float, P, P, S, P]),
            "numbat_conv_bwd_data": (ctypes.c_int, [CP, P, P, P, ctypes.c_int, P, S, P]),
            "numbat_conv_bwd_data_bn_silu_prologue": (ctypes.c_int, [CP, P, ctypes.c_int64, P, P, P, P, P, P, P, P, P,
                                                                     P, ctypes.c_int, P]),
            "numbat_conv_bwd_weight": (ctypes.c_int, [CP, P, P, P, ctypes.c_int, P, S, P]),
            "numbat_bn_silu_fwd": (ctypes.c_int, [BP, P, P, P, P, P, P, P, P, P, P, P, S, P]),
            "numbat_bn_silu_bwd": (ctypes.c_int, [BP, P, P, P, P, P, P, P, P, P, P, P, S, P]),
            "numbat_kernel_class_count": (ctypes.c_int, []),
            "numbat_kernel_class_name": (ctypes.c_char_p, [ctypes.c_int]),
            "numbat_timing_enable": (ctypes.c_int, [ctypes.c_int]),
            "numbat_timing_read": (ctypes.c_int, [ctypes.c_int, ctypes.POINTER(ctypes.c_double),
                                                   ctypes.POINTER(ctypes.c_int64)]),
        }
        for name, (res, args) in sig.items():
            fn = getattr(lib, name)
            fn.restype = res
            fn.argtypes = args
        _lib = lib
    return _lib


def _ptr(t) -> Optional[int]:
    if t is None:
        return None
    if isinstance(t, int):
        return t
    return t.data_ptr()


def _nbytes(t) -> int:
    if t is None:
        return 0
    if isinstance(t, int):
        raise TypeError("pass the workspace as a tensor, or as (pointer, size) through ws_bytes")
    return t.numel() * t.element_size()


def _stream(stream) -> Optional[int]:
    if stream is not None:
        return stream if isinstance(stream, int) else stream.cuda_stream
    import torch

    if not torch.cuda.is_available():
        return None  # NULL stream; only validation failures can happen without a GPU
    return torch.cuda.current_stream().cuda_stream


def _check(status: int, call: str) -> None:
    if status != OK:
        lib = load()
        raise NumbatError(status, lib.numbat_status_string(status).decode(), lib.numbat_last_error().decode(), call)


def conv_problem(n, h, w, c_in, c_out, kh, kw=None, stride=1, pad=None, x_pixel_stride=0, y_pixel_stride=0):
    kw = kh if kw is None else kw
    pad = kh // 2 if pad is None else pad
    return numbat_conv_problem(ctypes.sizeof(numbat_conv_problem), n, h, w, c_in, c_out, kh, kw, stride, stride, pad,
                               pad, x_pixel_stride, y_pixel_stride)


def bn_problem(m, c, eps=1e-3, momentum=0.03, y_pixel_stride=0, a_pixel_stride=0, r_pixel_stride=0,
               dy_pixel_stride=0):
    return numbat_bn_problem(ctypes.sizeof(numbat_bn_problem), c, m, eps, momentum, y_pixel_stride, a_pixel_stride,
                             r_pixel_stride, dy_pixel_stride)


def pool_problem(n, h, w, c, x_pixel_stride=0, y_pixel_stride=0):
    return numbat_pool_problem(ctypes.sizeof(numbat_pool_problem), n, h, w, c, x_pixel_stride, y_pixel_stride)


def numbat_maxpool5_fwd(p, x, y, idx=None, stream=None):
    _check(load().numbat_maxpool5_fwd(ctypes.byref(p), _ptr(x), _ptr(y), _ptr(idx), _stream(stream)),
           "numbat_maxpool5_fwd")


def numbat_maxpool5_bwd(p, dy, idx, dx, accumulate=False, stream=None):
    _check(load().numbat_maxpool5_bwd(ctypes.byref(p), _ptr(dy), _ptr(idx), _ptr(dx), int(bool(accumulate)),
                                      _stream(stream)),
           "numbat_maxpool5_bwd")


def numbat_upsample2x_fwd(p, x, y, stream=None):
    _check(load().numbat_upsample2x_fwd(ctypes.byref(p), _ptr(x), _ptr(y), _stream(stream)), "numbat_upsample2x_fwd")


def numbat_upsample2x_bwd(p, dy, dx, accumulate=False, stream=None):
    _check(load().numbat_upsample2x_bwd(ctypes.byref(p), _ptr(dy), _ptr(dx), int(bool(accumulate)), _stream(stream)),
           "numbat_upsample2x_bwd")


def numbat_abi_version() -> int:
    return int(load().numbat_abi_version())


def numbat_last_error() -> str:
    return load().numbat_last_error().decode()


def numbat_status_string(status: int) -> str:
    return load().numbat_status_string(status).decode()


def numbat_conv_output_shape(p: numbat_conv_problem):
    ho, wo = ctypes.c_int32(), ctypes.c_int32()
    _check(load().numbat_conv_output_shape(ctypes.byref(p), ctypes.byref(ho), ctypes.byref(wo)),
           "numbat_conv_output_shape")
    return ho.value, wo.value


def numbat_workspace_size(op: int, p) -> int:
    n = ctypes.c_size_t()
    _check(load().numbat_workspace_size(op, ctypes.cast(ctypes.pointer(p), ctypes.c_void_p), ctypes.byref(n)),
           "numbat_workspace_size")
    return n.value


def numbat_conv_fwd(p, x, w, y, batch_stats=None, ws=None, stream=None, ws_bytes=None):
    _check(load().numbat_conv_fwd(ctypes.byref(p), _ptr(x), _ptr(w), _ptr(y), _ptr(batch_stats), _ptr(ws),
                                  _nbytes(ws) if ws_bytes is None else ws_bytes, _stream(stream)),
           "numbat_conv_fwd")


def numbat_conv_fwd_bn_silu_prologue(p, y_prev, prev_stats, gamma, beta, eps, w, y, batch_stats=None, ws=None,
                                     stream=None, ws_bytes=None):
    _check(load().numbat_conv_fwd_bn_silu_prologue(ctypes.byref(p), _ptr(y_prev), _ptr(prev_stats), _ptr(gamma),
                                                   _ptr(beta), ctypes.c_float(eps), _ptr(w), _ptr(y),
                                                   _ptr(batch_stats), _ptr(ws),
                                                   _nbytes(ws) if ws_bytes is None else ws_bytes, _stream(stream)),
           "numbat_conv_fwd_bn_silu_prologue")


def numbat_conv_fwd_noalloc(p, x, w, y, batch_stats=None, stream=None):
    _check(load().numbat_conv_fwd_noalloc(ctypes.byref(p), _ptr(x), _ptr(w), _ptr(y), _ptr(batch_stats),
                                          _stream(stream)),
           "numbat_conv_fwd_noalloc")


def numbat_conv_fwd_bias(p, x, w, bias, y, stream=None):
    _check(load().numbat_conv_fwd_bias(ctypes.byref(p), _ptr(x), _ptr(w), _ptr(bias), _ptr(y), _stream(stream)),
           "numbat_conv_fwd_bias")


def numbat_conv_bn_silu_infer(p, x, w, gamma, beta, running_mean, running_var, eps, y, stream=None):
    _check(load().numbat_conv_bn_silu_infer(ctypes.byref(p), _ptr(x), _ptr(w), _ptr(gamma), _ptr(beta),
                                            _ptr(running_mean), _ptr(running_var), eps, _ptr(y), _stream(stream)),
           "numbat_conv_bn_silu_infer")


def numbat_bn_silu_infer(p, y, running_mean, running_var, gamma, beta, residual, out, stream=None):
    _check(load().numbat_bn_silu_infer(ctypes.byref(p), _ptr(y), _ptr(running_mean), _ptr(running_var), _ptr(gamma),
                                       _ptr(beta), _ptr(residual), _ptr(out), _stream(stream)),
           "numbat_bn_silu_infer")


def numbat_conv_bwd_data(p, dy, w, dx, accumulate=False, ws=None, stream=None, ws_bytes=None):
    _check(load().numbat_conv_bwd_data(ctypes.byref(p), _ptr(dy), _ptr(w), _ptr(dx), int(bool(accumulate)), _ptr(ws),
                                       _nbytes(ws) if ws_bytes is None else ws_bytes, _stream(stream)),
           "numbat_conv_bwd_data")


def numbat_conv_bwd_data_bn_silu_prologue(p, g, y, save_mean, save_rstd, gamma, beta, dgamma, dbeta, w, dx, dy,
                                          accumulate=False, g_pixel_stride=0, stream=None):
    _check(load().numbat_conv_bwd_data_bn_silu_prologue(ctypes.byref(p), _ptr(g), int(g_pixel_stride), _ptr(y),
                                                        _ptr(save_mean), _ptr(save_rstd), _ptr(gamma), _ptr(beta),
                                                        _ptr(dgamma), _ptr(dbeta), _ptr(w), _ptr(dx), _ptr(dy),
                                                        int(bool(accumulate)), _stream(stream)),
           "numbat_conv_bwd_data_bn_silu_prologue")


def numbat_conv_bwd_weight(p, x, dy, dw, accumulate=False, ws=None, stream=None, ws_bytes=None):
    _check(load().numbat_conv_bwd_weight(ctypes.byref(p), _ptr(x), _ptr(dy), _ptr(dw), int(bool(accumulate)),
                                         _ptr(ws), _nbytes(ws) if ws_bytes is None else ws_bytes, _stream(stream)),
           "numbat_conv_bwd_weight")


def numbat_bn_silu_fwd(p, y, batch_stats, gamma, beta, residual, out, save_mean, save_rstd, running_mean=None,
                       running_var=None, ws=None, stream=None, ws_bytes=None):
    _check(load().numbat_bn_silu_fwd(ctypes.byref(p), _ptr(y), _ptr(batch_stats), _ptr(gamma), _ptr(beta),
                                     _ptr(residual), _ptr(out), _ptr(save_mean), _ptr(save_rstd), _ptr(running_mean),
                                     _ptr(running_var), _ptr(ws), _nbytes(ws) if ws_bytes is None else ws_bytes,
                                     _stream(stream)),
           "numbat_bn_silu_fwd")


def numbat_bn_silu_bwd(p, g, y, save_mean, save_rstd, gamma, beta, dy, dgamma, dbeta, residual_grad=None, ws=None,
                       stream=None, ws_bytes=None):
    _check(load().numbat_bn_silu_bwd(ctypes.byref(p), _ptr(g), _ptr(y), _ptr(save_mean), _ptr(save_rstd), _ptr(gamma),
                                     _ptr(beta), _ptr(dy), _ptr(dgamma), _ptr(dbeta), _ptr(residual_grad), _ptr(ws),
                                     _nbytes(ws) if ws_bytes is None else ws_bytes, _stream(stream)),
           "numbat_bn_silu_bwd")


def param_table(entries):
    """numbat_param_tensor entries for (w, grad, momentum, group) tensor tuples, as bytes
    laid out like the C array (upload them to the device to pass as `tensors`)."""
    arr = (numbat_param_tensor * len(entries))()
    for e, (w, g, m, grp) in zip(arr, entries):
        e.w, e.grad, e.momentum, e.n, e.group, e.reserved = _ptr(w), _ptr(g), _ptr(m), w.numel(), grp, 0
    return bytes(arr)


def numbat_clip_sgd_nesterov(tensors, count, groups, momentum_factor, max_norm, total_norm=None, ws=None,
                             stream=None, ws_bytes=None):
    """tensors: device buffer holding `count` numbat_param_tensor entries; groups: list of
    (lr, weight_decay) pairs."""
    g = (numbat_sgd_group * len(groups))(*[numbat_sgd_group(lr, wd) for lr, wd in groups])
    _check(load().numbat_clip_sgd_nesterov(_ptr(tensors), count, g, len(groups), momentum_factor, max_norm,
                                           _ptr(total_norm), _ptr(ws), _nbytes(ws) if ws_bytes is None else ws_bytes,
                                           _stream(stream)),
           "numbat_clip_sgd_nesterov")


def numbat_kernel_class_count() -> int:
    return int(load().numbat_kernel_class_count())


def numbat_kernel_class_name(kernel_class: int) -> str:
    return load().numbat_kernel_class_name(kernel_class).decode()


def numbat_timing_enable(enable: bool) -> None:
    _check(load().numbat_timing_enable(int(bool(enable))), "numbat_timing_enable")


def numbat_timing_read(kernel_class: int):
    """(total milliseconds, launches) of one kernel class since timing was enabled."""
    t, n = ctypes.c_double(), ctypes.c_int64()
    _check(load().numbat_timing_read(kernel_class, ctypes.byref(t), ctypes.byref(n)), "numbat_timing_read")
    return t.value, n.value
