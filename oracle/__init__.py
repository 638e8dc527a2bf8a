"""ORACLE -- test infrastructure only.

A plain, slow, obviously-correct CPU reference of the Conv2d + BatchNorm(train) +
SiLU block of the paper's case-study detector (Sec. 6.1), in float64.  Only
``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of ``bench.py``
may import it.  It shares no code with the HIP path; the only common module is
the seeded input generator, which holds none of the method's arithmetic.

Pieces and the passages they follow:
  * convolution (forward, data gradient, weight gradient): ``conv_ref.c``,
    the defining sums of a cross-correlation with zero padding and no bias
    (Sec. 3 (iv) reference-default semantics; Sec. 6.1 conv blocks);
  * batch normalisation in training mode with batch statistics, computed in
    full precision (Sec. 3.2 mixed precision: BN kept in F32; Table 1
    precision row; Table 2 divergence #2) -- textbook definition of Ioffe and
    Szegedy: biased variance for normalisation, unbiased for the running
    variance, eps inside the square root;
  * SiLU a = z * sigmoid(z) (Sec. 6.1, Elfwing et al.);
  * backward of BN+SiLU derived by the chain rule from those definitions.

Every function here takes and returns float64 numpy arrays.  Activations are
NHWC; a BN input of shape [..., C] is treated as M = prod(leading dims) rows.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from dataclasses import dataclass

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "conv_ref.c")
_LIB = os.path.join(_HERE, "libconv_ref.so")


def build(force: bool = True) -> str:
    """Compile the C part of the oracle (gcc, OpenMP, strict IEEE fp64)."""
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp"
        subprocess.check_call(
            ["gcc", "-O2", "-fopenmp", "-fno-fast-math", "-ffp-contract=off", "-shared", "-fPIC",
             "-std=c11", _SRC, "-o", tmp]
        )
        os.replace(tmp, _LIB)
    return _LIB


class _Dims(ctypes.Structure):
    _fields_ = [(f, ctypes.c_int32) for f in ("n", "h", "w", "ci", "co", "kh", "kw", "sh", "sw", "ph", "pw")]


_lib = None


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build(force=True)
        lib = ctypes.CDLL(_LIB)
        P = ctypes.c_void_p
        D = ctypes.POINTER(_Dims)
        for name in ("ref_conv_fwd", "ref_conv_dgrad", "ref_conv_wgrad"):
            getattr(lib, name).argtypes = [P, P, P, D]
        for name in ("ref_conv_fwd_sample", "ref_conv_dgrad_sample", "ref_conv_wgrad_sample"):
            getattr(lib, name).argtypes = [P, P, D, P, ctypes.c_int64, P]
        lib.ref_conv_fwd_channel.argtypes = [P, P, D, ctypes.c_int32, P]
        lib.ref_num_threads.restype = ctypes.c_int
        _lib = lib
    return _lib


def num_threads() -> int:
    """OpenMP threads the C oracle runs on."""
    return int(_load().ref_num_threads())


@dataclass(frozen=True)
class ConvShape:
    n: int
    h: int
    w: int
    ci: int
    co: int
    kh: int
    kw: int
    sh: int = 1
    sw: int = 1
    ph: int = 0
    pw: int = 0

    @property
    def ho(self) -> int:
        return (self.h + 2 * self.ph - self.kh) // self.sh + 1

    @property
    def wo(self) -> int:
        return (self.w + 2 * self.pw - self.kw) // self.sw + 1

    def dims(self) -> _Dims:
        return _Dims(self.n, self.h, self.w, self.ci, self.co, self.kh, self.kw, self.sh, self.sw,
                     self.ph, self.pw)

    @property
    def x_shape(self):
        return (self.n, self.h, self.w, self.ci)

    @property
    def w_shape(self):
        return (self.co, self.kh, self.kw, self.ci)

    @property
    def y_shape(self):
        return (self.n, self.ho, self.wo, self.co)


def _f64(a: np.ndarray, shape) -> np.ndarray:
    a = np.ascontiguousarray(a, dtype=np.float64)
    if a.shape != tuple(shape):
        raise ValueError(f"expected shape {tuple(shape)}, got {a.shape}")
    return a


def conv_fwd(x, w, s: ConvShape) -> np.ndarray:
    x, w = _f64(x, s.x_shape), _f64(w, s.w_shape)
    y = np.empty(s.y_shape, np.float64)
    d = s.dims()
    _load().ref_conv_fwd(x.ctypes.data, w.ctypes.data, y.ctypes.data, ctypes.byref(d))
    return y


def conv_dgrad(dy, w, s: ConvShape) -> np.ndarray:
    dy, w = _f64(dy, s.y_shape), _f64(w, s.w_shape)
    dx = np.empty(s.x_shape, np.float64)
    d = s.dims()
    _load().ref_conv_dgrad(dy.ctypes.data, w.ctypes.data, dx.ctypes.data, ctypes.byref(d))
    return dx


def conv_wgrad(x, dy, s: ConvShape) -> np.ndarray:
    x, dy = _f64(x, s.x_shape), _f64(dy, s.y_shape)
    dw = np.empty(s.w_shape, np.float64)
    d = s.dims()
    _load().ref_conv_wgrad(x.ctypes.data, dy.ctypes.data, dw.ctypes.data, ctypes.byref(d))
    return dw


def _sample(fn, a, b, s: ConvShape, idx) -> np.ndarray:
    idx = np.ascontiguousarray(idx, dtype=np.int64)
    out = np.empty(idx.size, np.float64)
    d = s.dims()
    fn(a.ctypes.data, b.ctypes.data, ctypes.byref(d), idx.ctypes.data, idx.size, out.ctypes.data)
    return out


def conv_fwd_sample(x, w, s: ConvShape, idx) -> np.ndarray:
    """y at flat indices ``idx`` of the [N,Ho,Wo,Co] output."""
    return _sample(_load().ref_conv_fwd_sample, _f64(x, s.x_shape), _f64(w, s.w_shape), s, idx)


def conv_dgrad_sample(dy, w, s: ConvShape, idx) -> np.ndarray:
    """dx at flat indices ``idx`` of the [N,H,W,Ci] input gradient."""
    return _sample(_load().ref_conv_dgrad_sample, _f64(dy, s.y_shape), _f64(w, s.w_shape), s, idx)


def conv_wgrad_sample(x, dy, s: ConvShape, idx) -> np.ndarray:
    """dw at flat indices ``idx`` of the [Co,kh,kw,Ci] weight gradient."""
    return _sample(_load().ref_conv_wgrad_sample, _f64(x, s.x_shape), _f64(dy, s.y_shape), s, idx)


def conv_fwd_channel(x, w, s: ConvShape, o: int) -> np.ndarray:
    """Output channel ``o`` of the forward over all N*Ho*Wo rows (flat)."""
    x, w = _f64(x, s.x_shape), _f64(w, s.w_shape)
    col = np.empty(s.n * s.ho * s.wo, np.float64)
    d = s.dims()
    _load().ref_conv_fwd_channel(x.ctypes.data, w.ctypes.data, ctypes.byref(d), o, col.ctypes.data)
    return col


# ---------------------------------------------------------------------------
# Batch normalisation (training mode) and SiLU, float64 numpy.


def _rows(a: np.ndarray) -> np.ndarray:
    a = np.asarray(a, dtype=np.float64)
    return a.reshape(-1, a.shape[-1])


def bn_stats(y):
    """Batch mean and biased variance per channel over all rows: two passes in float64."""
    y2 = _rows(y)
    m = y2.shape[0]
    mean = y2.sum(axis=0) / m
    var = ((y2 - mean) ** 2).sum(axis=0) / m
    return mean, var


def sigmoid(z):
    return 1.0 / (1.0 + np.exp(-z))


def silu(z):
    """SiLU(z) = z * sigmoid(z)."""
    return z * sigmoid(z)


def bn_silu_fwd(y, mean, var, gamma, beta, eps, residual=None):
    """a = SiLU(gamma * (y - mean) / sqrt(var + eps) + beta) [+ residual]; same shape as y."""
    y = np.asarray(y, dtype=np.float64)
    rstd = 1.0 / np.sqrt(np.asarray(var, np.float64) + eps)
    xhat = (y - mean) * rstd
    z = gamma * xhat + beta
    a = silu(z)
    if residual is not None:
        a = a + np.asarray(residual, np.float64)
    return a


def bn_silu_bwd(g, y, mean, var, gamma, beta, eps):
    """Gradients of L = sum(g * a) for a = bn_silu_fwd(y, batch stats of y, ...).

    dz = g * sigmoid(z) * (1 + z * (1 - sigmoid(z)))        (SiLU derivative)
    dbeta = sum_rows dz,  dgamma = sum_rows dz * xhat
    dy = gamma * rstd * (dz - dbeta / M - xhat * dgamma / M) (batch-statistics BN)
    Returns (dy, dgamma, dbeta).
    """
    y = np.asarray(y, dtype=np.float64)
    g = np.asarray(g, dtype=np.float64)
    m = _rows(y).shape[0]
    rstd = 1.0 / np.sqrt(np.asarray(var, np.float64) + eps)
    xhat = (y - mean) * rstd
    z = gamma * xhat + beta
    sg = sigmoid(z)
    dz = g * sg * (1.0 + z * (1.0 - sg))
    dbeta = _rows(dz).sum(axis=0)
    dgamma = _rows(dz * xhat).sum(axis=0)
    dy = gamma * rstd * (dz - dbeta / m - xhat * dgamma / m)
    return dy, dgamma, dbeta


def running_update(running_mean, running_var, mean, var, m: int, momentum: float):
    """running <- (1 - momentum) * running + momentum * batch; the variance term is unbiased."""
    rm = (1.0 - momentum) * np.asarray(running_mean, np.float64) + momentum * mean
    rv = (1.0 - momentum) * np.asarray(running_var, np.float64) + momentum * var * m / (m - 1)
    return rm, rv


# ---------------------------------------------------------------------------
# One Conv+BN+SiLU block, forward and backward, straight from the pieces above.


def block_fwd(x, w, s: ConvShape, gamma, beta, eps, residual=None):
    """Returns dict(y, mean, var, a) for a = SiLU(BN(conv(x, w))) [+ residual]."""
    y = conv_fwd(x, w, s)
    mean, var = bn_stats(y)
    a = bn_silu_fwd(y, mean, var, gamma, beta, eps, residual)
    return {"y": y, "mean": mean, "var": var, "a": a}


def block_bwd(g, x, w, s: ConvShape, fwd, gamma, beta, eps):
    """Returns dict(dy, dgamma, dbeta, dx, dw) for upstream gradient g of the block output."""
    dy, dgamma, dbeta = bn_silu_bwd(g, fwd["y"], fwd["mean"], fwd["var"], gamma, beta, eps)
    dx = conv_dgrad(dy, w, s)
    dw = conv_wgrad(x, dy, s)
    return {"dy": dy, "dgamma": dgamma, "dbeta": dbeta, "dx": dx, "dw": dw}


# ---------------------------------------------------------------------------
# Inference (evaluation) mode: BN with running statistics (Table 2 divergence #9: eval-mode
# BN for validation), and the bias of the detect head's 1x1 prediction convolutions
# (Sec. 6.1 decoupled head).


def conv_fwd_bias(x, w, bias, s: ConvShape) -> np.ndarray:
    """y = conv(x, w) + bias[o] on every output pixel."""
    return conv_fwd(x, w, s) + np.asarray(bias, np.float64)


def bn_silu_eval(y, running_mean, running_var, gamma, beta, eps, residual=None):
    """a = SiLU(gamma * (y - running_mean) / sqrt(running_var + eps) + beta) [+ residual]: the
    training-mode formula with the running statistics in place of the batch's."""
    return bn_silu_fwd(y, running_mean, running_var, gamma, beta, eps, residual)
