"""ORACLE -- test infrastructure only.  The glue between the detector's conv blocks
(Sec. 6.1: the SPPF block of the backbone and the PAN-FPN neck), float64 numpy, NHWC.

  * max pooling, 5x5 window, stride 1, padding 2 (SPPF runs it three times in a row):
    y[n,p,q,c] = max over the window's in-image pixels (padding is -inf, so it never wins);
    the backward sends dy to the FIRST maximum of the window in row-major order (ties are
    likely in bf16), the reference ecosystem's rule;
  * nearest-neighbour 2x upsampling: y[n,2i+a,2j+b,c] = x[n,i,j,c]; its backward sums each
    2x2 block of dy.
"""
from __future__ import annotations

import numpy as np


def maxpool_fwd(x, k=5, pad=2):
    """Returns (y, idx): y the window maxima, idx the row-major window position (0 .. k*k-1)
    of each window's first maximum."""
    x = np.asarray(x, np.float64)
    n, h, w, c = x.shape
    xp = np.full((n, h + 2 * pad, w + 2 * pad, c), -np.inf)
    xp[:, pad:pad + h, pad:pad + w, :] = x
    y = np.full(x.shape, -np.inf)
    idx = np.zeros(x.shape, np.int64)
    for r in range(k):
        for s in range(k):
            win = xp[:, r:r + h, s:s + w, :]
            better = win > y  # strictly greater: an earlier position keeps a tie
            y = np.where(better, win, y)
            idx = np.where(better, r * k + s, idx)
    return y, idx


def maxpool_bwd(dy, idx, k=5, pad=2):
    """dx[n,h,w,c] = sum of dy over the windows whose first maximum is pixel (h, w)."""
    dy = np.asarray(dy, np.float64)
    n, h, w, c = dy.shape
    dxp = np.zeros((n, h + 2 * pad, w + 2 * pad, c))
    for r in range(k):
        for s in range(k):
            dxp[:, r:r + h, s:s + w, :] += np.where(idx == r * k + s, dy, 0.0)
    return dxp[:, pad:pad + h, pad:pad + w, :]


def upsample2x_fwd(x):
    x = np.asarray(x, np.float64)
    return x.repeat(2, axis=1).repeat(2, axis=2)


def upsample2x_bwd(dy):
    dy = np.asarray(dy, np.float64)
    n, h2, w2, c = dy.shape
    return dy.reshape(n, h2 // 2, 2, w2 // 2, 2, c).sum(axis=(2, 4))
