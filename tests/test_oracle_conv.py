"""Pins of the fp64 convolution oracle against things other than itself.

* torch.nn.functional.conv2d in float64 on the CPU (an independent library
  implementation), and its autograd for the two gradients;
* a closed form: all-ones input and kernel count the in-bounds taps;
* an explicitly zero-padded sliding-window evaluation (padding materialised
  instead of bounds-checked);
* 1x1 stride-1 conv == GEMM (numpy matmul);
* delta kernel == identity, off-centre delta == shift with zero fill;
* stride 2 == stride 1 subsampled;
* adjoint identities <conv(x,W),dy> = <x,dgrad(dy,W)> = <W,wgrad(x,dy)>;
* sampled evaluation == full evaluation.
"""
import itertools

import numpy as np
import pytest
import torch

import oracle
from oracle import ConvShape

SHAPES = [
    ConvShape(2, 7, 5, 3, 4, 3, 3, 2, 2, 1, 1),
    ConvShape(1, 6, 6, 8, 5, 3, 3, 1, 1, 1, 1),
    ConvShape(2, 9, 8, 4, 3, 3, 3, 2, 2, 1, 1),
    ConvShape(1, 5, 7, 6, 2, 1, 1, 1, 1, 0, 0),
    ConvShape(2, 8, 8, 3, 4, 5, 5, 2, 2, 2, 2),
    ConvShape(1, 6, 7, 2, 3, 3, 3, 1, 2, 0, 1),
    ConvShape(1, 4, 4, 2, 2, 3, 3, 3, 3, 1, 1),
]


def rng(seed):
    return np.random.default_rng(seed)


def torch_conv(x, w, s: ConvShape):
    xt = torch.from_numpy(x).permute(0, 3, 1, 2)
    wt = torch.from_numpy(w).permute(0, 3, 1, 2)
    y = torch.nn.functional.conv2d(xt, wt, stride=(s.sh, s.sw), padding=(s.ph, s.pw))
    return y.permute(0, 2, 3, 1).numpy()


@pytest.mark.parametrize("s", SHAPES, ids=str)
def test_fwd_matches_torch_float64(s):
    r = rng(1)
    x, w = r.standard_normal(s.x_shape), r.standard_normal(s.w_shape)
    y = oracle.conv_fwd(x, w, s)
    assert y.shape == s.y_shape
    np.testing.assert_allclose(y, torch_conv(x, w, s), rtol=0, atol=1e-12)


@pytest.mark.parametrize("s", SHAPES, ids=str)
def test_grads_match_torch_autograd_float64(s):
    r = rng(2)
    x, w, dy = r.standard_normal(s.x_shape), r.standard_normal(s.w_shape), r.standard_normal(s.y_shape)
    xt = torch.from_numpy(x).permute(0, 3, 1, 2).requires_grad_()
    wt = torch.from_numpy(w).permute(0, 3, 1, 2).requires_grad_()
    yt = torch.nn.functional.conv2d(xt, wt, stride=(s.sh, s.sw), padding=(s.ph, s.pw))
    yt.backward(torch.from_numpy(dy).permute(0, 3, 1, 2))
    np.testing.assert_allclose(oracle.conv_dgrad(dy, w, s), xt.grad.permute(0, 2, 3, 1).numpy(), atol=1e-12)
    np.testing.assert_allclose(oracle.conv_wgrad(x, dy, s), wt.grad.permute(0, 2, 3, 1).numpy(), atol=1e-12)


def test_all_ones_counts_in_bounds_taps():
    s = ConvShape(1, 4, 5, 1, 1, 3, 3, 1, 1, 1, 1)
    y = oracle.conv_fwd(np.ones(s.x_shape), np.ones(s.w_shape), s)[0, :, :, 0]
    expect = np.array([[4, 6, 6, 6, 4], [6, 9, 9, 9, 6], [6, 9, 9, 9, 6], [4, 6, 6, 6, 4]], float)
    assert np.array_equal(y, expect)


@pytest.mark.parametrize("s", SHAPES, ids=str)
def test_fwd_matches_padded_sliding_window(s):
    r = rng(3)
    x, w = r.standard_normal(s.x_shape), r.standard_normal(s.w_shape)
    xp = np.zeros((s.n, s.h + 2 * s.ph + s.kh, s.w + 2 * s.pw + s.kw, s.ci))
    xp[:, s.ph:s.ph + s.h, s.pw:s.pw + s.w, :] = x
    y = np.zeros(s.y_shape)
    for p, q in itertools.product(range(s.ho), range(s.wo)):
        win = xp[:, p * s.sh:p * s.sh + s.kh, q * s.sw:q * s.sw + s.kw, :]  # [n, kh, kw, ci]
        y[:, p, q, :] = np.tensordot(win, w, axes=([1, 2, 3], [1, 2, 3]))
    np.testing.assert_allclose(oracle.conv_fwd(x, w, s), y, atol=1e-12)


def test_1x1_is_gemm():
    s = ConvShape(3, 5, 4, 16, 24, 1, 1)
    r = rng(4)
    x, w = r.standard_normal(s.x_shape), r.standard_normal(s.w_shape)
    ref = (x.reshape(-1, 16) @ w.reshape(24, 16).T).reshape(s.y_shape)
    np.testing.assert_allclose(oracle.conv_fwd(x, w, s), ref, atol=1e-12)
    dy = r.standard_normal(s.y_shape)
    np.testing.assert_allclose(oracle.conv_dgrad(dy, w, s).reshape(-1, 16), dy.reshape(-1, 24) @ w.reshape(24, 16),
                               atol=1e-12)
    np.testing.assert_allclose(oracle.conv_wgrad(x, dy, s).reshape(24, 16), dy.reshape(-1, 24).T @ x.reshape(-1, 16),
                               atol=1e-11)


def test_delta_kernel_identity_and_shift():
    s = ConvShape(2, 6, 7, 4, 4, 3, 3, 1, 1, 1, 1)
    x = rng(5).standard_normal(s.x_shape)
    w = np.zeros(s.w_shape)
    for c in range(4):
        w[c, 1, 1, c] = 1.0
    assert np.array_equal(oracle.conv_fwd(x, w, s), x)
    assert np.array_equal(oracle.conv_dgrad(x, w, s), x)
    # off-centre tap (r=0, s=2): y[p,q] = x[p-1, q+1], zero where that leaves the image
    w = np.zeros(s.w_shape)
    for c in range(4):
        w[c, 0, 2, c] = 1.0
    y = oracle.conv_fwd(x, w, s)
    expect = np.zeros_like(x)
    expect[:, 1:, :-1, :] = x[:, :-1, 1:, :]
    assert np.array_equal(y, expect)


def test_stride2_is_subsampled_stride1():
    s2 = ConvShape(2, 9, 8, 3, 5, 3, 3, 2, 2, 1, 1)
    s1 = ConvShape(2, 9, 8, 3, 5, 3, 3, 1, 1, 1, 1)
    r = rng(6)
    x, w = r.standard_normal(s2.x_shape), r.standard_normal(s2.w_shape)
    np.testing.assert_allclose(oracle.conv_fwd(x, w, s2), oracle.conv_fwd(x, w, s1)[:, ::2, ::2, :], atol=1e-12)


def test_linearity():
    s = SHAPES[0]
    r = rng(7)
    x1, x2, w = r.standard_normal(s.x_shape), r.standard_normal(s.x_shape), r.standard_normal(s.w_shape)
    np.testing.assert_allclose(oracle.conv_fwd(2 * x1 - 3 * x2, w, s),
                               2 * oracle.conv_fwd(x1, w, s) - 3 * oracle.conv_fwd(x2, w, s), atol=1e-11)


@pytest.mark.parametrize("s", SHAPES, ids=str)
def test_adjoint_identities(s):
    r = rng(8)
    x, w, dy = r.standard_normal(s.x_shape), r.standard_normal(s.w_shape), r.standard_normal(s.y_shape)
    a = np.sum(oracle.conv_fwd(x, w, s) * dy)
    b = np.sum(x * oracle.conv_dgrad(dy, w, s))
    c = np.sum(w * oracle.conv_wgrad(x, dy, s))
    assert abs(a - b) <= 1e-12 * max(1.0, abs(a)) * 10
    assert abs(a - c) <= 1e-12 * max(1.0, abs(a)) * 10


@pytest.mark.parametrize("s", SHAPES[:3], ids=str)
def test_sampled_equals_full(s):
    r = rng(9)
    x, w, dy = r.standard_normal(s.x_shape), r.standard_normal(s.w_shape), r.standard_normal(s.y_shape)
    y, dx, dw = oracle.conv_fwd(x, w, s), oracle.conv_dgrad(dy, w, s), oracle.conv_wgrad(x, dy, s)
    for full, fn, a, b in ((y, oracle.conv_fwd_sample, x, w), (dx, oracle.conv_dgrad_sample, dy, w),
                           (dw, oracle.conv_wgrad_sample, x, dy)):
        idx = r.integers(0, full.size, 50)
        assert np.array_equal(fn(a, b, s, idx), full.reshape(-1)[idx])
    for o in range(s.co):
        assert np.array_equal(oracle.conv_fwd_channel(x, w, s, o), y[..., o].reshape(-1))
