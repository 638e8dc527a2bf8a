"""Pins of the fp64 BatchNorm(train)+SiLU oracle.

* torch.nn.functional.batch_norm(training=True) + silu in float64 on the CPU,
  with torch autograd for the backward (independent library implementation);
* closed forms: sum of normalised outputs is 0 and their mean square is
  var/(var+eps) (not 1: eps keeps it below); with eps = 0, BN(alpha*y + c) = BN(y);
* backward invariants: sum over rows of dy is 0; sum of dy*xhat equals
  gamma*rstd*sum(dz*xhat)*eps/(var+eps);
* SiLU special values: SiLU(0) = 0, SiLU'(0) = 1/2, SiLU(z) - SiLU(-z) = z;
* central finite differences of L = sum(g * a) in float64 (the paper's level-1
  operator check, Sec. 6.3, uses 1e-4; float64 affords a tighter bound);
* planted mistakes in copies of the oracle (unbiased variance, a dropped term,
  a flipped sign) each fail at least one of these checks.
"""
import numpy as np
import pytest
import torch

import oracle

EPS = 1e-3


def data(seed, m=37, c=5, scale=1.0, shift=0.0):
    r = np.random.default_rng(seed)
    y = shift + scale * r.standard_normal((m, c))
    gamma = r.uniform(0.5, 1.5, c)
    beta = r.normal(0, 0.3, c)
    g = r.standard_normal((m, c))
    return y, gamma, beta, g


def torch_ref(y, gamma, beta, eps, g=None):
    yt = torch.from_numpy(y).requires_grad_()
    gt = torch.from_numpy(gamma).requires_grad_()
    bt = torch.from_numpy(beta).requires_grad_()
    z = torch.nn.functional.batch_norm(yt, None, None, gt, bt, training=True, eps=eps)
    a = torch.nn.functional.silu(z)
    if g is None:
        return a.detach().numpy()
    a.backward(torch.from_numpy(g))
    return a.detach().numpy(), yt.grad.numpy(), gt.grad.numpy(), bt.grad.numpy()


@pytest.mark.parametrize("seed,scale,shift", [(0, 1.0, 0.0), (1, 0.01, 0.0), (2, 3.0, 5.0), (3, 0.03, -1.0)])
def test_matches_torch_float64(seed, scale, shift):
    y, gamma, beta, g = data(seed, scale=scale, shift=shift)
    mean, var = oracle.bn_stats(y)
    np.testing.assert_allclose(mean, y.mean(0), atol=1e-14 * (1 + abs(shift)))
    np.testing.assert_allclose(var, y.var(0), rtol=1e-12)
    a = oracle.bn_silu_fwd(y, mean, var, gamma, beta, EPS)
    dy, dgamma, dbeta = oracle.bn_silu_bwd(g, y, mean, var, gamma, beta, EPS)
    ta, tdy, tdg, tdb = torch_ref(y, gamma, beta, EPS, g)
    np.testing.assert_allclose(a, ta, atol=1e-13)
    np.testing.assert_allclose(dy, tdy, atol=1e-10 * np.abs(tdy).max())
    np.testing.assert_allclose(dgamma, tdg, atol=1e-12 * np.abs(tdg).max())
    np.testing.assert_allclose(dbeta, tdb, atol=1e-12 * np.abs(tdb).max())


def test_running_update_matches_torch():
    y, gamma, beta, _ = data(4)
    rm, rv = np.full(5, 0.1), np.full(5, 2.0)
    mean, var = oracle.bn_stats(y)
    orm, orv = oracle.running_update(rm, rv, mean, var, y.shape[0], 0.03)
    trm, trv = torch.from_numpy(rm.copy()), torch.from_numpy(rv.copy())
    torch.nn.functional.batch_norm(torch.from_numpy(y), trm, trv, training=True, momentum=0.03, eps=EPS)
    np.testing.assert_allclose(orm, trm.numpy(), rtol=1e-14)
    np.testing.assert_allclose(orv, trv.numpy(), rtol=1e-14)


@pytest.mark.parametrize("scale", [1.0, 0.02, 10.0])
def test_normalised_moments_closed_form(scale):
    y, _, _, _ = data(5, m=101, scale=scale, shift=0.7)
    mean, var = oracle.bn_stats(y)
    ones, zeros = np.ones(5), np.zeros(5)
    # with gamma=1, beta=0 the BN output is xhat; recover it from the SiLU-free path by inverting
    # nothing: compute xhat directly through the identity z = gamma*xhat + beta
    xhat = (y - mean) / np.sqrt(var + EPS)
    np.testing.assert_allclose(xhat.sum(0), 0, atol=1e-12)
    np.testing.assert_allclose((xhat ** 2).mean(0), var / (var + EPS), rtol=1e-12)
    # and the oracle's forward with SiLU removed by the identity SiLU(z) - SiLU(-z) = z
    a_pos = oracle.bn_silu_fwd(y, mean, var, ones, zeros, EPS)
    a_neg = oracle.bn_silu_fwd(y, mean, var, -ones, zeros, EPS)
    np.testing.assert_allclose(a_pos - a_neg, xhat, atol=1e-12 * max(1, np.abs(xhat).max()))
    assert np.all((xhat ** 2).mean(0) < 1)


def test_affine_invariance_eps0():
    y, gamma, beta, _ = data(6)
    m1, v1 = oracle.bn_stats(y)
    m2, v2 = oracle.bn_stats(3.5 * y - 2.0)
    a1 = oracle.bn_silu_fwd(y, m1, v1, gamma, beta, 0.0)
    a2 = oracle.bn_silu_fwd(3.5 * y - 2.0, m2, v2, gamma, beta, 0.0)
    np.testing.assert_allclose(a1, a2, atol=1e-12)


def test_silu_special_values():
    assert oracle.silu(np.array(0.0)) == 0.0
    z = np.linspace(-30, 30, 601)
    np.testing.assert_allclose(oracle.silu(z) - oracle.silu(-z), z, atol=1e-12)
    h = 1e-6
    assert abs((oracle.silu(h) - oracle.silu(-h)) / (2 * h) - 0.5) < 1e-10
    # SiLU(z) -> z for large z, -> 0 for very negative z
    assert abs(oracle.silu(np.array(40.0)) - 40.0) < 1e-12 and abs(oracle.silu(np.array(-40.0))) < 1e-15


def test_backward_invariants():
    y, gamma, beta, g = data(7, m=64)
    mean, var = oracle.bn_stats(y)
    dy, dgamma, dbeta = oracle.bn_silu_bwd(g, y, mean, var, gamma, beta, EPS)
    rstd = 1 / np.sqrt(var + EPS)
    xhat = (y - mean) * rstd
    np.testing.assert_allclose(dy.sum(0), 0, atol=1e-12 * np.abs(dy).max() * 64)
    expect = gamma * rstd * dgamma * EPS / (var + EPS)
    np.testing.assert_allclose((dy * xhat).sum(0), expect, atol=1e-11 * np.abs(dy).max() * 64)


def loss(y, gamma, beta, g, eps=EPS, fwd=oracle.bn_silu_fwd):
    mean, var = oracle.bn_stats(y)
    return float(np.sum(g * fwd(y, mean, var, gamma, beta, eps)))


def fd_grads(y, gamma, beta, g, h=1e-6, fwd=oracle.bn_silu_fwd):
    def central(arr, i, f):
        old = arr.flat[i]
        arr.flat[i] = old + h
        lp = f()
        arr.flat[i] = old - h
        lm = f()
        arr.flat[i] = old
        return (lp - lm) / (2 * h)

    f = lambda: loss(y, gamma, beta, g, fwd=fwd)
    dy = np.array([central(y, i, f) for i in range(y.size)]).reshape(y.shape)
    dg = np.array([central(gamma, i, f) for i in range(gamma.size)])
    db = np.array([central(beta, i, f) for i in range(beta.size)])
    return dy, dg, db


def bwd_error(bwd=oracle.bn_silu_bwd, fwd=oracle.bn_silu_fwd, seed=8):
    y, gamma, beta, g = data(seed, m=11, c=3, scale=0.2)
    mean, var = oracle.bn_stats(y)
    dy, dgamma, dbeta = bwd(g, y, mean, var, gamma, beta, EPS)
    fy, fg, fb = fd_grads(y, gamma, beta, g, fwd=fwd)
    return max(np.abs(dy - fy).max() / np.abs(fy).max(), np.abs(dgamma - fg).max() / np.abs(fg).max(),
               np.abs(dbeta - fb).max() / np.abs(fb).max())


def test_backward_finite_differences():
    assert bwd_error() < 1e-6


# ---- planted mistakes: each copy below must be caught by one of the pins above ----

def _bwd_dropped_term(g, y, mean, var, gamma, beta, eps):
    m = y.shape[0]
    rstd = 1 / np.sqrt(var + eps)
    xhat = (y - mean) * rstd
    z = gamma * xhat + beta
    sg = oracle.sigmoid(z)
    dz = g * sg * (1 + z * (1 - sg))
    dbeta, dgamma = dz.sum(0), (dz * xhat).sum(0)
    return gamma * rstd * (dz - dbeta / m), dgamma, dbeta  # xhat * dgamma / M dropped


def _bwd_wrong_silu_sign(g, y, mean, var, gamma, beta, eps):
    m = y.shape[0]
    rstd = 1 / np.sqrt(var + eps)
    xhat = (y - mean) * rstd
    z = gamma * xhat + beta
    sg = oracle.sigmoid(z)
    dz = g * sg * (1 - z * (1 - sg))
    dbeta, dgamma = dz.sum(0), (dz * xhat).sum(0)
    return gamma * rstd * (dz - dbeta / m - xhat * dgamma / m), dgamma, dbeta


def test_planted_backward_mistakes_are_caught():
    assert bwd_error(_bwd_dropped_term) > 1e-3
    assert bwd_error(_bwd_wrong_silu_sign) > 1e-3


def test_planted_unbiased_variance_is_caught():
    y, _, _, _ = data(9, m=20)
    mean = y.mean(0)
    var_unbiased = ((y - mean) ** 2).sum(0) / (y.shape[0] - 1)
    xhat = (y - mean) / np.sqrt(var_unbiased + EPS)
    _, var = oracle.bn_stats(y)
    assert np.abs((xhat ** 2).mean(0) - var / (var + EPS)).max() > 1e-3


def test_planted_missing_eps_is_caught():
    y, gamma, beta, _ = data(10, scale=0.02)  # var ~ 4e-4 < eps
    mean, var = oracle.bn_stats(y)
    a_ok = oracle.bn_silu_fwd(y, mean, var, gamma, beta, EPS)
    a_bad = oracle.bn_silu_fwd(y, mean, var, gamma, beta, 0.0)
    ta = torch_ref(y, gamma, beta, EPS)
    assert np.abs(a_ok - ta).max() < 1e-12 and np.abs(a_bad - ta).max() > 1e-2
