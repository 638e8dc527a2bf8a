"""Pins of the pooling / upsampling oracle: torch's max_pool2d and nearest interpolate in
float64 (values and, without ties, autograd gradients), brute force on a tiny input, the
first-maximum rule on hand-made ties, and the adjoint identity of upsampling."""
import numpy as np
import pytest

from oracle import pool

torch = pytest.importorskip("torch")
F = torch.nn.functional


def nchw(a):
    return torch.tensor(a, dtype=torch.float64).permute(0, 3, 1, 2)


def test_maxpool_matches_torch_values_and_gradients():
    rng = np.random.default_rng(0)
    x = rng.standard_normal((2, 9, 11, 5))  # continuous values: no ties
    dy = rng.standard_normal(x.shape)
    t = nchw(x).requires_grad_(True)
    yt = F.max_pool2d(t, 5, 1, 2)
    (yt * nchw(dy)).sum().backward()
    y, idx = pool.maxpool_fwd(x)
    assert np.array_equal(y, yt.detach().permute(0, 2, 3, 1).numpy())
    assert np.allclose(pool.maxpool_bwd(dy, idx), t.grad.permute(0, 2, 3, 1).numpy(), rtol=1e-14, atol=1e-14)


def test_maxpool_brute_force_and_first_max_ties():
    rng = np.random.default_rng(1)
    x = rng.integers(0, 3, (1, 6, 7, 2)).astype(np.float64)  # many ties
    y, idx = pool.maxpool_fwd(x)
    dy = rng.standard_normal(x.shape)
    dx = np.zeros_like(x)
    for p in range(6):
        for q in range(7):
            for c in range(2):
                best, at = -np.inf, None
                for r in range(5):          # row-major scan, first strict maximum wins
                    for s in range(5):
                        i, j = p + r - 2, q + s - 2
                        if 0 <= i < 6 and 0 <= j < 7 and x[0, i, j, c] > best:
                            best, at = x[0, i, j, c], (i, j, r * 5 + s)
                assert y[0, p, q, c] == best and idx[0, p, q, c] == at[2]
                dx[0, at[0], at[1], c] += dy[0, p, q, c]
    assert np.allclose(pool.maxpool_bwd(dy, idx), dx, rtol=1e-14, atol=1e-14)
    # a constant image: every window's first in-image pixel takes its gradient
    c0 = np.ones((1, 4, 4, 1))
    _, i0 = pool.maxpool_fwd(c0)
    g = pool.maxpool_bwd(np.ones_like(c0), i0)
    assert g[0, 0, 0, 0] == 9.0 and g[0, 3, 3, 0] == 0.0  # (0,0) is first for the 3x3 windows that hold it


def test_upsample_matches_torch_and_is_adjoint():
    rng = np.random.default_rng(2)
    x = rng.standard_normal((2, 5, 4, 3))
    y = pool.upsample2x_fwd(x)
    ref = F.interpolate(nchw(x), scale_factor=2, mode="nearest").permute(0, 2, 3, 1).numpy()
    assert np.array_equal(y, ref)
    dy = rng.standard_normal(y.shape)
    t = nchw(x).requires_grad_(True)
    (F.interpolate(t, scale_factor=2, mode="nearest") * nchw(dy)).sum().backward()
    dx = pool.upsample2x_bwd(dy)
    assert np.allclose(dx, t.grad.permute(0, 2, 3, 1).numpy(), rtol=1e-14, atol=1e-14)
    assert np.isclose(np.sum(y * dy), np.sum(x * dx), rtol=1e-13)
