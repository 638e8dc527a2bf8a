"""Pins of the optimiser-step oracle (global-norm clip + SGD-Nesterov in parameter groups)
against the reference ecosystem's own implementation (torch's clip_grad_norm_ and SGD with
nesterov=True in float64, several steps so the momentum recurrence is exercised), closed
forms, and planted mistakes that a wrong oracle would make."""
import numpy as np
import pytest

from oracle import optim

torch = pytest.importorskip("torch")


def make(seed, shapes, scale=1.0):
    rng = np.random.default_rng(seed)
    return [rng.standard_normal(s) * scale for s in shapes]


SHAPES = [(48, 3, 3, 3), (48,), (48,), (96, 3, 3, 48), (96,), (96,), (64,), (80, 1, 1, 64)]
GROUPS = [0, 1, 2, 0, 1, 2, 2, 0]  # decayed weights, normalisation gains, biases
HP = [(0.01, 3.75e-4), (0.01, 0.0), (0.1, 0.0)]


@pytest.mark.parametrize("gscale", [0.01, 10.0])  # below and above the clip threshold
def test_matches_torch_clip_and_nesterov_sgd_over_steps(gscale):
    params = make(1, SHAPES)
    bufs = [np.zeros(s) for s in SHAPES]
    tp = [torch.tensor(p, dtype=torch.float64, requires_grad=True) for p in params]
    opt = torch.optim.SGD([{"params": [t for t, g in zip(tp, GROUPS) if g == k], "lr": HP[k][0],
                            "weight_decay": HP[k][1]} for k in range(3)], lr=0.01, momentum=0.937, nesterov=True)
    for step in range(4):
        grads = make(10 + step, SHAPES, gscale)
        for t, g in zip(tp, grads):
            t.grad = torch.tensor(g, dtype=torch.float64)
        tn = torch.nn.utils.clip_grad_norm_(tp, max_norm=10.0)
        opt.step()
        params, bufs, total = optim.sgd_nesterov_step(params, grads, bufs, GROUPS, HP, 0.937, 10.0)
        assert abs(total - float(tn)) <= 1e-12 * total
        for p, t in zip(params, tp):
            assert np.allclose(p, t.detach().numpy(), rtol=1e-13, atol=1e-15)


def test_closed_forms():
    # no clipping (norm 3 < 10), no decay: d = 3, buf = 3, w = 1 - 0.1 (3 + 0.9 * 3)
    w, b, total = optim.sgd_nesterov_step([np.array([1.0])], [np.array([3.0])], [np.zeros(1)], [0], [(0.1, 0.0)],
                                          0.9, 10.0)
    assert total == 3.0 and np.isclose(w[0][0], 1 - 0.1 * (3 + 0.9 * 3)) and b[0][0] == 3.0
    # clipping: gradients (30, 40) have norm 50, so they are scaled by 10 / (50 + 1e-6)
    w, b, total = optim.sgd_nesterov_step([np.zeros(2)], [np.array([30.0, 40.0])], [np.zeros(2)], [0], [(1.0, 0.0)],
                                          0.0, 10.0)
    c = 10.0 / (50.0 + 1e-6)
    assert total == 50.0 and np.allclose(b[0], [30 * c, 40 * c]) and np.allclose(w[0], [-30 * c, -40 * c])
    # weight decay only in its group
    w, _, _ = optim.sgd_nesterov_step([np.array([2.0]), np.array([2.0])], [np.zeros(1), np.zeros(1)],
                                      [np.zeros(1), np.zeros(1)], [0, 1], [(0.5, 0.1), (0.5, 0.0)], 0.0, 10.0)
    assert np.isclose(w[0][0], 2 - 0.5 * 0.1 * 2) and w[1][0] == 2.0


def test_planted_mistakes_are_caught():
    """Per-tensor clipping, heavy-ball momentum or decay in every group each change the
    result the torch pin checks: the pin is sensitive to each."""
    params, grads = make(3, SHAPES), make(4, SHAPES, 10.0)
    bufs = [np.zeros(s) for s in SHAPES]
    ref, _, _ = optim.sgd_nesterov_step(params, grads, bufs, GROUPS, HP, 0.937, 10.0)
    # per-tensor clipping
    alt = []
    for p, g, k in zip(params, grads, GROUPS):
        c = optim.clip_coefficient(optim.global_norm([g]), 10.0)
        lr, wd = HP[k]
        d = g * c + wd * p
        alt.append(p - lr * (d + 0.937 * d))
    assert max(np.abs(a - r).max() for a, r in zip(alt, ref)) > 1e-4
    # heavy-ball momentum (no look-ahead)
    c = optim.clip_coefficient(optim.global_norm(grads), 10.0)
    alt = [p - HP[k][0] * (g * c + HP[k][1] * p) for p, g, k in zip(params, grads, GROUPS)]
    assert max(np.abs(a - r).max() for a, r in zip(alt, ref)) > 1e-5
    # decay in every group
    alt, _, _ = optim.sgd_nesterov_step(params, grads, bufs, GROUPS, [(h[0], 3.75e-4) for h in HP], 0.937, 10.0)
    assert max(np.abs(a - r).max() for a, r in zip(alt, ref)) > 1e-7
