"""ORACLE -- test infrastructure only.  The optimiser step that follows the weight
gradients, float64 numpy.

What it follows:
  * global-norm gradient clipping applied every step with max norm 10 (Sec. 3.2,
    optimisation: one squared-norm accumulation over every gradient; Table 1
    optimisation row; Table 2 divergence #7): the reference-default rule of
    Pascanu et al. as the reference ecosystem implements it -- total = sqrt of the
    sum of squares of every gradient element, coefficient = max_norm / (total +
    1e-6) capped at 1, every gradient multiplied by the coefficient;
  * SGD with Nesterov momentum in three parameter groups (Table 1 optimisation row:
    decayed weights, undecayed normalisation gains, undecayed biases; momentum 0.937,
    weight decay 5e-4 scaled by the effective batch) with the reference-default update:
        d   = g + weight_decay * w
        buf = momentum * buf + d          (buf starts at zero, so the first step gives d)
        w   = w - lr * (d + momentum * buf)
    (no dampening).  Each tensor names its group; a group carries (lr, weight_decay).

Inputs and outputs are lists of float64 arrays (one per parameter tensor).
"""
from __future__ import annotations

from typing import List, Sequence, Tuple

import numpy as np

CLIP_EPS = 1e-6


def global_norm(grads: Sequence[np.ndarray]) -> float:
    """sqrt(sum over every tensor and element of g^2)."""
    return float(np.sqrt(sum(float(np.sum(np.asarray(g, np.float64) ** 2)) for g in grads)))


def clip_coefficient(total: float, max_norm: float) -> float:
    """min(1, max_norm / (total + 1e-6))."""
    return min(1.0, max_norm / (total + CLIP_EPS))


def sgd_nesterov_step(params: Sequence[np.ndarray], grads: Sequence[np.ndarray], bufs: Sequence[np.ndarray],
                      groups: Sequence[int], group_hparams: Sequence[Tuple[float, float]], momentum: float,
                      max_norm: float):
    """One clipped SGD-Nesterov step.  group_hparams[k] = (lr, weight_decay) of group k.
    Returns (new params, new momentum buffers, total gradient norm before clipping)."""
    total = global_norm(grads)
    coef = clip_coefficient(total, max_norm)
    new_w: List[np.ndarray] = []
    new_b: List[np.ndarray] = []
    for w, g, b, k in zip(params, grads, bufs, groups):
        lr, wd = group_hparams[k]
        w = np.asarray(w, np.float64)
        d = np.asarray(g, np.float64) * coef + wd * w
        nb = momentum * np.asarray(b, np.float64) + d
        new_w.append(w - lr * (d + momentum * nb))
        new_b.append(nb)
    return new_w, new_b, total
