"""Shared helpers of the GPU parity tests: seeded inputs, tolerances, comparisons.

Tolerances (stated for every comparison):
  * bf16 outputs and all gradients: rel_inf = max|gpu - ref| / max|ref| <= 2e-2;
  * fp32 batch statistics: max_c |dvar| / var <= 1e-5 and max_c |dmean| / sqrt(var + eps) <= 1e-5.
"""
import numpy as np

from paper_2609_10632_amd import synth

REL_TOL = 2e-2
STAT_TOL = 1e-5

# one line per compared layer or chain (what was compared completely, what was sampled);
# printed in the session's terminal summary
REPORT = []


def report(line: str) -> None:
    REPORT.append(line)
    print(line, flush=True)


def rel_inf(gpu, ref) -> float:
    gpu = np.asarray(gpu, np.float64)
    ref = np.asarray(ref, np.float64)
    assert gpu.shape == ref.shape, (gpu.shape, ref.shape)
    den = np.abs(ref).max()
    return float(np.abs(gpu - ref).max() / (den if den > 0 else 1.0))


def assert_close(gpu, ref, what, tol=REL_TOL):
    e = rel_inf(gpu, ref)
    assert np.all(np.isfinite(gpu)), f"{what}: non-finite values"
    assert e <= tol, f"{what}: rel_inf {e:.3e} > {tol:.1e}"
    return e


def assert_stats(mean_gpu, var_gpu, mean_ref, var_ref, eps, what):
    mean_gpu, var_gpu = np.asarray(mean_gpu, np.float64), np.asarray(var_gpu, np.float64)
    ev = float(np.max(np.abs(var_gpu - var_ref) / var_ref))
    em = float(np.max(np.abs(mean_gpu - mean_ref) / np.sqrt(var_ref + eps)))
    assert ev <= STAT_TOL, f"{what}: variance rel err {ev:.3e} > {STAT_TOL:.0e}"
    assert em <= STAT_TOL, f"{what}: mean err {em:.3e} > {STAT_TOL:.0e}"
    return em, ev


class Inputs:
    """Seeded bf16 inputs for one test case (config number, layer index)."""

    def __init__(self, config: int, layer: int = 0):
        self.config, self.layer = config, layer

    def sid(self, t):
        return synth.stream_id(self.config, self.layer, t)

    def normal(self, shape, t, mean=0.0, std=1.0):
        return synth.bf16(shape, self.sid(t), synth.NORMAL, mean, std)

    def uniform(self, shape, t, lo, hi):
        return synth.bf16(shape, self.sid(t), synth.UNIFORM, lo, hi)

    def weight(self, co, k, ci, t=synth.T_W):
        b = synth.kaiming_uniform_bound(ci * k * k)
        return self.uniform((co, k, k, ci), t, -b, b)

    def f32_uniform(self, shape, t, lo, hi):
        return synth.f32(shape, self.sid(t), synth.UNIFORM, lo, hi)

    def f32_normal(self, shape, t, mean, std):
        return synth.f32(shape, self.sid(t), synth.NORMAL, mean, std)


f64 = synth.bf16_to_f64
