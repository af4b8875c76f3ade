"""Warm-up auto-tuning (Section 7.1): the oracle's variance l1 norm and the
freeze rule, pinned to library sums and a closed form."""
import math

import numpy as np
import pytest

import oracle
import synth
from paper_2102_02888_amd.freeze import VarianceFreezeDetector


def test_oracle_l1_norm_matches_exact_sum():
    L = oracle.Layout([1000, 0, 77, 4096, 1], 3)
    v = synth.host_normal(L.D, 1e-3, 5)
    mask = L.real_mask()
    ref = math.fsum(abs(float(a)) for a in v[mask])  # exactly rounded sum
    assert abs(oracle.l1_norm(L, v) - ref) <= 1e-13 * ref
    # padding does not count
    v2 = v.copy()
    v2[~mask] = 1e6
    assert oracle.l1_norm(L, v2) == oracle.l1_norm(L, v)


def _closed_form_v(t, beta2, c2, A, tau):
    """v_t of the recurrence v_t = beta2 v_{t-1} + (1-beta2) g_t^2, v_0 = 0,
    for g_t^2 = c2 (1 + A exp(-t/tau)), summed in closed form."""
    q = beta2 * math.exp(1.0 / tau)
    geo = t if abs(q - 1.0) < 1e-15 else (1.0 - q ** t) / (1.0 - q)
    return c2 * (1.0 - beta2 ** t) + A * c2 * (1.0 - beta2) * math.exp(-t / tau) * geo


def test_detector_on_closed_form_schedule():
    beta2, c2, A, tau = 0.9, 1e-6, 4.0, 25.0
    # while v grows from zero the ratio exceeds 1; the learning-rate warm-up
    # bound (min_steps) keeps the rule from firing there, as the paper requires
    det = VarianceFreezeDetector(beta2, threshold=0.96, min_steps=40)
    assert det.delta == 10
    vs = [_closed_form_v(t, beta2, c2, A, tau) for t in range(0, 400)]
    fired = None
    for t in range(1, 400):
        if det.update(t, 1000 * vs[t]):
            fired = t
            break
    # the rule, read off the closed-form sequence
    expect = next(t for t in range(40, 400) if vs[t] >= 0.96 * vs[t - 10])
    assert fired == expect and fired > 40   # the ratio is below 0.96 at step 40 and rises to 1
    assert vs[fired - 1] < 0.96 * vs[fired - 11]


def test_detector_respects_min_steps_and_order():
    det = VarianceFreezeDetector(0.9, min_steps=50)
    for t in range(1, 50):
        assert not det.update(t, 1.0)   # a constant norm satisfies the ratio at once
    assert det.update(50, 1.0) and det.frozen_at == 50
    with pytest.raises(ValueError):
        VarianceFreezeDetector(0.9).update(2, 1.0)


def test_oracle_warmup_variance_follows_closed_form():
    """The oracle's warm-up v on gradients of magnitude c sqrt(1 + A e^{-t/tau})
    follows the closed form (a pin of the v recurrence and of the l1 norm)."""
    beta2, A, tau, c = 0.9, 4.0, 25.0, 1e-3
    L = oracle.Layout([512], 1)
    sign = np.where(np.arange(512) % 3 == 0, -1.0, 1.0)
    x = np.zeros(512, np.float32); m = np.zeros(512, np.float32); v = np.zeros(512, np.float32)
    for t in range(1, 60):
        g = (sign * c * math.sqrt(1 + A * math.exp(-t / tau))).astype(np.float32)
        oracle.warmup_step(L, x, m, v, g[None, :].copy(), 1, 1e-4, 0.9, beta2, 1e-8, 0, t)
        g2 = float(np.float64(g[0]) ** 2)
        ref = _closed_form_v(t, beta2, c * c, A, tau)
        assert abs(oracle.l1_norm(L, v) / 512 - ref) <= 2e-6 * ref
