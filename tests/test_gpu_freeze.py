"""The variance l1 norm on the GPU versus the oracle, and the automatic end
of the warm-up decided on GPU norms versus on oracle norms."""
import math

import numpy as np
import pytest
import torch

import oracle
import synth
from parity_util import check_fp, host

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def ob():
    import paper_2102_02888_amd as ob
    return ob


@pytest.mark.parametrize("numel,n", [([1 << 20], 4), ([1000, 0, 77, 4096, 1, 70_001], 3),
                                     (synth.stress_sizes()[:300], 8)])
def test_l1_norm_parity(ob, dev, numel, n):
    L = oracle.Layout(numel, n)
    plan = ob.Plan(numel, n)
    v = synth.host_normal(L.D, 1e-3, 7)
    v[~L.real_mask()] = 1e6  # padding must not count
    out = torch.zeros(1, dtype=torch.float64, device=dev)
    ob.onebit_l1_norm(plan, torch.from_numpy(v).to(dev), plan.workspace(dev), out)
    got = float(out.item())
    ref = oracle.l1_norm(L, v)
    assert abs(got - ref) <= 1e-12 * ref, (got, ref)
    plan.close()


def test_l1_norm_full_size(ob, dev):
    wl = synth.get("bert_large")
    plan = ob.Plan(wl.numel, wl.n)
    L = oracle.Layout(wl.numel, wl.n)
    v = np.abs(synth.host_normal(plan.D, 1e-6, 8))
    out = torch.zeros(1, dtype=torch.float64, device=dev)
    ob.onebit_l1_norm(plan, torch.from_numpy(v).to(dev), plan.workspace(dev), out)
    got = float(out.item())
    ref = oracle.l1_norm(L, v)
    assert abs(got - ref) <= 1e-12 * ref, (got, ref)
    plan.close()


def test_auto_freeze_matches_oracle(ob, dev):
    """Warm-up with gradients whose magnitude decays to a floor (the variance
    first shrinks, then stabilises); beta2 = 0.9 so Delta = 10 steps."""
    beta2, A, tau = 0.9, 4.0, 25.0
    wl = synth.Workload(name="freeze", numel=[30_000, 500], n=2, warmup_steps=0, steps=0,
                        beta2=beta2)
    L = oracle.Layout(wl.numel, wl.n)
    plan = ob.Plan(wl.numel, wl.n)
    st = ob.State(plan, dev)
    mask = L.real_mask()
    x = synth.host_params(wl, L.D)
    x[~mask] = 0
    st.x.copy_(torch.from_numpy(x))
    m = np.zeros(L.D, np.float32)
    v = np.zeros(L.D, np.float32)
    det_gpu = ob.VarianceFreezeDetector(beta2, threshold=0.96, min_steps=40)
    det_ref = ob.VarianceFreezeDetector(beta2, threshold=0.96, min_steps=40)
    frozen = None
    for t in range(1, 300):
        g = synth.host_grads(wl, L.D, L.tensor_off, t)
        g *= np.float32(math.sqrt(1 + A * math.exp(-t / tau)))
        oracle.warmup_step(L, x, m, v, g, wl.n, wl.lr, wl.beta1, beta2, wl.eps, 0, t)
        st.grads.copy_(torch.from_numpy(g))
        st.warmup(wl.lr, wl.beta1, beta2, wl.eps, t)
        a = det_gpu.update(t, st.variance_l1_norm())
        b = det_ref.update(t, oracle.l1_norm(L, v))
        assert a == b, t
        if a:
            frozen = t
            break
    assert frozen is not None and frozen > 40
    check_fp("x at freeze", host(st.x), x, mask=mask)
    check_fp("v at freeze", host(st.v), v, mask=mask)
    plan.close()
