"""The paper's comparison variants of Section 7.2 on the GPU versus the oracle:
"1-bit Adam (32-bits)" (variance frozen, momenta averaged uncompressed) and
"Adam(1-bit Naive)" (the gradient error-compensated and compressed, Adam on
the decoded average, variance not frozen)."""
import numpy as np
import pytest
import torch

import oracle
import synth
from parity_util import check_bits, check_fp, check_scales, host

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def ob():
    import paper_2102_02888_amd as ob
    return ob


def _setup(ob, dev, wl, grad_dtype=torch.float32):
    L = oracle.Layout(wl.numel, wl.n)
    plan = ob.Plan(wl.numel, wl.n)
    mask = L.real_mask()
    x = synth.host_params(wl, L.D)
    x[~mask] = 0
    st = ob.State(plan, dev, grad_dtype=grad_dtype)
    st.x.copy_(torch.from_numpy(x))
    return L, plan, st, x, mask


def _grads(wl, L, t, grad_dtype):
    g = synth.host_grads(wl, L.D, L.tensor_off, t)
    gt = torch.from_numpy(g).to(grad_dtype)
    return gt, gt.float().numpy()


@pytest.mark.parametrize("grad_dtype", [torch.float32, torch.bfloat16])
def test_uncompressed_variant_free_running(ob, dev, grad_dtype):
    wl = synth.Workload(name="u32", numel=[70_001, 1000, 64, 5], n=4, warmup_steps=3, steps=5)
    L, plan, st, x, mask = _setup(ob, dev, wl, grad_dtype)
    m = np.zeros(L.D, np.float32)
    v = np.zeros(L.D, np.float32)
    for t in range(1, wl.warmup_steps + 1):
        gt, g = _grads(wl, L, t, grad_dtype)
        oracle.warmup_step(L, x, m, v, g, wl.n, wl.lr, wl.beta1, wl.beta2, wl.eps, 0, t)
        st.grads.copy_(gt.to(dev))
        st.warmup(wl.lr, wl.beta1, wl.beta2, wl.eps, t)
    for t in range(wl.warmup_steps + 1, wl.warmup_steps + wl.steps + 1):
        gt, g = _grads(wl, L, t, grad_dtype)
        oracle.step_uncompressed(L, x, m, v, g, wl.lr, wl.beta1, wl.eps)
        st.grads.copy_(gt.to(dev))
        st.step_uncompressed(wl.lr, wl.beta1, wl.eps)
    torch.cuda.synchronize()
    check_fp("x", host(st.x), x, mask=mask)
    check_fp("m", host(st.m), m, mask=mask)
    plan.close()


def test_naive_variant_free_running(ob, dev):
    wl = synth.Workload(name="naive", numel=[50_000, 300, 4097], n=3, warmup_steps=0, steps=5)
    L, plan, st, x, mask = _setup(ob, dev, wl)
    n = wl.n
    m = np.zeros(L.D, np.float32)
    v = np.zeros(L.D, np.float32)
    zero = np.zeros(L.D, np.float32)
    delta = np.zeros((n, L.D), np.float32)
    dbar = np.zeros(L.D, np.float32)
    wbits = np.zeros((n, L.W), np.uint64)
    wscales = np.zeros((n, L.S), np.float32)
    sbits = np.zeros(L.W, np.uint64)
    sscales = np.zeros(L.S, np.float32)
    z = np.zeros(L.D, np.float32)
    for t in range(1, wl.steps + 1):
        gt, g = _grads(wl, L, t, torch.float32)
        # oracle: compress g_i + delta_i per worker (the worker step with beta1 = 0 over a
        # zero momentum), chunk owners average and recompress, Adam on the decoded result
        for i in range(n):
            for q, (b, e) in enumerate(L.segments()):
                wscales[i, q] = oracle.worker_segment(b, e, 0.0, zero, g[i], delta[i], wbits[i], z)
        for q, (b, e) in enumerate(L.segments()):
            sscales[q] = oracle.server_segment(b, e, n, wbits.reshape(-1), L.W,
                                               np.ascontiguousarray(wscales[:, q]), 1, dbar,
                                               sbits, z)
        gdec = oracle.decode_message(L, sbits, sscales)
        oracle.warmup_step(L, x, m, v, gdec[None, :].copy(), 1, wl.lr, wl.beta1, wl.beta2,
                           wl.eps, 0, t)
        st.grads.copy_(gt.to(dev))
        st.step_naive(wl.lr, wl.beta1, wl.beta2, wl.eps, t)
        torch.cuda.synchronize()
        check_bits("step %d worker bits" % t, host(st.worker_bits), wbits)
        check_bits("step %d server bits" % t, host(st.server_bits), sbits)
        check_scales("step %d server scales" % t, host(st.server_scales), sscales)
    check_fp("x", host(st.x), x, mask=mask)
    check_fp("m", host(st.m), m, mask=mask)
    check_fp("v", host(st.v), v, mask=mask)
    check_fp("worker delta", host(st.worker_delta()), delta, mask=mask)
    check_fp("server delta", host(st.server_delta()), dbar, mask=mask)
    plan.close()


def test_naive_worker_pass_matches_zero_fp32_momentum_bitwise(ob, dev):
    """step_naive's worker call decodes m from all-ones sign words and zero
    scales (+0 everywhere) to take the packed-momentum pass; with beta1 = 0
    that is bit for bit the fp32-momentum row walk over a zero m, including
    ragged tiles and an empty tensor, over several steps of error feedback."""
    wl = synth.Workload(name="naive_eq", numel=[70_001, 0, 4097, 1000], n=5, warmup_steps=0,
                        steps=3)
    L, plan, a, x, mask = _setup(ob, dev, wl)
    b = ob.State(plan, dev)
    b.x.copy_(a.x)
    zero_m = torch.zeros_like(a.m)
    for t in range(1, wl.steps + 1):
        gt, _ = _grads(wl, L, t, torch.float32)
        a.grads.copy_(gt.to(dev))
        b.grads.copy_(gt.to(dev))
        a.step_naive(wl.lr, wl.beta1, wl.beta2, wl.eps, t)
        ob.onebit_worker_compress(plan, zero_m, b.grads, b.worker_err, b.worker_bits,
                                  b.worker_scales, 0.0, b.workspace)
        torch.cuda.synchronize()
        assert torch.equal(a.worker_bits, b.worker_bits), t
        assert torch.equal(a.worker_scales.view(torch.int32), b.worker_scales.view(torch.int32)), t
        assert torch.equal(a.worker_err.view(torch.int32), b.worker_err.view(torch.int32)), t
    plan.close()
