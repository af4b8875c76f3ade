"""OnebitAdam: Algorithm 1's two stages driven through the C ABI, against
the oracle's warm-up and compression steps."""
import math

import numpy as np
import pytest
import torch

import oracle
import synth
from parity_util import check_bits, check_fp, host


def test_driver_needs_one_warmup_rule():
    import paper_2102_02888_amd as ob
    with pytest.raises(ValueError):
        ob.OnebitAdam(None, "cpu", 1e-3)
    with pytest.raises(ValueError):
        ob.OnebitAdam(None, "cpu", 1e-3, warmup_steps=3,
                      freeze=ob.VarianceFreezeDetector(0.999))
    with pytest.raises(TypeError):
        ob.OnebitAdam(None, "cpu", 1e-3, freeze=0.96)


@pytest.mark.gpu
@pytest.mark.parametrize("packed", [True, False])
def test_fixed_warmup_then_compression_matches_oracle(dev, packed):
    """T_w = 3 Adam steps, then 5 compressed steps with a decaying lr."""
    import paper_2102_02888_amd as ob
    wl = synth.Workload(name="driver", numel=[40_000, 700, 64], n=4, warmup_steps=3, steps=5)
    L = oracle.Layout(wl.numel, wl.n)
    plan = ob.Plan(wl.numel, wl.n)
    opt = ob.OnebitAdam(plan, dev, wl.lr, wl.beta1, wl.beta2, wl.eps,
                        warmup_steps=wl.warmup_steps, packed_momentum=packed)
    mask = L.real_mask()
    x = synth.host_params(wl, L.D)
    x[~mask] = 0
    opt.x.copy_(torch.from_numpy(x))
    m = np.zeros(L.D, np.float32)
    v = np.zeros(L.D, np.float32)
    ref = None
    kinds = []
    for t in range(1, wl.warmup_steps + wl.steps + 1):
        g = synth.host_grads(wl, L.D, L.tensor_off, t)
        lr = wl.lr * (0.9 ** t)
        if t <= wl.warmup_steps:
            oracle.warmup_step(L, x, m, v, g, wl.n, lr, wl.beta1, wl.beta2, wl.eps, 0, t)
        else:
            if ref is None:
                ref = oracle.State(L, x, m, v)
            ref.step(g, lr, wl.beta1, wl.eps)
        opt.grads.copy_(torch.from_numpy(g))
        kinds.append(opt.step(lr=lr))
    torch.cuda.synchronize()
    assert kinds == ["warmup"] * 3 + ["compressed"] * 5 and opt.frozen_at == 3
    check_bits("server bits", host(opt.state.server_bits), ref.sbits)
    check_fp("x", host(opt.x), ref.x, mask=mask)
    check_fp("m", host(opt.state.momentum()), ref.m, mask=mask)
    plan.close()


@pytest.mark.gpu
def test_auto_freeze_driver(dev):
    """With a freeze detector the driver leaves the warm-up at the step the
    detector picks from the GPU's ||v||_1, the same step as on the oracle's
    variance, and compresses from then on."""
    import paper_2102_02888_amd as ob
    beta2, A, tau = 0.9, 4.0, 25.0
    wl = synth.Workload(name="autofreeze", numel=[20_000, 300], n=2, warmup_steps=0, steps=0,
                        beta2=beta2)
    L = oracle.Layout(wl.numel, wl.n)
    plan = ob.Plan(wl.numel, wl.n)
    opt = ob.OnebitAdam(plan, dev, wl.lr, wl.beta1, beta2, wl.eps,
                        freeze=ob.VarianceFreezeDetector(beta2, min_steps=40))
    det = ob.VarianceFreezeDetector(beta2, min_steps=40)
    x = synth.host_params(wl, L.D)
    x[~L.real_mask()] = 0
    opt.x.copy_(torch.from_numpy(x))
    m = np.zeros(L.D, np.float32)
    v = np.zeros(L.D, np.float32)
    ref_freeze = None
    for t in range(1, 300):
        g = synth.host_grads(wl, L.D, L.tensor_off, t)
        g *= np.float32(math.sqrt(1 + A * math.exp(-t / tau)))
        opt.grads.copy_(torch.from_numpy(g))
        kind = opt.step()
        if ref_freeze is None:
            oracle.warmup_step(L, x, m, v, g, wl.n, wl.lr, wl.beta1, beta2, wl.eps, 0, t)
            if det.update(t, oracle.l1_norm(L, v)):
                ref_freeze = t
            assert kind == "warmup"
        else:
            assert kind == "compressed"
            if t > ref_freeze + 3:
                break
    assert ref_freeze is not None and opt.frozen_at == ref_freeze > 40
    plan.close()


@pytest.mark.gpu
def test_graph_replay_matches_eager(dev):
    """graph=True replays a captured compressed step; after every step its
    state equals the eager driver's bit for bit, through an lr change (a new
    capture), with eager work and a host synchronisation between replays."""
    import paper_2102_02888_amd as ob
    wl = synth.Workload(name="graph", numel=[50_000, 900, 64], n=4, warmup_steps=2, steps=6)
    plan = ob.Plan(wl.numel, wl.n)
    eager = ob.OnebitAdam(plan, dev, wl.lr, wl.beta1, wl.beta2, wl.eps,
                          warmup_steps=wl.warmup_steps)
    graphed = ob.OnebitAdam(plan, dev, wl.lr, wl.beta1, wl.beta2, wl.eps,
                            warmup_steps=wl.warmup_steps, graph=True)
    x0 = torch.from_numpy(synth.host_params(wl, plan.D)).to(dev)
    eager.x.copy_(x0)
    graphed.x.copy_(x0)
    names = ("x", "worker_err", "worker_bits", "worker_scales", "server_err", "server_bits",
             "server_scales")
    captured = []
    for t in range(1, wl.warmup_steps + wl.steps + 1):
        g = torch.from_numpy(synth.host_grads(wl, plan.D, plan.tensor_off, t)).to(dev)
        lr = wl.lr if t < 6 else wl.lr * 0.5
        for opt in (eager, graphed):
            opt.grads.copy_(g)
            opt.step(lr=lr)
        captured.append(graphed._graph)
        torch.cuda.synchronize()
        for name in names:
            a, b = host(getattr(eager.state, name)), host(getattr(graphed.state, name))
            assert a.tobytes() == b.tobytes(), (t, name)
    # warm-up and the first compression step run eagerly; steps 4-5 replay one
    # graph, and the lr change at step 6 captures another
    assert captured[:3] == [None, None, None]
    assert captured[3] is not None and captured[4] is captured[3]
    assert captured[5] is not captured[4] and captured[7] is captured[5]
    plan.close()
