"""The C ABI driven without Python tensors, and the hot path under HIP graph
capture."""
import ctypes
import os
import subprocess

import numpy as np
import pytest
import torch

import synth
from parity_util import host

pytestmark = pytest.mark.gpu

HERE = os.path.dirname(os.path.abspath(__file__))


@pytest.mark.parametrize("tables", ["1", "2"])
def test_plain_c_program_matches_oracle(dev, tables):
    """tests/c/abi_step_check.c: hipMalloc'd buffers, warm-up + compression
    steps through the C ABI, compared with the oracle in the same process;
    with the chunk owners' tables chosen by the default rule (1: built per
    tile for this small plan) and kept in the workspace (2)."""
    from tests.c import build as cb
    if not os.path.exists(cb.BIN):
        cb.build()
    r = subprocess.run([cb.BIN, tables], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0 and r.stdout.strip() == "ok", (r.returncode, r.stdout, r.stderr)


@pytest.mark.parametrize("tables", ["auto", "on"])
def test_step_replays_from_a_hip_graph(dev, tables):
    """onebit_step captured once in a graph and replayed gives the eager
    result bit for bit, replay after replay (fresh gradients each time);
    'on': the chunk owners' tables are built in the workspace by their own
    kernel and copied into LDS by direct loads, inside the graph too."""
    import paper_2102_02888_amd as ob
    numel, n = [200_000, 3000, 64], 4
    plan = ob.Plan(numel, n)
    plan.set_server_tables(ob.SERVER_TABLES_ON if tables == "on" else ob.SERVER_TABLES_AUTO)
    wl = synth.Workload(name="graph", numel=numel, n=n, warmup_steps=2, steps=0)
    states = [ob.State(plan, dev), ob.State(plan, dev)]
    x0 = torch.from_numpy(synth.host_params(wl, plan.D)).to(dev)
    for st in states:
        st.x.copy_(x0)
    # Algorithm 1's order: both warm-up steps, then (v frozen) the first
    # compression step eagerly, with the warm-up's fp32 momentum
    for t in (1, 2):
        g = torch.from_numpy(synth.host_grads(wl, plan.D, plan.tensor_off, t)).to(dev)
        for st in states:
            st.grads.copy_(g)
            st.warmup(wl.lr, wl.beta1, wl.beta2, wl.eps, t)
    g = torch.from_numpy(synth.host_grads(wl, plan.D, plan.tensor_off, 3)).to(dev)
    for st in states:
        st.grads.copy_(g)
        st.step(wl.lr, wl.beta1, wl.eps)
        assert st.momentum_is_packed()  # the next step decodes m from the message
    torch.cuda.synchronize()
    eager, graphed = states
    graph = torch.cuda.CUDAGraph()
    # capture one packed-momentum step of the second state
    snapshot = [t.clone() for t in (graphed.x, graphed.worker_err, graphed.worker_scales,
                                    graphed.server_err, graphed.server_bits, graphed.server_scales)]
    with torch.cuda.graph(graph):
        graphed.step(wl.lr, wl.beta1, wl.eps)
    # capture does not run the kernels; restore the state anyway to be sure
    for dst, src in zip((graphed.x, graphed.worker_err, graphed.worker_scales,
                         graphed.server_err, graphed.server_bits, graphed.server_scales), snapshot):
        dst.copy_(src)
    torch.cuda.synchronize()
    for k in range(4):
        g = torch.from_numpy(synth.host_grads(wl, plan.D, plan.tensor_off, 10 + k)).to(dev)
        eager.grads.copy_(g)
        graphed.grads.copy_(g)
        eager.step(wl.lr, wl.beta1, wl.eps)
        graph.replay()
        torch.cuda.synchronize()
        for name in ("x", "worker_err", "worker_bits", "worker_scales", "server_err",
                     "server_bits", "server_scales"):
            a, b = host(getattr(eager, name)), host(getattr(graphed, name))
            assert a.tobytes() == b.tobytes(), (k, name)
    plan.close()


def test_argument_errors_on_device_buffers(dev):
    """Misaligned or out-of-range arguments on real device buffers are refused
    before any launch, and leave every buffer as it was."""
    import paper_2102_02888_amd as ob
    from paper_2102_02888_amd import _native
    L = _native.lib()
    numel, n = [1000, 64], 2
    plan = ob.Plan(numel, n)
    st = ob.State(plan, dev)
    st.x.normal_()
    st.grads.normal_()
    before = st.x.clone()
    vp = ctypes.c_void_p
    s0 = vp(torch.cuda.current_stream().cuda_stream)

    def p(t, byte_off=0):
        return vp(t.data_ptr() + byte_off)

    def step(**kw):
        a = dict(x=p(st.x), m=p(st.m), v=p(st.v), g=p(st.grads), gd=0, gld=plan.D,
                 we=p(st.worker_err), eld=plan.D, se=p(st.server_err), wb=p(st.worker_bits),
                 ws=p(st.worker_scales), sb=p(st.server_bits), ss=p(st.server_scales),
                 wsp=p(st.workspace))
        a.update(kw)
        return L.onebit_step(plan.handle, a["x"], a["m"], a["v"], a["g"], a["gd"], a["gld"],
                             a["we"], a["eld"], a["se"], a["wb"], a["ws"], a["sb"], a["ss"],
                             1e-3, 0.9, 1e-8, a["wsp"], s0)

    assert step(x=p(st.x, 4)) == -2 and b"x" in L.onebit_last_error()
    assert step(g=p(st.grads, 4)) == -2
    assert step(gd=3) == -1
    assert step(gld=plan.D - 4) == -1
    assert step(eld=plan.D + 2) == -2
    assert step(wb=p(st.worker_bits, 4)) == -2
    assert step(wsp=p(st.workspace, 8)) == -2
    assert step(ss=None) == -1
    # chunk range and per-rank offsets of the server entry point
    args = (p(st.worker_bits), plan.W, 0, p(st.worker_scales), plan.S, 0, p(st.server_err),
            p(st.server_bits), p(st.server_scales), p(st.workspace), s0)
    assert L.onebit_server_reduce_compress(plan.handle, 0, n + 1, *args) == -1
    assert L.onebit_server_reduce_compress(plan.handle, 1, 1, *args) == -1
    bad_base = (p(st.worker_bits), plan.W, plan.W + 1) + args[3:]
    assert L.onebit_server_reduce_compress(plan.handle, 0, n, *bad_base) == -1
    # n_local outside [1, n]
    assert L.onebit_worker_compress(plan.handle, p(st.m), None, None, p(st.grads), 0, plan.D,
                                    n + 1, p(st.worker_err), plan.D, p(st.worker_bits), plan.W,
                                    p(st.worker_scales), plan.S, 0.9, p(st.workspace), s0) == -1
    # warm-up step numbers are 1-based
    assert L.onebit_warmup_adam_step(plan.handle, p(st.x), p(st.m), p(st.v), p(st.grads), 0,
                                     plan.D, n, 1e-3, 0.9, 0.999, 1e-8, 0, 0, s0) == -1
    # plans over 2^25 tiles are refused (one wave per tile must fit a launch)
    huge = (ctypes.c_int64 * 1)(1 << 35)
    out = ctypes.c_void_p()
    assert L.onebit_plan_create(huge, 1, 1, ctypes.byref(out)) == -1
    assert b"tiles" in L.onebit_last_error() and out.value is None
    torch.cuda.synchronize()
    assert torch.equal(st.x, before)
    # a correct call still goes through afterwards
    assert step() == 0
    torch.cuda.synchronize()
    assert not torch.equal(st.x, before)
    plan.close()


def test_one_plan_two_streams(dev):
    """One plan driven from two streams at once, each state with its own
    workspace, gives the same bits as running the two states one after the
    other."""
    import paper_2102_02888_amd as ob
    numel, n = [300_000, 5000, 64], 4
    plan = ob.Plan(numel, n)
    wl = synth.Workload(name="streams", numel=numel, n=n, warmup_steps=2, steps=0)

    def make():
        st = ob.State(plan, dev)
        st.x.copy_(torch.from_numpy(synth.host_params(wl, plan.D)).to(dev))
        return st

    states = [make() for _ in range(4)]  # [a, b] concurrent, [c, d] sequential
    grads = [torch.from_numpy(synth.host_grads(wl, plan.D, plan.tensor_off, t)).to(dev)
             for t in range(1, 6)]
    torch.cuda.synchronize()
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    for t, g in enumerate(grads, start=1):
        for k, st in enumerate(states):
            st.grads.copy_(g if k % 2 == 0 else g * 0.5)
        torch.cuda.synchronize()
        for k in (0, 1):
            with torch.cuda.stream(streams[k]):
                if t <= 2:
                    states[k].warmup(wl.lr, wl.beta1, wl.beta2, wl.eps, t)
                else:
                    states[k].step(wl.lr, wl.beta1, wl.eps)
        for k in (2, 3):
            if t <= 2:
                states[k].warmup(wl.lr, wl.beta1, wl.beta2, wl.eps, t)
            else:
                states[k].step(wl.lr, wl.beta1, wl.eps)
        torch.cuda.synchronize()
    for a, b in ((0, 2), (1, 3)):
        for name in ("x", "worker_err", "worker_bits", "worker_scales", "server_err",
                     "server_bits", "server_scales"):
            assert host(getattr(states[a], name)).tobytes() == \
                host(getattr(states[b], name)).tobytes(), (a, name)
    plan.close()


@pytest.mark.parametrize("packed", [True, False])
def test_checkpoint_resume_bit_exact(dev, tmp_path, packed):
    """2 warm-up + 3 compression steps, state saved to a safetensors file and
    loaded into a fresh plan and state, 3 more steps: identical to 6 straight
    compression steps (the errors and the last server message are state)."""
    from safetensors.torch import load_file, save_file
    import paper_2102_02888_amd as ob
    numel, n = [100_000, 3000, 64, 0, 777], 4
    wl = synth.Workload(name="ckpt", numel=numel, n=n, warmup_steps=2, steps=6)

    def run(st, t0, t1):
        for t in range(t0, t1):
            g = synth.host_grads(wl, st.plan.D, st.plan.tensor_off, t)
            st.grads.copy_(torch.from_numpy(g))
            if t <= wl.warmup_steps:
                st.warmup(wl.lr, wl.beta1, wl.beta2, wl.eps, t)
            else:
                st.step(wl.lr, wl.beta1, wl.eps)

    plan = ob.Plan(numel, n)
    x0 = torch.from_numpy(synth.host_params(wl, plan.D))
    straight = ob.State(plan, dev, packed_momentum=packed)
    straight.x.copy_(x0)
    run(straight, 1, 9)
    first = ob.State(plan, dev, packed_momentum=packed)
    first.x.copy_(x0)
    run(first, 1, 6)
    torch.cuda.synchronize()
    path = str(tmp_path / "state.safetensors")
    save_file(first.state_dict(), path)
    plan2 = ob.Plan(numel, n)
    resumed = ob.State(plan2, dev, packed_momentum=not packed)  # flag restored from the file
    resumed.load_state_dict(load_file(path))
    assert resumed.packed_momentum == packed and resumed.compression_steps == 3
    run(resumed, 6, 9)
    torch.cuda.synchronize()
    for name in ("x", "worker_err", "worker_bits", "worker_scales", "server_err", "server_bits",
                 "server_scales"):
        assert host(getattr(resumed, name)).tobytes() == \
            host(getattr(straight, name)).tobytes(), name
    assert host(resumed.momentum()).tobytes() == host(straight.momentum()).tobytes()
    plan.close()
    plan2.close()


def test_binding_refuses_short_buffers(dev):
    """The Python binding checks every buffer against the plan's sizes, so a
    short tensor raises instead of reaching a kernel."""
    import paper_2102_02888_amd as ob
    plan = ob.Plan([5000, 64], 4)
    st = ob.State(plan, dev)
    short = torch.zeros(plan.D - 64, device=dev)
    with pytest.raises(ValueError, match="x"):
        ob.onebit_decompress_update(plan, st.server_bits, st.server_scales, short, None, st.v,
                                    1e-3, 1e-8)
    with pytest.raises(ValueError, match="grads"):
        ob.onebit_worker_compress(plan, st.m, st.grads[:, :plan.D - 64], st.worker_err,
                                  st.worker_bits, st.worker_scales, 0.9, st.workspace)
    with pytest.raises(ValueError, match="worker_bits"):
        ob.onebit_server_reduce_compress(plan, 0, 4, st.worker_bits[:3], st.worker_scales,
                                         st.server_err, st.server_bits, st.server_scales,
                                         st.workspace)
    with pytest.raises(ValueError, match="workspace"):
        ob.onebit_l1_norm(plan, st.v, st.workspace[:4], torch.zeros(1, dtype=torch.float64,
                                                                     device=dev))
    with pytest.raises(ValueError, match="worker_scales"):
        ob.onebit_server_reduce_compress(plan, 0, 4, st.worker_bits, st.worker_scales.reshape(-1),
                                         st.server_err, st.server_bits, st.server_scales,
                                         st.workspace, scales_ld=plan.S + 1)
    torch.cuda.synchronize()
    plan.close()


def test_plan_without_elements(dev):
    """Only empty tensors (d = 0): every call succeeds without touching an
    element buffer (zero-size tensors pass NULL), and every segment's scale
    is 0."""
    import paper_2102_02888_amd as ob
    plan = ob.Plan([0, 0], 3)
    assert (plan.d, plan.D, plan.W, plan.S, plan.T) == (0, 0, 0, 6, 0)
    st = ob.State(plan, dev)
    st.worker_scales.fill_(7.0)
    st.server_scales.fill_(7.0)
    for t in (1, 2):
        st.warmup(1e-3, 0.9, 0.999, 1e-8, t)
    for _ in range(3):
        st.step(1e-3, 0.9, 1e-8)
    st.step_uncompressed(1e-3, 0.9, 1e-8)
    assert st.variance_l1_norm() == 0.0
    torch.cuda.synchronize()
    assert not host(st.worker_scales).any() and not host(st.server_scales).any()
    assert st.momentum().numel() == 0 and st.worker_delta().numel() == 0
    plan.close()


def test_step_events_form_matches_plain_step(dev):
    """onebit_step_events runs the launches of onebit_step bit for bit and
    marks the stream in order around the three phases."""
    import paper_2102_02888_amd as ob
    from paper_2102_02888_amd import _native
    numel, n = [300_000, 5000, 64], 4
    plan = ob.Plan(numel, n)
    wl = synth.Workload(name="events", numel=numel, n=n, warmup_steps=1, steps=0)
    states = [ob.State(plan, dev), ob.State(plan, dev)]
    x0 = torch.from_numpy(synth.host_params(wl, plan.D)).to(dev)
    g = torch.from_numpy(synth.host_grads(wl, plan.D, plan.tensor_off, 1)).to(dev)
    for st in states:
        st.x.copy_(x0)
        st.grads.copy_(g)
        st.warmup(wl.lr, wl.beta1, wl.beta2, wl.eps, 1)
    events = [torch.cuda.Event(enable_timing=True) for _ in range(4)]
    for e in events:
        e.record()
    for t in (2, 3, 4):
        g = torch.from_numpy(synth.host_grads(wl, plan.D, plan.tensor_off, t)).to(dev)
        for st in states:
            st.grads.copy_(g)
        states[0].step(wl.lr, wl.beta1, wl.eps)
        states[1].step(wl.lr, wl.beta1, wl.eps, events=events)
        torch.cuda.synchronize()
        for name in ("x", "m", "worker_err", "worker_bits", "worker_scales", "server_err",
                     "server_bits", "server_scales"):
            a, b = host(getattr(states[0], name)), host(getattr(states[1], name))
            assert a.tobytes() == b.tobytes(), (t, name)
        spans = [events[k].elapsed_time(events[k + 1]) for k in range(3)]
        assert all(s >= 0 for s in spans) and spans[0] > 0, spans
    # a NULL event array is refused before any launch
    st = states[1]
    before = host(st.x).copy()
    vp = ctypes.c_void_p
    L = _native.lib()
    rc = L.onebit_step_events(plan.handle, vp(st.x.data_ptr()), None, vp(st.v.data_ptr()),
                              vp(st.grads.data_ptr()), 0, plan.D, vp(st.worker_err.data_ptr()),
                              plan.D, vp(st.server_err.data_ptr()),
                              vp(st.worker_bits.data_ptr()), vp(st.worker_scales.data_ptr()),
                              vp(st.server_bits.data_ptr()), vp(st.server_scales.data_ptr()),
                              1e-3, 0.9, 1e-8, vp(st.workspace.data_ptr()), None,
                              vp(torch.cuda.current_stream().cuda_stream))
    torch.cuda.synchronize()
    assert rc == -1 and b"events" in L.onebit_last_error()
    assert host(st.x).tobytes() == before.tobytes()
    plan.close()
