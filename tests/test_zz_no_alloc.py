"""onebit_step_noalloc, the step for callers that cannot allocate, against
onebit_step with a caller workspace: identical results, bit for bit, over
two runs in a row on one device (the second plan smaller than the first, so
the second run reuses the library's scratch array with less of it live),
with the chunk owners' tables built per tile (the default for plans this
small) and kept in the workspace, here the scratch array."""
import ctypes

import pytest
import torch

import synth
from parity_util import host

pytestmark = pytest.mark.gpu

NAMES = ("x", "m", "worker_err", "worker_bits", "worker_scales", "server_err", "server_bits",
         "server_scales")


def _compare_runs(ob, dev, numel, n, steps, seed, tables):
    plan = ob.Plan(numel, n)
    plan.set_server_tables(tables)
    assert plan.workspace_bytes <= (96 << 20)
    wl = synth.Workload(name="noalloc", numel=numel, n=n, warmup_steps=1, steps=steps,
                        seed_grads=seed)
    ref, new = ob.State(plan, dev), ob.State(plan, dev)
    x0 = torch.from_numpy(synth.host_params(wl, plan.D)).to(dev)
    g = torch.from_numpy(synth.host_grads(wl, plan.D, plan.tensor_off, 1)).to(dev)
    for st in (ref, new):
        st.x.copy_(x0)
        st.grads.copy_(g)
        st.warmup(wl.lr, wl.beta1, wl.beta2, wl.eps, 1)
    for t in range(2, 2 + steps):
        g = torch.from_numpy(synth.host_grads(wl, plan.D, plan.tensor_off, t)).to(dev)
        ref.grads.copy_(g)
        new.grads.copy_(g)
        packed = t > 2  # the first compression step reads the warm-up's fp32 m
        ref.step(wl.lr, wl.beta1, wl.eps)
        ob.onebit_step_noalloc(plan, new.x, None if packed else new.m, new.v, new.grads,
                               new.worker_err, new.server_err, new.worker_bits,
                               new.worker_scales, new.server_bits, new.server_scales, wl.lr,
                               wl.beta1, wl.eps)
        torch.cuda.synchronize()
        for name in NAMES:
            a, b = host(getattr(ref, name)), host(getattr(new, name))
            assert a.tobytes() == b.tobytes(), (numel, n, t, name)
    plan.close()


@pytest.mark.parametrize("tables", ["auto", "on"])
def test_noalloc_step_matches_workspace_step(dev, tables):
    import paper_2102_02888_amd as ob
    mode = ob.SERVER_TABLES_AUTO if tables == "auto" else ob.SERVER_TABLES_ON
    # a plan of 1,079 tiles, then a smaller one of 96 tiles
    _compare_runs(ob, dev, [1_000_000, 70_001, 5000, 64, 0, 300], 8, steps=3, seed=21,
                  tables=mode)
    _compare_runs(ob, dev, [90_000, 3000, 1], 4, steps=2, seed=22, tables=mode)


def test_noalloc_step_refuses_plans_beyond_its_scratch(dev):
    """A plan whose workspace exceeds the static array is refused before any
    buffer is touched (the buffers may then be anything, NULL included)."""
    import paper_2102_02888_amd as ob
    from paper_2102_02888_amd import _native
    L = _native.lib()
    plan = ob.Plan([1 << 27], 128)  # 131,072 tiles, (128 + 1) partial sums each
    assert plan.workspace_bytes > (96 << 20)
    vp = ctypes.c_void_p
    rc = L.onebit_step_noalloc(plan.handle, None, None, None, None, 0, plan.D, None, plan.D,
                               None, None, None, None, None, 1e-3, 0.9, 1e-8,
                               vp(torch.cuda.current_stream().cuda_stream))
    assert rc == -1 and b"scratch" in L.onebit_last_error()
    plan.close()


def test_noalloc_step_bert_large_matches_workspace_step(dev):
    """At the BERT-Large shape (d = 334,088,192, n = 32: an 86 MB workspace
    with the chunk owners' tables, inside the scratch array), two States fed
    one shared gradient tensor run 3 compression steps, one through
    onebit_step with its workspace and one through onebit_step_noalloc (fp32
    momentum first, then packed): every word, scale and element agrees bit for
    bit over all of d and all 32 rows."""
    import paper_2102_02888_amd as ob
    wl = synth.get("bert_large")
    plan = ob.Plan(wl.numel, wl.n)
    assert plan.workspace_bytes <= (96 << 20)
    ref = ob.State(plan, dev)
    new = ob.State(plan, dev, grads=ref.grads)
    scale_vec = torch.from_numpy(synth.grad_scale_per_element(wl, plan.D, plan.tensor_off)).to(dev)
    ref.x.copy_(synth.device_params(wl, plan.D, dev))
    synth.device_grads(wl, plan.D, plan.tensor_off, 1, ref.grads, scale_vec)
    ref.warmup(wl.lr, wl.beta1, wl.beta2, wl.eps, 1)
    for name in ("x", "m", "v"):
        getattr(new, name).copy_(getattr(ref, name))
    for t in (2, 3, 4):
        synth.device_grads(wl, plan.D, plan.tensor_off, t, ref.grads, scale_vec)
        packed = t > 2
        ref.step(wl.lr, wl.beta1, wl.eps)
        ob.onebit_step_noalloc(plan, new.x, None if packed else new.m, new.v, new.grads,
                               new.worker_err, new.server_err, new.worker_bits,
                               new.worker_scales, new.server_bits, new.server_scales, wl.lr,
                               wl.beta1, wl.eps)
        torch.cuda.synchronize()
        for name in NAMES:
            u, w = getattr(ref, name), getattr(new, name)
            if u.dtype == torch.float32:
                u, w = u.view(torch.int32), w.view(torch.int32)
            assert torch.equal(u, w), (t, name, int((u != w).sum()))
    del ref, new
    plan.close()
    torch.cuda.empty_cache()
