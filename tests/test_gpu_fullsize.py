"""Parity at the benchmark's full sizes, in the launch configuration bench.py
times, on sampled segments.

The GPU runs every step over the whole buffer; the oracle free-runs the same
seeded inputs on a few whole segments (each segment is an independent
parameter-server problem, so its history needs only its own slice of the
inputs).  Inputs are drawn on the device by the seeded generators and copied
to the host for the oracle; nothing the GPU path computes is fed to the oracle.
"""
import numpy as np
import pytest
import torch

import oracle
import synth
from parity_util import SegmentOracle, check_bits, check_fp, check_scales, host

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def ob():
    import paper_2102_02888_amd as ob
    return ob


def _np(t):
    if t.dtype in (torch.bfloat16, torch.float16):
        t = t.float()
    return np.ascontiguousarray(t.detach().cpu().numpy())


def _check_segments(st, so, mom=None, wdelta=None, sdelta=None, final=True):
    """Device state against the oracle on every sampled segment: sign words
    bit for bit, scales within 1 ulp, fp32 state within the tolerance."""
    for sg in so.segs:
        q, b, e = sg["q"], sg["b"], sg["e"]
        w0, w1 = b // 64, (e + 63) // 64
        check_bits("worker bits seg %d" % q, host(st.worker_bits[:so.n, w0:w1]), sg["wbits"])
        check_bits("server bits seg %d" % q, host(st.server_bits[w0:w1]), sg["sbits"])
        check_scales("worker scales seg %d" % q, host(st.worker_scales[:so.n, q]), sg["wscales"])
        check_scales("server scale seg %d" % q, host(st.server_scales[q:q + 1]),
                     np.array([sg["sscale"]], np.float32))
        if not final:
            continue
        check_fp("x seg %d" % q, _np(st.x[b:e]), sg["x"])
        check_fp("m seg %d" % q, _np(mom[b:e]), sg["m"])
        check_fp("worker delta seg %d" % q, _np(wdelta[:so.n, b:e]), sg["delta"])
        if sdelta is not None:
            check_fp("server delta seg %d" % q, _np(sdelta[b:e]), sg["dbar"])


def _free_run_sampled(ob, dev, wl, warm, steps, sample_segs, grad_dtype=torch.float32):
    """`warm` Adam warm-up steps, then `steps` compression steps through
    State.step (the fused onebit_step, packed momentum from the second
    compression step on: the launch configuration bench.py times), checked
    against the oracle on whole sampled segments after the warm-up, after
    every step (sign words and scales) and at the end (all fp32 state)."""
    n = wl.n
    plan = ob.Plan(wl.numel, n)
    L = oracle.Layout(wl.numel, n)
    assert (plan.D, plan.W, plan.S) == (L.D, L.W, L.S)
    np.testing.assert_array_equal(plan.seg_begin, L.seg_begin)
    np.testing.assert_array_equal(plan.seg_end, L.seg_end)
    st = ob.State(plan, dev, grad_dtype=grad_dtype)
    scale_vec = torch.from_numpy(synth.grad_scale_per_element(wl, plan.D, plan.tensor_off)).to(dev)
    st.x.copy_(synth.device_params(wl, plan.D, dev))
    so = SegmentOracle(L, sample_segs, lambda b, e: _np(st.x[b:e]), n)
    grads = lambda b, e: _np(st.grads[:, b:e])
    try:
        for t in range(1, warm + 1):
            synth.device_grads(wl, plan.D, plan.tensor_off, t, st.grads, scale_vec)
            so.warmup(grads, t, wl.lr, wl.beta1, wl.beta2, wl.eps)
            st.warmup(wl.lr, wl.beta1, wl.beta2, wl.eps, t)
        torch.cuda.synchronize()
        for sg in so.segs:
            b, e = sg["b"], sg["e"]
            check_fp("warm-up x seg %d" % sg["q"], _np(st.x[b:e]), sg["x"])
            check_fp("warm-up m seg %d" % sg["q"], _np(st.m[b:e]), sg["m"])
            check_fp("warm-up v seg %d" % sg["q"], _np(st.v[b:e]), sg["v"])
        for t in range(warm + 1, warm + steps + 1):
            synth.device_grads(wl, plan.D, plan.tensor_off, t, st.grads, scale_vec)
            so.step(grads, wl.lr, wl.beta1, wl.eps)
            st.step(wl.lr, wl.beta1, wl.eps)
            torch.cuda.synchronize()
            _check_segments(st, so, final=False)
            print("%s step %d ok" % (wl.name, t), flush=True)
        assert st.momentum_is_packed() == (steps > 1)
        wdelta = st.worker_delta()
        sdelta = st.server_delta()
        mom = st.momentum()
        torch.cuda.synchronize()
        _check_segments(st, so, mom, wdelta, sdelta)
        del wdelta, sdelta, mom
    finally:
        so.close()
        del st
        plan.close()
        torch.cuda.empty_cache()


def test_bert_large_full_size(ob, dev):
    """d = 334,088,192, n = 32, 5 warm-up + 10 compression steps: the first,
    a middle and the last of the 32 chunks."""
    wl = synth.get("bert_large")
    _free_run_sampled(ob, dev, wl, warm=wl.warmup_steps, steps=10, sample_segs=[0, 15, 31])


def test_bert_large_full_size_bf16_grads(ob, dev):
    """BERT-Large with bfloat16 gradients (the paper trains in 16-bit), 5
    warm-up + 10 compression steps: chunk 7."""
    wl = synth.get("bert_large")
    _free_run_sampled(ob, dev, wl, warm=wl.warmup_steps, steps=10, sample_segs=[7],
                      grad_dtype=torch.bfloat16)


def test_bert_base_full_size_fp16_grads(ob, dev):
    """BERT-Base with float16 gradients, 5 warm-up + 10 compression steps:
    the per-tensor gradient scale puts many of them in fp16's subnormal
    range, which the widening keeps exact: chunk 3."""
    wl = synth.get("bert_base")
    _free_run_sampled(ob, dev, wl, warm=wl.warmup_steps, steps=10, sample_segs=[3],
                      grad_dtype=torch.float16)


def test_bert_base_full_size(ob, dev):
    """d = 108,888,576, n = 16, 5 warm-up + 10 compression steps: the first,
    a middle and the last (short) chunk."""
    wl = synth.get("bert_base")
    _free_run_sampled(ob, dev, wl, warm=wl.warmup_steps, steps=10, sample_segs=[0, 7, 15])


def test_stress_full_size(ob, dev):
    """All 5,000 tensors (per-tensor chunking, n = 8), 5 warm-up + 10
    compression steps: segments of the smallest, a median, the largest and
    the last tensor, each tensor's first and last non-empty chunk."""
    wl = synth.get("stress")
    L = oracle.Layout(wl.numel, wl.n)
    order = np.argsort(wl.numel)
    picks = []
    for k in [int(order[0]), int(order[len(order) // 2]), int(order[-1]), 4999]:
        for j in range(wl.n):
            q = k * wl.n + j
            if L.seg_end[q] > L.seg_begin[q]:
                last = q
                if j == 0:
                    picks.append(q)
        picks.append(last)
    _free_run_sampled(ob, dev, wl, warm=wl.warmup_steps, steps=10,
                      sample_segs=sorted(set(picks)))


def test_share256_full_size(ob, dev):
    """One GPU's share of a 256-worker BERT-Large run at its real shape, in
    bench.py's calls: 5 warm-up steps of the local worker, then 10
    compression steps (fp32 momentum first, then packed), each with the
    local worker over all d, the owner of chunk 0 reducing 256 incoming
    packed chunks (synthetic, seeded per step), and the update over all d
    with the other 255 gathered chunks synthetic as well."""
    wl = synth.get("share256")
    n, j = wl.n, wl.server_chunk
    plan = ob.Plan(wl.numel, n)
    L = oracle.Layout(wl.numel, n)
    D, W, S = plan.D, plan.W, plan.S
    st = ob.State(plan, dev, n_local=1)
    scale_vec = torch.from_numpy(synth.grad_scale_per_element(wl, D, plan.tensor_off)).to(dev)
    st.x.copy_(synth.device_params(wl, D, dev))
    so = SegmentOracle(L, [0, 77, 255], lambda b, e: _np(st.x[b:e]), 1)
    grads = lambda b, e: _np(st.grads[:, b:e])
    b0, e0 = int(L.seg_begin[j]), int(L.seg_end[j])
    cw0, cw1 = b0 // 64, (e0 + 63) // 64
    assert cw0 == 0 and S == n  # one flat tensor: segment q is chunk q
    try:
        for t in range(1, wl.warmup_steps + 1):
            synth.device_grads(wl, D, plan.tensor_off, t, st.grads, scale_vec)
            so.warmup(grads, t, wl.lr, wl.beta1, wl.beta2, wl.eps)
            st.warmup(wl.lr, wl.beta1, wl.beta2, wl.eps, t)
        torch.cuda.synchronize()
        for sg in so.segs:
            check_fp("warm-up x seg %d" % sg["q"], _np(st.x[sg["b"]:sg["e"]]), sg["x"])
            check_fp("warm-up v seg %d" % sg["q"], _np(st.v[sg["b"]:sg["e"]]), sg["v"])
        for k in range(10):
            t = wl.warmup_steps + 1 + k
            synth.device_grads(wl, D, plan.tensor_off, t, st.grads, scale_vec)
            so.workers(grads, wl.beta1)
            if k == 0:
                ob.onebit_worker_compress(plan, st.m, st.grads, st.worker_err, st.worker_bits,
                                          st.worker_scales, wl.beta1, st.workspace)
            else:
                ob.onebit_worker_compress(plan, None, st.grads, st.worker_err, st.worker_bits,
                                          st.worker_scales, wl.beta1, st.workspace,
                                          m_bits=st.server_bits, m_scales=st.server_scales)
            recv_bits, recv_scales = synth.device_bits_and_scales(n, cw1 - cw0,
                                                                  wl.seed_incoming + 2 * t, dev)
            ob.onebit_server_reduce_compress(plan, j, j + 1, recv_bits, recv_scales,
                                             st.server_err, st.server_bits, st.server_scales,
                                             st.workspace, bits_word_base=cw0,
                                             scales_seg_base=j, scales_ld=1)
            # what the all-gather brings for the other 255 chunks this step
            gbits, _ = synth.device_bits_and_scales(1, W - cw1, wl.seed_incoming + 2 * t + 1, dev)
            _, gscales = synth.device_bits_and_scales(S - 1, 1, wl.seed_incoming + 2 * t + 1, dev)
            st.server_bits[cw1:] = gbits[0]
            st.server_scales[j + 1:] = gscales
            ob.onebit_decompress_update(plan, st.server_bits, st.server_scales, st.x, None, st.v,
                                        wl.lr, wl.eps)
            sbits_h, sscales_h = host(st.server_bits), _np(st.server_scales)
            gathered = {sg["q"]: (sbits_h[sg["b"] // 64:(sg["e"] + 63) // 64], sscales_h[sg["q"]])
                        for sg in so.segs if sg["q"] != j}
            so.owners_and_updates(wl.lr, wl.eps, received={j: (host(recv_bits), _np(recv_scales))},
                                  gathered=gathered)
            torch.cuda.synchronize()
            _check_segments(st, so, final=False)
            print("share256 step %d ok" % t, flush=True)
        wdelta = st.worker_delta()
        sdelta = st.server_delta()
        mom = torch.zeros_like(st.m)
        ob.onebit_decode(plan, st.server_bits, st.server_scales, mom)
        torch.cuda.synchronize()
        # the server error exists only for the owned chunk
        _check_segments(st, so, mom, wdelta, None)
        sg0 = so.segs[0]
        assert sg0["q"] == j
        check_fp("server delta chunk %d" % j, _np(sdelta[b0:e0]), sg0["dbar"])
        del wdelta, sdelta, mom
    finally:
        so.close()
        del st
        plan.close()
        torch.cuda.empty_cache()


def test_bert_large_two_states_bitwise(ob, dev):
    """Two States fed identical BERT-Large inputs (one shared gradient
    tensor) run 3 compression steps, the first with the fp32 momentum
    (k_worker_rows at its full grid) and two packed: every sign word, scale
    and element of x and both error states agree bit for bit over all of d
    and all 32 rows.  A regression test of run-to-run determinism at the
    benchmark's grid size."""
    wl = synth.get("bert_large")
    plan = ob.Plan(wl.numel, wl.n)
    a = ob.State(plan, dev)
    b = ob.State(plan, dev, grads=a.grads)
    scale_vec = torch.from_numpy(synth.grad_scale_per_element(wl, plan.D, plan.tensor_off)).to(dev)
    a.x.copy_(synth.device_params(wl, plan.D, dev))
    synth.device_grads(wl, plan.D, plan.tensor_off, 1, a.grads, scale_vec)
    a.warmup(wl.lr, wl.beta1, wl.beta2, wl.eps, 1)
    for name in ("x", "m", "v"):
        getattr(b, name).copy_(getattr(a, name))
    names = ("x", "worker_err", "worker_bits", "worker_scales", "server_err", "server_bits",
             "server_scales")
    for t in (2, 3, 4):
        synth.device_grads(wl, plan.D, plan.tensor_off, t, a.grads, scale_vec)
        a.step(wl.lr, wl.beta1, wl.eps)
        b.step(wl.lr, wl.beta1, wl.eps)
        torch.cuda.synchronize()
        for name in names:
            u, w = getattr(a, name), getattr(b, name)
            if u.dtype == torch.float32:
                u, w = u.view(torch.int32), w.view(torch.int32)
            same = torch.equal(u, w)
            if not same:
                diff = int((u != w).sum())
                raise AssertionError("step %d: %s differs in %d of %d elements"
                                     % (t, name, diff, u.numel()))
    del a, b
    plan.close()
    torch.cuda.empty_cache()


def _random_message(plan, seed):
    rng = np.random.default_rng(seed)
    bits = rng.integers(0, np.iinfo(np.uint64).max, size=plan.W, dtype=np.uint64, endpoint=True)
    scales = np.exp(rng.normal(-9, 1.0, size=plan.S)).astype(np.float32)
    return bits, scales


def test_decode_full_size_exact(ob, dev):
    """Every element of a BERT-Large-sized message decoded exactly, twice
    (a regression test: a wave that loads after a non-temporal store has been
    seen to read wrong data on this hardware)."""
    wl = synth.get("bert_large")
    plan = ob.Plan(wl.numel, wl.n)
    L = oracle.Layout(wl.numel, wl.n)
    bits, scales = _random_message(plan, 11)
    ref = oracle.decode_message(L, bits, scales)
    bt = torch.from_numpy(bits.view(np.int64)).to(dev)
    sc = torch.from_numpy(scales).to(dev)
    for rep in range(2):
        out = torch.zeros(plan.D, dtype=torch.float32, device=dev)
        ob.onebit_decode(plan, bt, sc, out)
        torch.cuda.synchronize()
        check_fp("decode rep %d" % rep, _np(out), ref, rel=0, abs_=0)
        del out
    plan.close()
    torch.cuda.empty_cache()


def test_update_full_size_exact(ob, dev):
    """The decompress + update over all d = 334,088,192 elements against the
    oracle, element by element."""
    wl = synth.get("bert_large")
    plan = ob.Plan(wl.numel, wl.n)
    L = oracle.Layout(wl.numel, wl.n)
    bits, scales = _random_message(plan, 12)
    x = synth.host_normal(plan.D, 0.02, 12, 1)
    v = np.abs(synth.host_normal(plan.D, 1e-7, 12, 2))
    xg = torch.from_numpy(x).to(dev)
    mg = torch.zeros(plan.D, dtype=torch.float32, device=dev)
    ob.onebit_decompress_update(plan, torch.from_numpy(bits.view(np.int64)).to(dev),
                                torch.from_numpy(scales).to(dev), xg, mg,
                                torch.from_numpy(v).to(dev), wl.lr, wl.eps)
    torch.cuda.synchronize()
    m = np.zeros(plan.D, np.float32)
    for q, (b, e) in enumerate(L.segments()):
        oracle.update_segment(b, e, bits, scales[q], wl.lr, wl.eps, x, m, v)
    check_fp("x", _np(xg), x, rel=0, abs_=0)
    check_fp("m", _np(mg), m, rel=0, abs_=0)
    del xg, mg
    plan.close()
    torch.cuda.empty_cache()


def test_first_step_over_two_launch_pieces(ob, dev):
    """The first compression step's kernel (two waves per tile) is launched
    over at most 2^22 tiles at a time.  One tensor of 2^22 + 3 tiles (a short
    last tile), n = 1: the step runs as two launches.  The error state starts
    at zero, so every element's new compensated value must be the first step's
    z = fl(beta1 m) + fl((1 - beta1) g) (Algorithm 1's momentum step with a
    zero error); an element processed twice or not at all would differ.  A
    plain fp32 torch reference checks all 4.3e9 elements, in chunks; the sign
    words around the boundary between the launches and the segment's scale
    are checked too.  (The step's update overwrites m with the decoded server
    message, so the reference uses a copy of m taken before the step.)  Needs
    about 125 GB of device memory."""
    torch.cuda.empty_cache()
    tiles = (1 << 22) + 3
    d = tiles * 1024 - 100
    plan = ob.Plan([d], 1)
    assert plan.T == tiles
    st = ob.State(plan, dev)
    gen = torch.Generator(device=dev)
    gen.manual_seed(2102)
    st.m[:d].normal_(0.0, 1e-3, generator=gen)
    st.grads[0, :d].normal_(0.0, 1e-2, generator=gen)
    st.v[:d].uniform_(1e-8, 1e-6, generator=gen)
    beta1, lr, eps = 0.9, 1e-4, 1e-8
    m0 = st.m.clone()
    st.step(lr, beta1, eps)  # first compression step: fp32 momentum, k_worker_rows
    torch.cuda.synchronize()
    b1 = torch.tensor(beta1, dtype=torch.float32, device=dev)
    omb1 = torch.tensor(1.0, dtype=torch.float32, device=dev) - b1
    chunk = 1 << 28
    sq = torch.zeros((), dtype=torch.float64, device=dev)
    for c0 in range(0, plan.D, chunk):
        c1 = min(plan.D, c0 + chunk)
        z = b1 * m0[c0:c1] + omb1 * st.grads[0, c0:c1]
        got = st.worker_err[0, c0:c1]
        bad = int((got != z).sum())
        assert bad == 0, "%d elements of [%d, %d) differ from the first step's z" % (bad, c0, c1)
        sq += (z.double() ** 2).sum()
        del z, got
    # sign words of the tiles on both sides of the boundary between the launches
    t0, t1 = (1 << 22) - 2, (1 << 22) + 2
    zb = (b1 * m0[t0 * 1024:t1 * 1024] + omb1 * st.grads[0, t0 * 1024:t1 * 1024]).cpu().numpy()
    want = np.packbits((zb >= 0).reshape(-1, 64)[:, ::-1], axis=1).view(">u8").ravel()
    got_w = host(st.worker_bits[0, t0 * 16:t1 * 16]).view(np.uint64)
    np.testing.assert_array_equal(got_w, want.astype(np.uint64))
    scale = float(np.sqrt(float(sq) / d).astype(np.float32))
    assert abs(float(st.worker_scales[0, 0]) - scale) <= 1e-6 * scale
    del st, m0
    plan.close()
    torch.cuda.empty_cache()
