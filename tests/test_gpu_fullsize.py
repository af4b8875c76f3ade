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
from parity_util import check_bits, check_fp, check_scales, host

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def ob():
    import paper_2102_02888_amd as ob
    return ob


def _np(t):
    if t.dtype in (torch.bfloat16, torch.float16):
        t = t.float()
    return np.ascontiguousarray(t.detach().cpu().numpy())


def _free_run_sampled(ob, dev, wl, warm, steps, sample_segs, grad_dtype=torch.float32):
    n = wl.n
    plan = ob.Plan(wl.numel, n)
    L = oracle.Layout(wl.numel, n)
    assert (plan.D, plan.W, plan.S) == (L.D, L.W, L.S)
    np.testing.assert_array_equal(plan.seg_begin, L.seg_begin)
    np.testing.assert_array_equal(plan.seg_end, L.seg_end)
    st = ob.State(plan, dev, grad_dtype=grad_dtype)
    scale_vec = torch.from_numpy(synth.grad_scale_per_element(wl, plan.D, plan.tensor_off)).to(dev)
    st.x.copy_(synth.device_params(wl, plan.D, dev))
    segs = []
    for q in sample_segs:
        b, e = int(L.seg_begin[q]), int(L.seg_end[q])
        assert e > b
        segs.append(dict(q=q, b=b, e=e, ln=e - b, x=_np(st.x[b:e]),
                         m=np.zeros(e - b, np.float32), v=np.zeros(e - b, np.float32)))
    for t in range(1, warm + 1):
        synth.device_grads(wl, plan.D, plan.tensor_off, t, st.grads, scale_vec)
        for sg in segs:
            g = _np(st.grads[:, sg["b"]:sg["e"]])
            oracle.warmup_range(0, sg["ln"], sg["x"], sg["m"], sg["v"], g, sg["ln"], n,
                                wl.lr, wl.beta1, wl.beta2, wl.eps, 0, t)
        st.warmup(wl.lr, wl.beta1, wl.beta2, wl.eps, t)
    torch.cuda.synchronize()
    for sg in segs:
        b, e = sg["b"], sg["e"]
        check_fp("warm-up x seg %d" % sg["q"], _np(st.x[b:e]), sg["x"])
        check_fp("warm-up v seg %d" % sg["q"], _np(st.v[b:e]), sg["v"])
        nw = (sg["ln"] + 63) // 64
        sg.update(delta=np.zeros((n, sg["ln"]), np.float32), dbar=np.zeros(sg["ln"], np.float32),
                  wbits=np.zeros((n, nw), np.uint64), wscales=np.zeros(n, np.float32),
                  sbits=np.zeros(nw, np.uint64), z=np.zeros(sg["ln"], np.float32))
    for t in range(warm + 1, warm + steps + 1):
        synth.device_grads(wl, plan.D, plan.tensor_off, t, st.grads, scale_vec)
        for sg in segs:
            g = _np(st.grads[:, sg["b"]:sg["e"]])
            for i in range(n):
                sg["wscales"][i] = oracle.worker_segment(0, sg["ln"], wl.beta1, sg["m"], g[i],
                                                         sg["delta"][i], sg["wbits"][i], sg["z"])
            del g
            sg["sscale"] = oracle.server_segment(0, sg["ln"], n, sg["wbits"].reshape(-1),
                                                 sg["wbits"].shape[1], sg["wscales"], 1,
                                                 sg["dbar"], sg["sbits"], sg["z"])
            oracle.update_segment(0, sg["ln"], sg["sbits"], sg["sscale"], wl.lr, wl.eps,
                                  sg["x"], sg["m"], sg["v"])
        st.step(wl.lr, wl.beta1, wl.eps)
    torch.cuda.synchronize()
    wdelta = st.worker_delta()
    sdelta = st.server_delta()
    mom = st.momentum()
    torch.cuda.synchronize()
    for sg in segs:
        q, b, e = sg["q"], sg["b"], sg["e"]
        w0, w1 = b // 64, (e + 63) // 64
        check_bits("worker bits seg %d" % q, host(st.worker_bits[:, w0:w1]), sg["wbits"])
        check_bits("server bits seg %d" % q, host(st.server_bits[w0:w1]), sg["sbits"])
        check_scales("worker scales seg %d" % q, host(st.worker_scales[:, q]), sg["wscales"])
        check_scales("server scale seg %d" % q, host(st.server_scales[q:q + 1]),
                     np.array([sg["sscale"]], np.float32))
        check_fp("x seg %d" % q, _np(st.x[b:e]), sg["x"])
        check_fp("m seg %d" % q, _np(mom[b:e]), sg["m"])
        check_fp("worker delta seg %d" % q, _np(wdelta[:, b:e]), sg["delta"])
        check_fp("server delta seg %d" % q, _np(sdelta[b:e]), sg["dbar"])
    del wdelta, sdelta, mom, st
    plan.close()
    torch.cuda.empty_cache()


def test_bert_large_full_size(ob, dev):
    """d = 334,088,192, n = 32: first and last of the 32 chunks."""
    _free_run_sampled(ob, dev, synth.get("bert_large"), warm=2, steps=2, sample_segs=[0, 31])


def test_bert_large_full_size_bf16_grads(ob, dev):
    """BERT-Large with bfloat16 gradients (the paper trains in 16-bit): chunk 7."""
    _free_run_sampled(ob, dev, synth.get("bert_large"), warm=1, steps=2, sample_segs=[7],
                      grad_dtype=torch.bfloat16)


def test_bert_base_full_size_fp16_grads(ob, dev):
    """BERT-Base with float16 gradients: the per-tensor gradient scale puts
    many of them in fp16's subnormal range, which the widening keeps exact:
    chunk 3."""
    _free_run_sampled(ob, dev, synth.get("bert_base"), warm=1, steps=2, sample_segs=[3],
                      grad_dtype=torch.float16)


def test_bert_base_full_size(ob, dev):
    """d = 108,888,576, n = 16: the last chunk is the short one."""
    _free_run_sampled(ob, dev, synth.get("bert_base"), warm=2, steps=3, sample_segs=[0, 15])


def test_stress_full_size(ob, dev):
    """All 5,000 tensors (per-tensor chunking, n = 8): a few segments of
    small, medium and large tensors, including a tensor's short last chunk."""
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
    _free_run_sampled(ob, dev, wl, warm=2, steps=3, sample_segs=sorted(set(picks)))


def test_share256_full_size(ob, dev):
    """One GPU's share of a 256-worker BERT-Large step at its real shape: the
    local worker over all d, the owner of chunk 0 reducing 256 incoming
    packed chunks (synthetic, seeded), and the update over all d with the
    other 255 gathered chunks synthetic as well."""
    wl = synth.get("share256")
    n, j = wl.n, wl.server_chunk
    plan = ob.Plan(wl.numel, n)
    L = oracle.Layout(wl.numel, n)
    D, W = plan.D, plan.W
    st = ob.State(plan, dev, n_local=1)
    scale_vec = torch.from_numpy(synth.grad_scale_per_element(wl, D, plan.tensor_off)).to(dev)
    st.x.copy_(synth.device_params(wl, D, dev))
    sample = [0, 77, 255]
    segs = {q: dict(b=int(L.seg_begin[q]), e=int(L.seg_end[q])) for q in sample}
    for q, sg in segs.items():
        sg["ln"] = sg["e"] - sg["b"]
        sg["x"] = _np(st.x[sg["b"]:sg["e"]])
        sg["m"] = np.zeros(sg["ln"], np.float32)
        sg["v"] = np.zeros(sg["ln"], np.float32)
    warm = 2
    for t in range(1, warm + 1):
        synth.device_grads(wl, D, plan.tensor_off, t, st.grads, scale_vec)
        for sg in segs.values():
            g = _np(st.grads[:, sg["b"]:sg["e"]])
            oracle.warmup_range(0, sg["ln"], sg["x"], sg["m"], sg["v"], g, sg["ln"], 1,
                                wl.lr, wl.beta1, wl.beta2, wl.eps, 0, t)
        st.warmup(wl.lr, wl.beta1, wl.beta2, wl.eps, t)
    # one compression step
    synth.device_grads(wl, D, plan.tensor_off, warm + 1, st.grads, scale_vec)
    ob.onebit_worker_compress(plan, st.m, st.grads, st.worker_err, st.worker_bits,
                              st.worker_scales, wl.beta1, st.workspace)  # first step: fp32 m
    b0, e0 = int(L.seg_begin[j]), int(L.seg_end[j])
    cw0, cw1 = b0 // 64, (e0 + 63) // 64
    recv_bits, recv_scales = synth.device_bits_and_scales(n, cw1 - cw0, wl.seed_incoming, dev)
    # what the all-gather would bring for the other chunks
    gath_bits, gath_scales = synth.device_bits_and_scales(1, W, wl.seed_incoming + 1, dev)
    st.server_bits.copy_(gath_bits[0])
    st.server_scales.copy_(gath_scales.expand(plan.S) * torch.linspace(0.5, 1.5, plan.S, device=dev))
    # the owned chunk's scale is part of the server error state: zero at the
    # first compression step, like the zero server error buffer
    st.server_scales[j] = 0.0
    ob.onebit_server_reduce_compress(plan, j, j + 1, recv_bits, recv_scales, st.server_err,
                                     st.server_bits, st.server_scales, st.workspace,
                                     bits_word_base=cw0, scales_seg_base=j, scales_ld=1)
    x_before_update = {q: _np(st.x[sg["b"]:sg["e"]]) for q, sg in segs.items()}
    ob.onebit_decompress_update(plan, st.server_bits, st.server_scales, st.x, st.m, st.v,
                                wl.lr, wl.eps)
    torch.cuda.synchronize()
    # oracle: the local worker on the sampled segments
    gh = {q: _np(st.grads[0, sg["b"]:sg["e"]]) for q, sg in segs.items()}
    for q, sg in segs.items():
        nw = (sg["ln"] + 63) // 64
        delta = np.zeros(sg["ln"], np.float32)
        bits = np.zeros(nw, np.uint64)
        z = np.zeros(sg["ln"], np.float32)
        s = oracle.worker_segment(0, sg["ln"], wl.beta1, sg["m"], gh[q], delta, bits, z)
        w0, w1 = sg["b"] // 64, (sg["e"] + 63) // 64
        check_bits("worker bits seg %d" % q, host(st.worker_bits[0, w0:w1]), bits)
        check_scales("worker scale seg %d" % q, host(st.worker_scales[0, q:q + 1]),
                     np.array([s], np.float32))
        sg["delta"] = delta
        check_fp("warm-up x seg %d" % q, x_before_update[q], sg["x"])
        check_fp("v seg %d" % q, _np(st.v[sg["b"]:sg["e"]]), sg["v"])
    # oracle: the owner of chunk j from the received rows
    rb = host(recv_bits).copy()
    rs = _np(recv_scales)
    ln0 = e0 - b0
    dbar = np.zeros(ln0, np.float32)
    sb = np.zeros(cw1 - cw0, np.uint64)
    z = np.zeros(ln0, np.float32)
    s_bar = oracle.server_segment(0, ln0, n, rb.reshape(-1), cw1 - cw0, rs, 1, dbar, sb, z)
    check_bits("server bits chunk %d" % j, host(st.server_bits[cw0:cw1]), sb)
    check_scales("server scale chunk %d" % j, host(st.server_scales[j:j + 1]),
                 np.array([s_bar], np.float32))
    check_fp("server delta chunk %d" % j, _np(st.server_delta()[b0:e0]), dbar)
    # oracle: the update on the sampled segments with the gathered words
    sbits_all = host(st.server_bits)
    sscales_all = _np(st.server_scales)
    for q, sg in segs.items():
        w0, w1 = sg["b"] // 64, (sg["e"] + 63) // 64
        x = x_before_update[q].copy()
        m = np.zeros(sg["ln"], np.float32)
        oracle.update_segment(0, sg["ln"], np.ascontiguousarray(sbits_all[w0:w1]),
                              sscales_all[q], wl.lr, wl.eps, x, m, sg["v"])
        check_fp("x seg %d" % q, _np(st.x[sg["b"]:sg["e"]]), x)
        check_fp("m seg %d" % q, _np(st.m[sg["b"]:sg["e"]]), m)
    del st
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
