"""GPU path (through the C ABI) versus the CPU oracle, element by element.

Sizes here are small enough for the oracle to finish in seconds while still
spanning many 1024-element tiles, ragged tails, empty segments and every
entry point.  Bits, scales' routing and layout must match exactly; fp32
state within rel 1e-5 / abs 1e-6; scales within 1 ulp (counted).
"""
import numpy as np
import pytest
import torch

import oracle
import synth
from parity_util import check_bits, check_fp, check_scales, host

pytestmark = pytest.mark.gpu

LR, B1, B2, EPS = 1e-4, 0.9, 0.999, 1e-8


@pytest.fixture(scope="module")
def ob():
    import paper_2102_02888_amd as ob
    return ob


def _put(a, dev):
    t = torch.from_numpy(np.ascontiguousarray(a))
    if t.dtype == torch.uint64:
        t = t.view(torch.int64)
    return t.to(dev)


def _layouts_agree(plan, L):
    assert plan.D == L.D and plan.W == L.W and plan.S == L.S
    assert [int(c) for c in plan.chunk_len] == [L.chunk_len(k) for k in range(len(L.numel))]
    np.testing.assert_array_equal(plan.tensor_off, L.tensor_off)
    np.testing.assert_array_equal(plan.seg_begin, L.seg_begin)
    np.testing.assert_array_equal(plan.seg_end, L.seg_end)


# ---------------------------------------------------------------------------
# Layout / routing tables (integer, exact)
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("numel,n", [([1 << 20], 4), ([100, 1 << 20, 5, 0, 4097], 4),
                                     (synth.stress_sizes()[:500], 8), ([334_088_192], 32),
                                     ([334_088_192], 256), ([1], 1)])
def test_plan_layout_matches_oracle(ob, dev, numel, n):
    plan = ob.Plan(numel, n)
    _layouts_agree(plan, oracle.Layout(numel, n))
    assert plan.d == sum(numel)
    plan.close()


# ---------------------------------------------------------------------------
# Single-call parity with re-synced inputs
# ---------------------------------------------------------------------------

def _random_state(L, seed, n_rows):
    mask = L.real_mask()
    m = synth.host_normal(L.D, 1e-4, seed, 1)
    g = np.stack([synth.host_normal(L.D, 1e-3, seed, 2, i) for i in range(n_rows)])
    delta = np.stack([synth.host_normal(L.D, 3e-5, seed, 3, i) for i in range(n_rows)])
    x = synth.host_normal(L.D, 0.02, seed, 4)
    v = np.abs(synth.host_normal(L.D, 1e-7, seed, 5))
    dbar = synth.host_normal(L.D, 1e-5, seed, 6)
    for a in (m, x, v, dbar):
        a[~mask] = 0
    g[:, ~mask] = 0
    delta[:, ~mask] = 0
    return m, g, delta, x, v, dbar


CASES = [([1 << 20], 4), ([100, 5000, 64, 0, 4097, 1, 65, 1023, 1025], 3),
         ([3 * 1024 + 17, 70_000], 8), ([2048], 1)]


@pytest.mark.parametrize("numel,n", CASES)
def test_worker_compress_parity(ob, dev, numel, n):
    L = oracle.Layout(numel, n)
    plan = ob.Plan(numel, n)
    m, g, delta, *_ = _random_state(L, 10 + n, n)
    # GPU: explicit delta loaded as the error state with zero scales
    err = _put(delta, dev)
    bits = torch.zeros((n, L.W), dtype=torch.int64, device=dev)
    scales = torch.zeros((n, L.S), dtype=torch.float32, device=dev)
    ws = plan.workspace(dev)
    ob.onebit_worker_compress(plan, _put(m, dev), _put(g, dev), err, bits, scales, B1, ws)
    d_out = torch.zeros_like(err)
    ob.onebit_error_materialize(plan, err, scales, d_out)
    torch.cuda.synchronize()
    # oracle
    wbits = np.zeros((n, L.W), np.uint64)
    wscales = np.zeros((n, L.S), np.float32)
    z = np.zeros(L.D, np.float32)
    zs = np.zeros((n, L.D), np.float32)
    for i in range(n):
        for q, (b, e) in enumerate(L.segments()):
            wscales[i, q] = oracle.worker_segment(b, e, B1, m, g[i], delta[i], wbits[i], z)
        zs[i] = z
    mask = L.real_mask()
    check_bits("worker bits", host(bits), wbits)
    nscale = check_scales("worker scales", host(scales), wscales)
    check_fp("compensated z", host(err), zs, mask=mask)
    ex = check_fp("worker delta", host(d_out), delta, mask=mask)
    print("worker: scales off by 1 ulp: %d; delta bit-identical %.6f" % (nscale, ex))
    plan.close()


@pytest.mark.parametrize("numel,n", CASES)
def test_worker_compress_packed_momentum_parity(ob, dev, numel, n):
    """Momentum given as a message (sign words + segment scales): the worker
    pass decodes it; the oracle gets the decoded values as m."""
    L = oracle.Layout(numel, n)
    plan = ob.Plan(numel, n)
    _, g, delta, *_ = _random_state(L, 40 + n, n)
    rng = np.random.default_rng(40 + n)
    mbits = rng.integers(0, np.iinfo(np.uint64).max, size=L.W, dtype=np.uint64, endpoint=True)
    mscales = np.exp(rng.normal(-9, 1.0, size=L.S)).astype(np.float32)
    m = oracle.decode_message(L, mbits, mscales)
    err = _put(delta, dev)
    bits = torch.zeros((n, L.W), dtype=torch.int64, device=dev)
    scales = torch.zeros((n, L.S), dtype=torch.float32, device=dev)
    ws = plan.workspace(dev)
    ob.onebit_worker_compress(plan, None, _put(g, dev), err, bits, scales, B1, ws,
                              m_bits=_put(mbits, dev), m_scales=_put(mscales, dev))
    dec = torch.zeros(L.D, dtype=torch.float32, device=dev)
    ob.onebit_decode(plan, _put(mbits, dev), _put(mscales, dev), dec)
    torch.cuda.synchronize()
    wbits = np.zeros((n, L.W), np.uint64)
    wscales = np.zeros((n, L.S), np.float32)
    z = np.zeros(L.D, np.float32)
    zs = np.zeros((n, L.D), np.float32)
    for i in range(n):
        for q, (b, e) in enumerate(L.segments()):
            wscales[i, q] = oracle.worker_segment(b, e, B1, m, g[i], delta[i], wbits[i], z)
        zs[i] = z
    mask = L.real_mask()
    check_fp("decoded message", host(dec), m, rel=0, abs_=0, mask=mask)
    check_bits("worker bits", host(bits), wbits)
    check_scales("worker scales", host(scales), wscales)
    check_fp("compensated z", host(err), zs, mask=mask)
    plan.close()


SERVER_CASES = [c + ("lognormal",) for c in CASES] + [
    ([1 << 20], 4, "wide"), ([5000, 300, 64], 5, "wide"), ([70_000], 37, "lognormal"),
    ([70_000], 37, "zeros"), ([100_000], 256, "lognormal"), ([100_000], 256, "wide"),
    # n = 32: four groups of 8; n = 37 and 100: the split pass, whose last
    # group has 5 and 4 rows
    ([1 << 20], 32, "lognormal"), ([1 << 20], 4, "zeros"), ([300_000], 37, "lognormal"),
    ([300_000], 37, "wide"), ([300_000], 37, "zeros"), ([700_000], 100, "lognormal"),
    # 32 batches of 32 rows; chunks of 256 elements, 782 non-empty (tables of
    # all 1,000 segments would take 250 MB, so the plan keeps none)
    ([200_000], 1000, "lognormal"), ([200_000], 1000, "wide")]


@pytest.mark.parametrize("tables", ["on", "off"])
@pytest.mark.parametrize("numel,n,scales", SERVER_CASES)
def test_server_parity(ob, dev, numel, n, scales, tables):
    """Incoming scales 'lognormal' have a narrow exponent span (the grouped
    summation path); 'wide' spans ~80 binades (one-by-one path); 'zeros'
    mixes zero scales in.  tables 'on': the chunk owners' tables are built
    once per call in the workspace (every plan here reserves it); 'off': per
    tile."""
    L = oracle.Layout(numel, n)
    plan = ob.Plan(numel, n)
    plan.set_server_tables(ob.SERVER_TABLES_ON if tables == "on" else ob.SERVER_TABLES_OFF)
    *_, dbar = _random_state(L, 20 + n, n)
    rng = np.random.default_rng(n)
    wbits = rng.integers(0, np.iinfo(np.uint64).max, size=(n, L.W), dtype=np.uint64,
                         endpoint=True)
    wscales = np.exp(rng.normal(-7, 0.5, size=(n, L.S))).astype(np.float32)
    if scales == "wide":
        wscales *= np.float32(2.0) ** rng.integers(-40, 40, size=(n, L.S)).astype(np.float32)
    elif scales == "zeros":
        wscales[rng.random((n, L.S)) < 0.3] = 0
    serr = _put(dbar, dev)
    sbits = torch.zeros(L.W, dtype=torch.int64, device=dev)
    sscales = torch.zeros(L.S, dtype=torch.float32, device=dev)
    ws = plan.workspace(dev)
    ob.onebit_server_reduce_compress(plan, 0, n, _put(wbits, dev), _put(wscales, dev), serr,
                                     sbits, sscales, ws)
    d_out = torch.zeros_like(serr)
    ob.onebit_error_materialize(plan, serr, sscales, d_out, rows=1)
    torch.cuda.synchronize()
    ref_bits = np.zeros(L.W, np.uint64)
    ref_scales = np.zeros(L.S, np.float32)
    z = np.zeros(L.D, np.float32)
    for q, (b, e) in enumerate(L.segments()):
        ref_scales[q] = oracle.server_segment(b, e, n, wbits.reshape(-1), L.W,
                                              np.ascontiguousarray(wscales[:, q]), 1, dbar,
                                              ref_bits, z)
    mask = L.real_mask()
    check_bits("server bits", host(sbits), ref_bits)
    check_scales("server scales", host(sscales), ref_scales)
    check_fp("server z", host(serr), z, mask=mask)
    check_fp("server delta", host(d_out), dbar, mask=mask)
    plan.close()


@pytest.mark.parametrize("numel,n", CASES)
def test_update_parity(ob, dev, numel, n):
    L = oracle.Layout(numel, n)
    plan = ob.Plan(numel, n)
    _, _, _, x, v, _ = _random_state(L, 30 + n, 1)
    rng = np.random.default_rng(3)
    sbits = rng.integers(0, np.iinfo(np.uint64).max, size=L.W, dtype=np.uint64, endpoint=True)
    sscales = np.exp(rng.normal(-9, 1.0, size=L.S)).astype(np.float32)
    xg = _put(x, dev)
    mg = torch.zeros(L.D, dtype=torch.float32, device=dev)
    ob.onebit_decompress_update(plan, _put(sbits, dev), _put(sscales, dev), xg, mg,
                                _put(v, dev), LR, EPS)
    torch.cuda.synchronize()
    xr, mr = x.copy(), np.zeros(L.D, np.float32)
    for q, (b, e) in enumerate(L.segments()):
        oracle.update_segment(b, e, sbits, sscales[q], LR, EPS, xr, mr, v)
    ex = check_fp("x", host(xg), xr)
    check_fp("m", host(mg), mr, rel=0, abs_=0)
    print("update: x bit-identical fraction %.6f" % ex)
    plan.close()


@pytest.mark.parametrize("bias_correction", [0, 1])
def test_warmup_parity(ob, dev, bias_correction):
    numel, n = [100, 5000, 0, 70_001], 3
    L = oracle.Layout(numel, n)
    plan = ob.Plan(numel, n)
    wl = synth.Workload(name="w", numel=numel, n=n, warmup_steps=4, steps=0)
    x = synth.host_params(wl, L.D)
    x[~L.real_mask()] = 0
    m = np.zeros(L.D, np.float32)
    v = np.zeros(L.D, np.float32)
    xg, mg, vg = _put(x, dev), _put(m, dev), _put(v, dev)
    for t in range(1, 5):
        g = synth.host_grads(wl, L.D, L.tensor_off, t)
        oracle.warmup_step(L, x, m, v, g, n, LR, B1, B2, EPS, bias_correction, t)
        ob.onebit_warmup_adam_step(plan, xg, mg, vg, _put(g, dev), LR, B1, B2, EPS,
                                   bias_correction, t)
    torch.cuda.synchronize()
    for name, a, b in (("x", xg, x), ("m", mg, m), ("v", vg, v)):
        ex = check_fp(name, host(a), b)
        print("warm-up %s bit-identical %.6f" % (name, ex))
    plan.close()


# ---------------------------------------------------------------------------
# Free-running: warm-up then compression steps, no re-sync
# ---------------------------------------------------------------------------

def _lowp(g, dtype):
    """Gradients rounded to a 16-bit type: (device tensor of that type, the
    same values as exact fp32 numpy for the oracle)."""
    t = torch.from_numpy(np.ascontiguousarray(g)).to(dtype)
    return t, t.float().numpy()


def _free_run(ob, dev, wl, numel=None, warm=None, steps=None, packed=True,
              grad_dtype=torch.float32, perturb=None, final_check=None):
    numel = wl.numel if numel is None else numel
    n = wl.n
    warm = wl.warmup_steps if warm is None else warm
    steps = wl.steps if steps is None else steps
    L = oracle.Layout(numel, n)
    plan = ob.Plan(numel, n)
    _layouts_agree(plan, L)
    mask = L.real_mask()
    x = synth.host_params(wl, L.D)
    x[~mask] = 0
    m = np.zeros(L.D, np.float32)
    v = np.zeros(L.D, np.float32)
    st = ob.State(plan, dev, packed_momentum=packed, grad_dtype=grad_dtype)
    st.x.copy_(_put(x, dev))
    for t in range(1, warm + 1):
        g = synth.host_grads(wl, L.D, L.tensor_off, t)
        gt, g = _lowp(g, grad_dtype)
        oracle.warmup_step(L, x, m, v, g, n, wl.lr, wl.beta1, wl.beta2, wl.eps, 0, t)
        st.grads.copy_(gt.to(dev))
        st.warmup(wl.lr, wl.beta1, wl.beta2, wl.eps, t)
    torch.cuda.synchronize()
    check_fp("warm-up x", host(st.x), x)
    check_fp("warm-up m", host(st.m), m)
    check_fp("warm-up v (frozen)", host(st.v), v)
    ref = oracle.State(L, x, m, v)
    scale_ulps = 0
    for t in range(warm + 1, warm + steps + 1):
        g = synth.host_grads(wl, L.D, L.tensor_off, t)
        if perturb is not None:
            perturb(t - warm, g, L)
        gt, g = _lowp(g, grad_dtype)
        ref.step(g, wl.lr, wl.beta1, wl.eps)
        st.grads.copy_(gt.to(dev))
        st.step(wl.lr, wl.beta1, wl.eps)
        torch.cuda.synchronize()
        tag = "step %d" % (t - warm)
        check_bits(tag + " worker bits", host(st.worker_bits), ref.wbits)
        check_bits(tag + " server bits", host(st.server_bits), ref.sbits)
        scale_ulps += check_scales(tag + " worker scales", host(st.worker_scales), ref.wscales)
        scale_ulps += check_scales(tag + " server scales", host(st.server_scales), ref.sscales)
    ex = {}
    ex["x"] = check_fp("x", host(st.x), ref.x, mask=mask)
    ex["m"] = check_fp("m", host(st.momentum()), ref.m, mask=mask)
    ex["worker delta"] = check_fp("worker delta", host(st.worker_delta()), ref.delta, mask=mask)
    ex["server delta"] = check_fp("server delta", host(st.server_delta()), ref.delta_bar,
                                  mask=mask)
    print("%s: scales differing by 1 ulp: %d; bit-identical fractions %s"
          % (wl.name, scale_ulps, ex))
    if final_check is not None:
        final_check(st, ref, L)
    plan.close()
    return ex


@pytest.mark.parametrize("packed", [True, False])
def test_free_running_tiny(ob, dev, packed):
    """Tiny workload in full: d = 2^20, n = 4, 10 warm-up + 10 compression
    steps; momentum packed (decoded from the server message) or fp32."""
    _free_run(ob, dev, synth.get("tiny"), packed=packed)


@pytest.mark.parametrize("grad_dtype", [torch.bfloat16, torch.float16])
def test_free_running_tiny_16bit_grads(ob, dev, grad_dtype):
    """Tiny workload with 16-bit gradients (widened exactly to fp32)."""
    _free_run(ob, dev, synth.get("tiny"), grad_dtype=grad_dtype)


@pytest.mark.parametrize("grad_dtype", [torch.bfloat16, torch.float16])
def test_free_running_ragged_16bit_grads(ob, dev, grad_dtype):
    wl = synth.Workload(name="ragged16", numel=[1, 63, 64, 65, 0, 1000, 1025, 4097, 12345],
                        n=3, warmup_steps=2, steps=4)
    _free_run(ob, dev, wl, grad_dtype=grad_dtype)


def test_free_running_many_small_tensors(ob, dev):
    """The stress workload's first 400 tensors (per-tensor chunking, many
    empty and short segments), n = 8, 5 warm-up + 10 compression steps."""
    wl = synth.get("stress")
    _free_run(ob, dev, wl, numel=wl.numel[:400])


@pytest.mark.parametrize("packed", [True, False])
def test_free_running_ragged_edges(ob, dev, packed):
    wl = synth.Workload(name="ragged", numel=[1, 63, 64, 65, 0, 1000, 1024, 1025, 4097, 12345],
                        n=5, warmup_steps=3, steps=6)
    _free_run(ob, dev, wl, packed=packed)


def test_free_running_more_scale_pairs_than_grid(ob, dev):
    """4,202 small tensors with n = 64: 64 x 268,928 (worker, segment) scale
    reductions, more than one launch of the scale kernel covers in one pass
    (its grid strides), and 63 of every 64 segments empty."""
    wl = synth.Workload(name="pairs", numel=[64] * 4200 + [100, 3], n=64, warmup_steps=2,
                        steps=3)
    _free_run(ob, dev, wl)


def test_free_running_nonfinite_gradients(ob, dev):
    """A NaN and an infinity in two workers' gradients at the second
    compression step: the affected segments turn non-finite the same way on
    both sides (NaN scales take the one-by-one server path), the others stay
    finite and equal."""
    wl = synth.Workload(name="nonfinite", numel=[5000, 3000, 700], n=4, warmup_steps=2,
                        steps=4)

    def perturb(step, g, L):
        if step == 2:
            g[1, L.tensor_off[0] + 17] = np.nan
            g[2, L.tensor_off[1] + 900] = np.inf

    def final_check(st, ref, L):
        # the two hit segments went non-finite, the third tensor did not
        # element 900 of tensor 1 is in its chunk 1 (chunks of 768): segment n + 1
        assert np.isnan(ref.sscales[0]) and not np.isfinite(ref.sscales[wl.n + 1])
        assert np.isfinite(ref.sscales[2 * wl.n:]).all()
        assert np.isnan(host(st.x)[L.tensor_off[0]:L.tensor_off[0] + 64]).all()
        assert np.isfinite(host(st.x)[L.tensor_off[2]:L.tensor_off[2] + 700]).all()

    _free_run(ob, dev, wl, perturb=perturb, final_check=final_check)


def test_free_running_single_worker(ob, dev):
    wl = synth.Workload(name="n1", numel=[70_000, 33], n=1, warmup_steps=2, steps=5)
    _free_run(ob, dev, wl)


def test_identical_workers_on_gpu(ob, dev):
    """n identical workers: server bits equal worker bits and the server
    error stays zero (a property the paper's averaging fixes)."""
    numel, n = [50_000], 4
    plan = ob.Plan(numel, n)
    st = ob.State(plan, dev)
    L = oracle.Layout(numel, n)
    st.m.copy_(_put(synth.host_normal(L.D, 1e-4, 8), dev))
    st.v.fill_(1e-8)
    for t in range(3):
        g = synth.host_normal(L.D, 1e-3, 9, t)
        st.grads.copy_(_put(np.repeat(g[None], n, 0), dev))
        st.step(LR, B1, EPS)
    torch.cuda.synchronize()
    wb = host(st.worker_bits)
    for i in range(1, n):
        check_bits("row %d" % i, wb[i], wb[0])
    check_bits("server", host(st.server_bits), wb[0])
    assert not host(st.server_delta()).any()
    plan.close()


def test_deterministic(ob, dev):
    numel, n = [200_000, 3000], 4
    outs = []
    for _ in range(2):
        plan = ob.Plan(numel, n)
        st = ob.State(plan, dev)
        L = oracle.Layout(numel, n)
        st.m.copy_(_put(synth.host_normal(L.D, 1e-4, 8), dev))
        st.v.fill_(1e-8)
        for t in range(3):
            st.grads.copy_(_put(np.stack([synth.host_normal(L.D, 1e-3, 9, t, i)
                                          for i in range(n)]), dev))
            st.step(LR, B1, EPS)
        torch.cuda.synchronize()
        outs.append([host(a).copy() for a in (st.x, st.worker_err, st.worker_scales,
                                             st.server_bits, st.server_scales)])
        plan.close()
    for a, b in zip(*outs):
        assert a.tobytes() == b.tobytes()


# ---------------------------------------------------------------------------
# Real-share server input form: a received buffer of one chunk
# ---------------------------------------------------------------------------

def test_server_received_chunk_form(ob, dev):
    """Rows of only chunk j's words (bits_word_base) and one scale per row
    (scales_seg_base) give the same result as the full simulated rows."""
    numel, n, j = [130_000], 8, 5
    L = oracle.Layout(numel, n)
    plan = ob.Plan(numel, n)
    rng = np.random.default_rng(4)
    wbits = rng.integers(0, np.iinfo(np.uint64).max, size=(n, L.W), dtype=np.uint64,
                         endpoint=True)
    wscales = np.exp(rng.normal(-7, 0.5, size=(n, L.S))).astype(np.float32)
    b, e = L.seg_begin[j], L.seg_end[j]
    w0, w1 = b // 64, (e + 63) // 64
    recv_bits = np.ascontiguousarray(wbits[:, w0:w1])
    recv_scales = np.ascontiguousarray(wscales[:, j])
    res = []
    for form in ("full", "received"):
        serr = torch.zeros(L.D, dtype=torch.float32, device=dev)
        sbits = torch.zeros(L.W, dtype=torch.int64, device=dev)
        sscales = torch.zeros(L.S, dtype=torch.float32, device=dev)
        ws = plan.workspace(dev)
        if form == "full":
            ob.onebit_server_reduce_compress(plan, j, j + 1, _put(wbits, dev),
                                             _put(wscales, dev), serr, sbits, sscales, ws)
        else:
            ob.onebit_server_reduce_compress(plan, j, j + 1, _put(recv_bits, dev),
                                             _put(recv_scales, dev), serr, sbits, sscales, ws,
                                             bits_word_base=w0, scales_seg_base=j, scales_ld=1)
        torch.cuda.synchronize()
        res.append((host(serr), host(sbits), host(sscales)))
    for a, c in zip(res[0], res[1]):
        assert a.tobytes() == c.tobytes()
    # only chunk j's words and scale were written
    sb = res[0][1]
    assert not sb[:w0].any() and not sb[w1:].any()
    assert np.count_nonzero(res[0][2]) == 1
    plan.close()


@pytest.mark.parametrize("numel,n,scales", [
    ([1 << 20], 4, "lognormal"), ([1 << 20], 32, "lognormal"), ([1 << 20], 32, "wide"),
    ([300_000], 37, "zeros"), ([700_000], 100, "lognormal"), ([600_000, 3000, 70], 8, "zeros"),
    ([1 << 23], 32, "lognormal")])
def test_server_tables_and_per_tile_paths_agree(ob, dev, numel, n, scales):
    """The chunk owners' lookup tables built once per call in the workspace
    (ON), built per tile (OFF) and the default choice (AUTO: the workspace for
    the 2^23-element case, 8,192 tiles x 4 groups) give the same words, scales
    and error state, bit for bit (both sums are exact, or both one by one)."""
    L = oracle.Layout(numel, n)
    plan = ob.Plan(numel, n)
    rng = np.random.default_rng(40 + n)
    wbits = rng.integers(0, np.iinfo(np.uint64).max, size=(n, L.W), dtype=np.uint64,
                         endpoint=True)
    wscales = np.exp(rng.normal(-7, 0.5, size=(n, L.S))).astype(np.float32)
    if scales == "wide":
        wscales *= np.float32(2.0) ** rng.integers(-40, 40, size=(n, L.S)).astype(np.float32)
    elif scales == "zeros":
        wscales[rng.random((n, L.S)) < 0.3] = 0
    serr0 = rng.normal(0, 1e-3, size=L.D).astype(np.float32)
    sscales0 = np.exp(rng.normal(-8, 0.5, size=L.S)).astype(np.float32)
    wb, ws_ = _put(wbits, dev), _put(wscales, dev)
    with pytest.raises(ob.OnebitError):
        plan.set_server_tables(3)
    res = []
    for mode in (ob.SERVER_TABLES_ON, ob.SERVER_TABLES_OFF, ob.SERVER_TABLES_AUTO):
        plan.set_server_tables(mode)
        serr = _put(serr0, dev)
        sscales = _put(sscales0, dev)
        sbits = torch.zeros(L.W, dtype=torch.int64, device=dev)
        ws = plan.workspace(dev)
        ob.onebit_server_reduce_compress(plan, 0, n, wb, ws_, serr, sbits, sscales, ws)
        torch.cuda.synchronize()
        res.append((host(serr), host(sbits), host(sscales)))
    for other in res[1:]:
        for name, a, c in zip(("server_err", "server_bits", "server_scales"), res[0], other):
            assert a.tobytes() == c.tobytes(), name
    plan.close()


def test_hand_worked_example_on_gpu(ob, dev):
    """The two hand-worked compression steps of tests/golden/ through the
    ABI (first step with the fp32 momentum, second with it packed)."""
    import json
    import os
    gd = json.load(open(os.path.join(os.path.dirname(__file__), "golden",
                                     "hand_worked_two_steps.json")))
    su = gd["setup"]
    plan = ob.Plan(su["tensor_numel"], su["n_workers"])
    st = ob.State(plan, dev)
    st.x[:2] = torch.tensor(su["x"])
    st.m[:2] = torch.tensor(su["m"])
    st.v[:2] = torch.tensor(su["v_frozen"])
    for sd in gd["steps"]:
        st.grads.zero_()
        st.grads[:, :2] = torch.tensor(sd["grads"])
        st.step(su["lr"], su["beta1"], su["eps"])
        torch.cuda.synchronize()
        assert host(st.worker_scales)[:, 0].tolist() == sd["worker_scales_chunk0"]
        assert [int(w) for w in host(st.worker_bits)[:, 0]] == sd["worker_bits_word0"]
        assert host(st.worker_delta())[:, :2].tolist() == sd["worker_delta"]
        assert float(host(st.server_scales)[0]) == sd["server_scale_chunk0"]
        assert int(host(st.server_bits)[0]) == sd["server_bits_word0"]
        assert host(st.server_delta())[:2].tolist() == sd["server_delta"]
        assert host(st.x)[:2].tolist() == sd["x"]
        assert host(st.momentum())[:2].tolist() == sd["m"]
    plan.close()


def test_eps_placement_on_gpu(ob, dev):
    """tests/golden/eps_placement.json through the ABI: the warm-up divides by
    sqrt(v) + eps, the compression update by sqrt(v_frozen + eps), exactly."""
    import json
    import os
    gd = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "eps_placement.json")))
    su = gd["warmup"]
    k = su["tensor_numel"][0]
    plan = ob.Plan(su["tensor_numel"], su["n_workers"])
    st = ob.State(plan, dev)
    st.x[:k] = torch.tensor(su["x"])
    for t, sd in enumerate(su["steps"], start=1):
        st.grads.zero_()
        st.grads[:, :k] = torch.tensor(sd["grads"])
        st.warmup(su["lr"], su["beta1"], su["beta2"], su["eps"], t,
                  bias_correction=su["bias_correction"])
        torch.cuda.synchronize()
        assert host(st.m)[:k].tolist() == sd["m"]
        assert host(st.v)[:k].tolist() == sd["v"]
        assert host(st.x)[:k].tolist() == sd["x"]
    plan.close()
    su = gd["compression"]
    plan = ob.Plan(su["tensor_numel"], su["n_workers"])
    st = ob.State(plan, dev)
    st.x[:2] = torch.tensor(su["x"])
    st.m[:2] = torch.tensor(su["m"])
    st.v[:2] = torch.tensor(su["v_frozen"])
    for sd in su["steps"]:
        st.grads.zero_()
        st.grads[:, :2] = torch.tensor(sd["grads"])
        st.step(su["lr"], su["beta1"], su["eps"])
        torch.cuda.synchronize()
        assert float(host(st.server_scales)[0]) == sd["server_scale_chunk0"]
        assert int(host(st.server_bits)[0]) == sd["server_bits_word0"]
        assert host(st.x)[:2].tolist() == sd["x"]
        assert host(st.momentum())[:2].tolist() == sd["m"]
    # the update call alone, from the first step's message
    x = torch.zeros(plan.D, dtype=torch.float32, device=dev)
    x[:2] = torch.tensor(su["x"])
    bits = torch.zeros(plan.W, dtype=torch.int64, device=dev)
    bits[0] = su["steps"][0]["server_bits_word0"]
    scales = torch.zeros(plan.S, dtype=torch.float32, device=dev)
    scales[0] = su["steps"][0]["server_scale_chunk0"]
    ob.onebit_decompress_update(plan, bits, scales, x, None, st.v, su["lr"], su["eps"])
    torch.cuda.synchronize()
    assert host(x)[:2].tolist() == su["steps"][0]["x"]
    plan.close()


def _random_config(seed):
    rng = np.random.default_rng(1000 + seed)
    k = int(rng.integers(1, 21))
    numel = [int(v) for v in np.exp(rng.uniform(0, np.log(50_000), size=k)).astype(np.int64)]
    numel[int(rng.integers(0, k))] = 0 if k > 1 else numel[0]
    n = int(rng.choice([1, 2, 3, 5, 8, 16, 33]))
    packed = bool(rng.integers(0, 2))
    gdt = [torch.float32, torch.bfloat16, torch.float16][int(rng.integers(0, 3))]
    return numel, n, packed, gdt


@pytest.mark.parametrize("seed", range(8))
def test_free_running_random_configs(ob, dev, seed):
    """Seeded random layouts (1-20 tensors of 1-50,000 elements, one of them
    possibly empty), worker counts, momentum forms and gradient types."""
    numel, n, packed, gdt = _random_config(seed)
    wl = synth.Workload(name="random%d" % seed, numel=numel, n=n, warmup_steps=2, steps=3,
                        seed_grads=50 + seed)
    _free_run(ob, dev, wl, packed=packed, grad_dtype=gdt)
