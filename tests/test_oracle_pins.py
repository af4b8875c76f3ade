"""Pins the CPU oracle to what the paper and the mathematics fix.

Each test checks the oracle against something other than itself: a closed
form, a library routine (numpy's bit packing and norms, torch.optim.Adam and
torch.optim.SGD), an identity the paper proves, a hand-worked example with
exactly representable numbers, or a special case that reduces to a textbook
method.  A plausible slip in the oracle (a dropped error term, a wrong sign,
a transposed bit order, eps in the wrong place, a wrong chunk cut) fails at
least one of them.
"""
import math

import numpy as np
import pytest

import oracle
import synth

BETA1, BETA2, EPS, LR = 0.9, 0.999, 1e-8, 1e-4


def assert_close_scaled(a, b, rel):
    """|a - b| <= rel * (|b| + mean|b|): relative, with a floor at the typical
    magnitude so that fp32 cancellation in tiny entries is not flagged."""
    a = np.asarray(a, np.float64); b = np.asarray(b, np.float64)
    tol = rel * (np.abs(b) + np.abs(b).mean())
    bad = np.abs(a - b) > tol
    assert not bad.any(), (int(bad.sum()), float(np.abs(a - b).max()))


def ulp32(a):
    a = np.abs(np.asarray(a, np.float32))
    return np.spacing(a).astype(np.float64)


# ---------------------------------------------------------------------------
# Layout: chunk cut of each tensor into n chunks (64-aligned), segments
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("numel,n", [([1], 1), ([100, 1 << 20, 5], 4), ([64, 65, 128, 129, 4096], 8),
                                     ([0, 7, 0, 1000], 3), ([10_000], 256)])
def test_layout_brute_force(numel, n):
    L = oracle.Layout(numel, n)
    off = 0
    for k, d in enumerate(numel):
        assert L.tensor_off[k] == off
        assert off % 64 == 0
        c = L.chunk_len(k)
        assert c % 64 == 0
        if d:
            # the smallest 64-multiple c with n*c >= d
            assert n * c >= d and (c == 64 or n * (c - 64) < d)
        # brute force: element r of tensor k belongs to chunk r // c
        for j in range(n):
            b, e = L.seg_begin[k * n + j], L.seg_end[k * n + j]
            members = [r for r in range(d) if c and r // c == j] if d <= 20000 else None
            if members is not None:
                if members:
                    assert (b, e) == (off + members[0], off + members[-1] + 1)
                else:
                    assert b == e
            assert (b - off) % 64 == 0 or b == e
        off += 64 * ((d + 63) // 64)
    assert L.D == off and L.W * 64 == L.D


def test_layout_bert_large_chunks():
    wl = synth.get("bert_large")
    L = oracle.Layout(wl.numel, wl.n)
    assert wl.d == 334_088_192 and L.D == wl.d
    assert L.chunk_len(0) == 10_440_256 == wl.d // 32
    wb = synth.get("bert_base")
    assert wb.d == 108_888_576
    assert sum(int(np.prod(s)) for s, _ in synth.bert_tensor_shapes(24, 1024, 4096)) == wl.d
    assert len(synth.bert_tensor_shapes(24, 1024, 4096)) == 386
    assert len(synth.bert_tensor_shapes(12, 768, 3072)) == 194
    s = synth.get("share256")
    Ls = oracle.Layout(s.numel, s.n)
    assert Ls.chunk_len(0) == 1_305_088
    assert Ls.seg_end[255] - Ls.seg_begin[255] == 1_290_752


# ---------------------------------------------------------------------------
# The compression operator: bit order, sign convention, scale
# ---------------------------------------------------------------------------

def test_bits_match_numpy_packbits():
    rng = np.random.default_rng(5)
    for length in [1, 63, 64, 65, 200, 4096 + 17]:
        z = rng.standard_normal(length).astype(np.float32)
        z[:: 7] = 0.0
        z[3 % length] = -0.0
        bits, _ = oracle.compress(z)
        ref = np.packbits(z >= 0, bitorder="little")
        ref = np.concatenate([ref, np.zeros(len(bits) * 8 - len(ref), np.uint8)])
        assert bits.view(np.uint8).tobytes() == ref.tobytes()


def test_sign_convention_zero_nan_padding():
    z = np.array([0.0, -0.0, np.nan, -1.0, 1.0], np.float32)
    bits, s = oracle.compress(z)
    assert int(bits[0]) == 0b10011  # +0 -> 1, -0 -> 1, NaN -> 0, -1 -> 0, 1 -> 1
    assert np.isnan(s)
    # padding bits beyond the segment are zero
    z = np.ones(70, np.float32)
    bits, _ = oracle.compress(z)
    assert int(bits[1]) == (1 << 6) - 1


def test_scale_same_l2_magnitude():
    rng = np.random.default_rng(7)
    for length in [1, 2, 3, 64, 1000, 262_144]:
        z = (rng.standard_normal(length) * rng.uniform(1e-6, 10)).astype(np.float32)
        bits, s = oracle.compress(z)
        norm = np.linalg.norm(z.astype(np.float64))
        # ||C[z]||_2 = s * sqrt(len) equals ||z||_2 up to fp32 rounding of s
        assert abs(float(s) - norm / math.sqrt(length)) <= 0.5 * ulp32(s) * 1.0001
    # an l1 (mean |z|) scale would differ on a non-constant vector
    z = np.array([3.0, 4.0], np.float32)
    _, s = oracle.compress(z)
    assert s == np.float32(math.sqrt(12.5))


def test_empty_segment_scale_zero():
    z = np.ones(10, np.float32)
    bits = np.zeros(1, np.uint64)
    assert oracle.lib().orc_compress(5, 5, z, bits) == 0.0
    assert int(bits[0]) == 0


# ---------------------------------------------------------------------------
# Hand-worked two-step example (Algorithm 1, exact dyadic arithmetic; the
# inputs, results and derivation are in tests/golden/hand_worked_two_steps.json)
# ---------------------------------------------------------------------------

def _golden(name):
    import json
    import os
    return json.load(open(os.path.join(os.path.dirname(__file__), "golden", name)))


def test_hand_worked_two_steps():
    """tests/golden/hand_worked_two_steps.json: two compression steps of
    Algorithm 1 worked by hand in exact dyadic arithmetic."""
    gd = _golden("hand_worked_two_steps.json")
    su = gd["setup"]
    L = oracle.Layout(su["tensor_numel"], su["n_workers"])
    assert L.D == 64 and L.segments() == [(0, 2), (2, 2)]
    x = np.zeros(64, np.float32); x[:2] = su["x"]
    m = np.zeros(64, np.float32); m[:2] = su["m"]
    v = np.zeros(64, np.float32); v[:2] = su["v_frozen"]
    st = oracle.State(L, x, m, v)
    g = np.zeros((2, 64), np.float32)
    for sd in gd["steps"]:
        g[:, :2] = sd["grads"]
        st.step(g, lr=su["lr"], beta1=su["beta1"], eps=su["eps"])
        np.testing.assert_array_equal(st.wscales[:, 0], sd["worker_scales_chunk0"])
        np.testing.assert_array_equal(st.wscales[:, 1], [0, 0])
        assert [int(w) for w in st.wbits[:, 0]] == sd["worker_bits_word0"]
        np.testing.assert_array_equal(st.delta[:, :2], sd["worker_delta"])
        assert st.sscales[0] == sd["server_scale_chunk0"] and st.sscales[1] == 0
        assert int(st.sbits[0]) == sd["server_bits_word0"]
        np.testing.assert_array_equal(st.delta_bar[:2], sd["server_delta"])
        np.testing.assert_array_equal(st.x[:2], sd["x"])
        np.testing.assert_array_equal(st.m[:2], sd["m"])
    # padding untouched
    assert not st.x[2:].any() and not st.delta[:, 2:].any()


def test_eps_placement_warmup():
    """tests/golden/eps_placement.json, warm-up part: eq. (alg:v) divides by
    sqrt(v) + eps; the hand-worked values differ from sqrt(v + eps)'s."""
    su = _golden("eps_placement.json")["warmup"]
    L = oracle.Layout(su["tensor_numel"], su["n_workers"])
    k = su["tensor_numel"][0]
    x = np.zeros(L.D, np.float32); x[:k] = su["x"]
    m = np.zeros(L.D, np.float32); m[:k] = su["m"]
    v = np.zeros(L.D, np.float32); v[:k] = su["v"]
    g = np.zeros((su["n_workers"], L.D), np.float32)
    for t, sd in enumerate(su["steps"], start=1):
        g[:, :k] = sd["grads"]
        oracle.warmup_step(L, x, m, v, g, su["n_workers"], su["lr"], su["beta1"], su["beta2"],
                           su["eps"], su["bias_correction"], t)
        np.testing.assert_array_equal(m[:k], sd["m"])
        np.testing.assert_array_equal(v[:k], sd["v"])
        np.testing.assert_array_equal(x[:k], sd["x"])
    # the other placement of eps would move x[0] to 1 - 0.5/sqrt(2) at step 1
    assert su["steps"][0]["x"][0] != np.float32(1 - 0.5 / np.sqrt(2.0))


def test_eps_placement_compression_update():
    """tests/golden/eps_placement.json, compression part: Algorithm 1's final
    step divides the decoded momentum by sqrt(v_frozen + eps)."""
    su = _golden("eps_placement.json")["compression"]
    L = oracle.Layout(su["tensor_numel"], su["n_workers"])
    x = np.zeros(L.D, np.float32); x[:2] = su["x"]
    m = np.zeros(L.D, np.float32); m[:2] = su["m"]
    v = np.zeros(L.D, np.float32); v[:2] = su["v_frozen"]
    st = oracle.State(L, x, m, v)
    g = np.zeros((su["n_workers"], L.D), np.float32)
    for sd in su["steps"]:
        g[:, :2] = sd["grads"]
        st.step(g, lr=su["lr"], beta1=su["beta1"], eps=su["eps"])
        assert st.sscales[0] == sd["server_scale_chunk0"]
        assert int(st.sbits[0]) == sd["server_bits_word0"]
        np.testing.assert_array_equal(st.x[:2], sd["x"])
        np.testing.assert_array_equal(st.m[:2], sd["m"])
    # and the update alone, from the first step's message: sqrt(v + eps) = [2, 4]
    x1 = np.array(su["x"], np.float32)
    oracle.update_segment(0, 2, np.array([3], np.uint64), 13.0, su["lr"], su["eps"], x1,
                          None, np.array(su["v_frozen"], np.float32))
    np.testing.assert_array_equal(x1, su["steps"][0]["x"])


# ---------------------------------------------------------------------------
# Error-feedback identity and telescoping (appendix "Proof to the updating form")
# ---------------------------------------------------------------------------

def _run_compression(numel, n, steps, seed=11, start_m=None):
    wl = synth.Workload(name="t", numel=numel, n=n, warmup_steps=0, steps=steps, seed_grads=seed)
    L = oracle.Layout(numel, n)
    x = synth.host_params(wl, L.D)
    m = synth.host_normal(L.D, 1e-4, seed, 99) if start_m is None else start_m
    v = np.abs(synth.host_normal(L.D, 1e-6, seed, 98))
    mask = L.real_mask()
    x[~mask] = 0; m[~mask] = 0; v[~mask] = 0
    return wl, L, oracle.State(L, x, m, v)


def test_error_feedback_identity_worker_and_server():
    wl, L, st = _run_compression([5000, 300], 4, 0)
    z = np.zeros(L.D, np.float32)
    for t in range(3):
        g = synth.host_grads(wl, L.D, L.tensor_off, t)
        for i in range(L.n):
            for q, (b, e) in enumerate(L.segments()):
                delta_prev = st.delta[i].copy()
                s = oracle.worker_segment(b, e, BETA1, st.m, g[i], st.delta[i], st.wbits[i], z)
                st.wscales[i, q] = s
                dec = np.array([oracle.decode(st.wbits[i], idx, s) for idx in range(b, e)], np.float64)
                zz = z[b:e].astype(np.float64)
                # C[z] + delta_new == z, up to one rounding of the subtraction
                err = np.abs(dec + st.delta[i, b:e] - zz)
                assert np.all(err <= 0.5 * np.maximum(ulp32(zz), ulp32(s)))
                assert not np.array_equal(delta_prev[b:e], st.delta[i, b:e]) or e == b
        for q, (b, e) in enumerate(L.segments()):
            s = oracle.server_segment(b, e, L.n, st.wbits.reshape(-1), L.W,
                                      np.ascontiguousarray(st.wscales[:, q]), 1,
                                      st.delta_bar, st.sbits, z)
            dec = np.array([oracle.decode(st.sbits, idx, s) for idx in range(b, e)], np.float64)
            err = np.abs(dec + st.delta_bar[b:e] - z[b:e].astype(np.float64))
            assert np.all(err <= 0.5 * np.maximum(ulp32(z[b:e]), ulp32(s)))
            st.sscales[q] = s
            oracle.update_segment(b, e, st.sbits, s, LR, EPS, st.x, st.m, st.v)


@pytest.mark.parametrize("n", [1, 3, 4])
def test_telescoping_update_form(n):
    """m_t = beta1 m_{t-1} + (1-beta1) g_avg_t + Delta_{t-1} - Delta_t with
    Delta_t = mean_i delta_t^(i) + delta_bar_t, checked in float64."""
    wl, L, st = _run_compression([3000, 130, 64], n, 6)
    mask = L.real_mask()
    Delta_prev = np.zeros(L.D)
    for t in range(6):
        g = synth.host_grads(wl, L.D, L.tensor_off, t)
        m_prev = st.m.astype(np.float64)
        st.step(g, LR, BETA1, EPS)
        Delta = st.delta.astype(np.float64).mean(0) + st.delta_bar
        rhs = BETA1 * m_prev + (1 - BETA1) * g.astype(np.float64).mean(0) + Delta_prev - Delta
        mag = np.maximum.reduce([np.abs(m_prev), np.abs(st.m), np.abs(Delta), np.abs(Delta_prev),
                                 np.abs(g).max(0) * (1 - BETA1)])
        assert np.all(np.abs(st.m - rhs)[mask] <= 16 * 2.0 ** -24 * mag[mask] + 1e-30)
        Delta_prev = Delta
    # the errors carry real information: dropping them breaks the identity
    assert np.abs(Delta_prev[mask]).max() > 1e-6


# ---------------------------------------------------------------------------
# Special cases
# ---------------------------------------------------------------------------

def test_identical_workers_server_is_passthrough():
    """n identical workers: the server average equals one worker's decoded
    message, server bits equal worker bits, the server error stays zero."""
    wl, L, st = _run_compression([4096, 1000], 4, 0)
    for t in range(4):
        g1 = synth.host_grads(wl, L.D, L.tensor_off, t, workers=[0])
        g = np.repeat(g1, L.n, axis=0)
        st.step(g, LR, BETA1, EPS)
        for i in range(1, L.n):
            np.testing.assert_array_equal(st.wbits[i], st.wbits[0])
            np.testing.assert_array_equal(st.wscales[i], st.wscales[0])
        np.testing.assert_array_equal(st.sbits, st.wbits[0])
        np.testing.assert_array_equal(st.sscales, st.wscales[0, :])
        assert not st.delta_bar.any()


def test_single_worker():
    wl, L, st = _run_compression([777, 64], 1, 0)
    for t in range(3):
        st.step(synth.host_grads(wl, L.D, L.tensor_off, t), LR, BETA1, EPS)
        np.testing.assert_array_equal(st.sbits, st.wbits[0])
        np.testing.assert_array_equal(st.sscales, st.wscales[0])
        assert not st.delta_bar.any()


def test_chunk_independence():
    """Each segment is an independent parameter-server problem: running the
    per-segment pieces on a segment copied out alone gives the same bits."""
    wl, L, st = _run_compression([3000, 200], 3, 0)
    g = synth.host_grads(wl, L.D, L.tensor_off, 0)
    before = (st.x.copy(), st.m.copy(), st.v.copy())
    st.step(g, LR, BETA1, EPS)
    z = np.zeros(L.D, np.float32)
    for q, (b, e) in enumerate(L.segments()):
        ln = e - b
        if ln == 0:
            continue
        W = (ln + 63) // 64
        wb = np.zeros((L.n, W), np.uint64)
        ws = np.zeros(L.n, np.float32)
        for i in range(L.n):
            d_i = np.zeros(ln, np.float32)
            ws[i] = oracle.worker_segment(0, ln, BETA1, np.ascontiguousarray(before[1][b:e]),
                                          np.ascontiguousarray(g[i, b:e]), d_i, wb[i], z)
            np.testing.assert_array_equal(d_i, st.delta[i, b:e])
        assert np.array_equal(ws, st.wscales[:, q])
        np.testing.assert_array_equal(wb, st.wbits[:, b // 64:b // 64 + W])
        db = np.zeros(ln, np.float32)
        sb = np.zeros(W, np.uint64)
        s = oracle.server_segment(0, ln, L.n, wb.reshape(-1), W, ws, 1, db, sb, z)
        assert s == st.sscales[q]
        np.testing.assert_array_equal(sb, st.sbits[b // 64:b // 64 + W])
        x = before[0][b:e].copy(); m = np.zeros(ln, np.float32)
        oracle.update_segment(0, ln, sb, s, LR, EPS, x, m, np.ascontiguousarray(before[2][b:e]))
        np.testing.assert_array_equal(x, st.x[b:e])


def test_message_volume():
    """One sign bit per element plus one fp32 scale per segment: about 1/32
    of the fp32 volume (the paper's 97% reduction versus fp32)."""
    wl = synth.get("bert_large")
    L = oracle.Layout(wl.numel, wl.n)
    packed = L.W * 8 + 4 * L.S
    assert packed / (4 * wl.d) < 0.0313
    assert 1 - packed / (4 * wl.d) > 0.968


# ---------------------------------------------------------------------------
# Warm-up: textbook Adam (library) and the paper's no-bias-correction form
# ---------------------------------------------------------------------------

def _torch_adam_trajectory(x0, gbar_steps, lr, b1, b2, eps, bias_correction):
    import torch
    p = torch.nn.Parameter(torch.from_numpy(x0.astype(np.float64)).clone())
    opt = torch.optim.Adam([p], lr=lr, betas=(b1, b2), eps=eps, foreach=False)
    for t, gb in enumerate(gbar_steps, start=1):
        if not bias_correction:
            # torch always divides by bc1 and bc2; undo it with per-step lr, eps
            bc1, bc2 = 1 - b1 ** t, 1 - b2 ** t
            opt.param_groups[0]["lr"] = lr * bc1 / math.sqrt(bc2)
            opt.param_groups[0]["eps"] = eps / math.sqrt(bc2)
        p.grad = torch.from_numpy(gb.astype(np.float64))
        opt.step()
    st = opt.state[p]
    return p.detach().numpy(), st["exp_avg"].numpy(), st["exp_avg_sq"].numpy()


@pytest.mark.parametrize("bias_correction", [1, 0])
def test_warmup_matches_torch_adam(bias_correction):
    wl = synth.get("tiny")
    L = oracle.Layout([5000], 4)
    x = synth.host_params(wl, L.D)
    x0 = x.copy()
    m = np.zeros(L.D, np.float32); v = np.zeros(L.D, np.float32)
    gbars = []
    for t in range(1, 11):
        g = synth.host_grads(wl, L.D, L.tensor_off, t)
        gbars.append(g.astype(np.float64).mean(0))
        oracle.warmup_step(L, x, m, v, g, 4, LR, BETA1, BETA2, EPS, bias_correction, t)
    # the oracle's hyperparameters are binary32; give torch the same values
    f = lambda a: float(np.float32(a))
    xr, mr, vr = _torch_adam_trajectory(x0[:5000], [gb[:5000] for gb in gbars],
                                        f(LR), f(BETA1), f(BETA2), f(EPS), bias_correction)
    assert_close_scaled(m[:5000], mr, 1e-5)
    assert_close_scaled(v[:5000], vr, 1e-5)
    assert_close_scaled(x[:5000] - x0[:5000], xr - x0[:5000], 1e-4)
    # the update is not negligible relative to the tolerance
    assert np.abs(x[:5000] - x0[:5000]).max() > 1e-4


def test_warmup_constant_gradient_closed_form():
    """Constant gradient g: m_t = (1-beta1^t) g, v_t = (1-beta2^t) g^2 and
    x_t = x_0 - lr sum_s m_s / (sqrt(v_s) + eps) (no bias correction)."""
    L = oracle.Layout([256], 1)
    gc = np.linspace(-2e-3, 2e-3, 256).astype(np.float32)
    x = np.ones(256, np.float32); m = np.zeros(256, np.float32); v = np.zeros(256, np.float32)
    g64 = gc.astype(np.float64)
    b1, b2, lr, eps = (float(np.float32(a)) for a in (BETA1, BETA2, LR, EPS))
    acc = np.zeros(256)
    for t in range(1, 9):
        oracle.warmup_step(L, x, m, v, gc[None, :].copy(), 1, LR, BETA1, BETA2, EPS, 0, t)
        mt = (1 - b1 ** t) * g64
        vt = (1 - b2 ** t) * g64 ** 2
        acc += mt / (np.sqrt(vt) + eps)
        np.testing.assert_allclose(m, mt, rtol=4e-6, atol=1e-30)
        np.testing.assert_allclose(v, vt, rtol=4e-6, atol=1e-30)
        np.testing.assert_allclose(x, 1 - lr * acc, rtol=1e-6, atol=1e-7)


def test_warmup_gradient_average_over_workers():
    """n identical gradient rows average to that row exactly."""
    L = oracle.Layout([300], 5)
    g = synth.host_normal(320, 1e-3, 4)
    g[300:] = 0
    xa, ma, va = (np.ones(320, np.float32), np.zeros(320, np.float32), np.zeros(320, np.float32))
    xb, mb, vb = xa.copy(), ma.copy(), va.copy()
    oracle.warmup_step(L, xa, ma, va, np.repeat(g[None], 5, 0), 5, LR, BETA1, BETA2, EPS, 0, 1)
    oracle.warmup_step(L, xb, mb, vb, g[None].copy(), 1, LR, BETA1, BETA2, EPS, 0, 1)
    np.testing.assert_array_equal(xa, xb)
    np.testing.assert_array_equal(ma, mb)


# ---------------------------------------------------------------------------
# Identity compressor: momentum SGD with the frozen preconditioner
# ---------------------------------------------------------------------------

def test_identity_compressor_is_preconditioned_momentum_sgd():
    import torch
    n = 3
    L = oracle.Layout([4000], n)
    wl = synth.Workload(name="t", numel=[4000], n=n, warmup_steps=0, steps=5, seed_grads=21)
    x = synth.host_params(wl, L.D)
    m = synth.host_normal(L.D, 1e-4, 21, 1)
    v = np.abs(synth.host_normal(L.D, 1e-6, 21, 2))
    p = 1.0 / np.sqrt(v[:4000].astype(np.float64) + EPS)
    # change of variables y = x / p turns the preconditioned step into plain SGD
    y = torch.nn.Parameter(torch.from_numpy(x[:4000].astype(np.float64) / p))
    f = lambda a: float(np.float32(a))
    opt = torch.optim.SGD([y], lr=f(LR), momentum=f(BETA1), dampening=f(BETA1), foreach=False)
    opt.state[y]["momentum_buffer"] = torch.from_numpy(m[:4000].astype(np.float64)).clone()
    for t in range(5):
        g = synth.host_grads(wl, L.D, L.tensor_off, t)
        oracle.step_uncompressed(L, x, m, v, g, LR, BETA1, EPS)
        y.grad = torch.from_numpy(g[:, :4000].astype(np.float64).mean(0))
        opt.step()
    assert_close_scaled(m[:4000], opt.state[y]["momentum_buffer"].numpy(), 1e-5)
    assert_close_scaled(x[:4000], y.detach().numpy() * p, 1e-6)


# ---------------------------------------------------------------------------
# Exact rational references (fractions.Fraction): the oracle's fp64 paths
# give the correctly rounded fp32 value of the exact quantity
# ---------------------------------------------------------------------------

def _nearest_f32(q):
    """The fp32 value nearest to the rational q (ties to even mantissa)."""
    from fractions import Fraction
    c = np.float32(float(q))
    cands = [np.nextafter(c, np.float32(-np.inf)), c, np.nextafter(c, np.float32(np.inf))]
    best = min(cands, key=lambda a: (abs(Fraction(float(a)) - q),
                                     int(np.float32(a).view(np.uint32)) & 1))
    return np.float32(best)


def _sqrt_nearest_f32(q):
    """The fp32 value nearest to sqrt(q) for a rational q >= 0, decided
    exactly: sqrt(q) lies below the midpoint mid of two neighbours iff
    q < mid^2."""
    from fractions import Fraction
    c = np.float32(math.sqrt(float(q)))
    lo = np.nextafter(c, np.float32(-np.inf))
    hi = np.nextafter(c, np.float32(np.inf))
    pts = [lo, c, hi]
    # walk to the pair of neighbours that brackets sqrt(q)
    best = c
    for a, b in zip(pts, pts[1:]):
        if Fraction(float(a)) ** 2 <= q <= Fraction(float(b)) ** 2:
            mid = (Fraction(float(a)) + Fraction(float(b))) / 2
            if q < mid * mid:
                best = a
            elif q > mid * mid:
                best = b
            else:
                best = a if (int(np.float32(a).view(np.uint32)) & 1) == 0 else b
    return np.float32(best)


@pytest.mark.parametrize("n", [1, 2, 3, 5, 8, 32])
def test_server_average_is_correctly_rounded_exact_mean(n):
    """With a zero server error, the compensated server value is the exact
    mean of the n decoded messages (+-scale), rounded once to fp32."""
    from fractions import Fraction
    rng = np.random.default_rng(100 + n)
    ln = 200
    nw = (ln + 63) // 64
    wbits = rng.integers(0, 2 ** 63, size=(n, nw), dtype=np.uint64) * np.uint64(2) + \
        rng.integers(0, 2, size=(n, nw), dtype=np.uint64)
    wscale = rng.lognormal(-7.0, 1.5, size=n).astype(np.float32)
    dbar = np.zeros(ln, np.float32)
    z = np.zeros(ln, np.float32)
    sbits = np.zeros(nw, np.uint64)
    oracle.server_segment(0, ln, n, wbits.reshape(-1), nw, wscale, 1, dbar, sbits, z)
    for e in range(ln):
        tot = Fraction(0)
        for i in range(n):
            bit = (int(wbits[i, e // 64]) >> (e % 64)) & 1
            tot += Fraction(float(wscale[i])) * (1 if bit else -1)
        assert z[e] == _nearest_f32(tot / n), (n, e)


@pytest.mark.parametrize("length", [1, 3, 64, 100, 200])
def test_scale_is_correctly_rounded_rms(length):
    """scale = sqrt(sum z^2 / len) rounded once to fp32 (the fp64 path is
    exact up to a final rounding for these sizes)."""
    from fractions import Fraction
    rng = np.random.default_rng(length)
    for trial in range(20):
        z = (rng.standard_normal(length) * 10.0 ** rng.uniform(-6, 2)).astype(np.float32)
        _, s = oracle.compress(z)
        q = sum(Fraction(float(v)) ** 2 for v in z) / length
        assert s == _sqrt_nearest_f32(q), (length, trial)


@pytest.mark.parametrize("length", [64, 128, 1024])
def test_equal_magnitudes_compress_exactly(length):
    """|z| constant (signs arbitrary, power-of-two length): the scale is |c|
    exactly, C[z] = z and the new error is exactly zero."""
    rng = np.random.default_rng(length)
    c = np.float32(0.3721)
    z = (c * rng.choice([-1.0, 1.0], size=length)).astype(np.float32)
    m = np.zeros(length, np.float32)
    delta = np.zeros(length, np.float32)
    bits = np.zeros((length + 63) // 64, np.uint64)
    zs = np.zeros(length, np.float32)
    s = oracle.worker_segment(0, length, 0.0, m, z, delta, bits, zs)  # beta1 = 0: momentum = g
    assert s == c
    assert not delta.any()  # delta = z - C[z] = 0
    signs = np.array([(int(bits[e // 64]) >> (e % 64)) & 1 for e in range(length)])
    assert np.array_equal(signs == 1, z >= 0)


def test_state_resumes_bit_exactly_from_a_copy():
    """Checkpoint/resume: the state (x, m, v, every worker error, the server
    error) is complete; 3 + 3 steps through a serialised copy equal 6
    straight steps."""
    import io
    wl = synth.Workload(name="ckpt", numel=[3000, 64, 1000], n=3, warmup_steps=0, steps=6)
    L = oracle.Layout(wl.numel, wl.n)
    x = synth.host_params(wl, L.D)
    x[~L.real_mask()] = 0
    rng = np.random.default_rng(5)
    m = (rng.standard_normal(L.D) * 1e-4).astype(np.float32)
    v = (rng.random(L.D) * 1e-7).astype(np.float32)
    grads = [synth.host_grads(wl, L.D, L.tensor_off, t) for t in range(1, 7)]
    straight = oracle.State(L, x.copy(), m.copy(), v.copy())
    for g in grads:
        straight.step(g, LR, BETA1, EPS)
    first = oracle.State(L, x.copy(), m.copy(), v.copy())
    for g in grads[:3]:
        first.step(g, LR, BETA1, EPS)
    buf = io.BytesIO()
    np.savez(buf, x=first.x, m=first.m, v=first.v, delta=first.delta, delta_bar=first.delta_bar)
    buf.seek(0)
    saved = np.load(buf)
    resumed = oracle.State(L, saved["x"].copy(), saved["m"].copy(), saved["v"].copy())
    resumed.delta[...] = saved["delta"]
    resumed.delta_bar[...] = saved["delta_bar"]
    for g in grads[3:]:
        resumed.step(g, LR, BETA1, EPS)
    for name in ("x", "m", "delta", "delta_bar", "wbits", "sbits", "wscales", "sscales"):
        assert np.array_equal(getattr(resumed, name), getattr(straight, name)), name
    # dropping the errors (a plausible incomplete checkpoint) changes the result
    lossy = oracle.State(L, saved["x"].copy(), saved["m"].copy(), saved["v"].copy())
    for g in grads[3:]:
        lossy.step(g, LR, BETA1, EPS)
    assert not np.array_equal(lossy.x, straight.x)


def test_oracle_matches_its_recorded_reference_run():
    """Regression guard: the oracle reproduces the state digests that
    tests/golden/make_oracle_reference.py recorded (re-run that script only
    with a change to the oracle's arithmetic that the paper justifies)."""
    import importlib.util
    import os
    path = os.path.join(os.path.dirname(__file__), "golden", "make_oracle_reference.py")
    spec = importlib.util.spec_from_file_location("make_oracle_reference", path)
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    gd = _golden("oracle_reference_run.json")
    assert gd["workload"] == mod.WORKLOAD
    assert mod.digests(mod.run()) == gd["sha256"]


# ---------------------------------------------------------------------------
# Brute force on tiny sizes: the whole compression step written again with
# numpy scalar semantics (fp32 operations one at a time, fp64 reductions),
# over sizes that cross word and chunk boundaries and special values
# ---------------------------------------------------------------------------

def _numpy_step(L, x, m, v, delta, dbar, g, lr, beta1, eps):
    f32 = np.float32
    n = L.n
    omb1 = f32(f32(1.0) - f32(beta1))
    b1 = f32(beta1)
    segs = L.segments()
    wsign = np.zeros((n, L.D), bool)
    wscale = np.zeros((n, len(segs)), np.float32)
    for i in range(n):
        for q, (b, e) in enumerate(segs):
            if e == b:
                continue
            z = [f32(f32(f32(b1 * m[k]) + f32(omb1 * g[i, k])) + delta[i, k]) for k in range(b, e)]
            s = f32(math.sqrt(sum(float(t) * float(t) for t in z) / (e - b)))
            wscale[i, q] = s
            for k, t in zip(range(b, e), z):
                wsign[i, k] = t >= 0
                delta[i, k] = f32(t - s) if t >= 0 else f32(t + s)
    for q, (b, e) in enumerate(segs):
        if e == b:
            continue
        zb = []
        for k in range(b, e):
            acc = 0.0
            for i in range(n):
                acc += float(wscale[i, q]) if wsign[i, k] else -float(wscale[i, q])
            zb.append(f32(f32(acc / n) + dbar[k]))
        s = f32(math.sqrt(sum(float(t) * float(t) for t in zb) / (e - b)))
        for k, t in zip(range(b, e), zb):
            mb = s if t >= 0 else f32(-s)
            dbar[k] = f32(t - mb)
            x[k] = f32(x[k] - f32(f32(lr) * f32(mb / f32(math.sqrt(f32(v[k] + f32(eps)))))))
            m[k] = mb


@pytest.mark.parametrize("numel,n", [([1], 1), ([63, 64, 65], 2), ([130, 7], 3), ([200], 4),
                                     ([129, 0, 64], 8), ([1, 2, 3, 190], 4)])
def test_brute_force_tiny_step_against_numpy(numel, n):
    L = oracle.Layout(numel, n)
    rng = np.random.default_rng(sum(numel) + n)
    mask = L.real_mask()
    x = (rng.standard_normal(L.D) * 0.02).astype(np.float32)
    m = (rng.standard_normal(L.D) * 1e-3).astype(np.float32)
    v = (rng.random(L.D) * 1e-5).astype(np.float32)
    for a in (x, m, v):
        a[~mask] = 0
    st = oracle.State(L, x, m, v)
    X, M, V = x.copy(), m.copy(), v.copy()
    delta = np.zeros((n, L.D), np.float32)
    dbar = np.zeros(L.D, np.float32)
    for t in range(3):
        g = (rng.standard_normal((n, L.D)) * 1e-3).astype(np.float32)
        g[:, ::11] = 0.0                 # exact zeros
        g[:, 5::13] = -0.0
        if t == 1:
            g[:, :] = g[0]              # all workers equal for one step
        g[:, ~mask] = 0
        st.step(g, LR, BETA1, EPS)
        _numpy_step(L, X, M, V, delta, dbar, g, LR, BETA1, EPS)
        assert np.array_equal(st.x[mask], X[mask]), t
        assert np.array_equal(st.m[mask], M[mask]), t
        assert np.array_equal(st.delta[:, mask], delta[:, mask]), t
        assert np.array_equal(st.delta_bar[mask], dbar[mask]), t
