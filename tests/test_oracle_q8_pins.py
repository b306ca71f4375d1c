"""Pins of the two-plane INT8 key oracle against facts other than itself (CPU).

Each test names what fixes the expected value: a hand-computed fixture,
exact rational arithmetic, a closed form, library softmax over the
dequantized operands, or an invariant of the method.
"""

import json
import math
import os
from fractions import Fraction

import numpy as np
import pytest
import torch

from oracle import q8_oracle as q8
from oracle import bf16_bits_to_f64, combine
from tests import _adapt
from workloads import host_bits, make_cascade, make_custom

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
INF = float("inf")


def _bits(x):
    """BF16 bits of FP32-representable values that BF16 holds exactly."""
    return (np.asarray(x, dtype=np.float32).view(np.uint32) >> 16).astype(np.uint16)


def _rand_bits(shape, seed, scale=1.0):
    g = torch.Generator().manual_seed(seed)
    t = (torch.randn(*shape, generator=g) * scale).to(torch.bfloat16)
    return host_bits(t)


# ------------------------------------------------------------------ Q1 -----
@pytest.mark.parametrize("d", [1, 2, 4, 8, 64, 128])
def test_hadamard_is_orthogonal_up_to_d(d):
    """Closed form: H H^T = D I, entries +-1, first row and column all ones."""
    h = q8.hadamard(d)
    assert np.array_equal(np.abs(h), np.ones((d, d)))
    assert np.array_equal(h @ h.T, d * np.eye(d))
    assert np.all(h[0] == 1) and np.all(h[:, 0] == 1)


def test_rotation_is_exact_rational_sum():
    """Exact arithmetic: each rotated coordinate equals the rational sum of +-inputs."""
    bits = _rand_bits((6, 128), seed=11)
    rot = q8.rotate(bf16_bits_to_f64(bits))
    h = q8.hadamard(128)
    vals = bf16_bits_to_f64(bits)
    for r in range(bits.shape[0]):
        for i in (0, 1, 37, 127):
            exact = sum(Fraction(float(vals[r, j])) * int(h[i, j]) for j in range(128))
            assert Fraction(float(rot[r, i])) == exact


def test_rotated_dot_product_is_d_times_original():
    """Closed form: (Hq).(Hk) = D q.k."""
    q = bf16_bits_to_f64(_rand_bits((3, 64), seed=1))
    k = bf16_bits_to_f64(_rand_bits((5, 64), seed=2))
    lhs = q8.rotate(q) @ q8.rotate(k).T
    np.testing.assert_allclose(lhs, 64 * (q @ k.T), rtol=1e-12, atol=1e-12)


# ------------------------------------------------------------------ Q2 -----
def test_key_split_hand_example():
    """Hand-computed fixture (Section 4, cache format; worked with H_4)."""
    fx = json.load(open(os.path.join(GOLDEN, "q8_split_example.json")))
    for key in fx["keys"]:
        a, b, e = q8.split_keys(_bits(key["k"])[None, :])
        assert np.array_equal(q8.rotate(np.array(key["k"])[None, :])[0], key["rotated"])
        assert int(e[0]) == key["scale_bits"]
        assert float(bf16_bits_to_f64(e)[0]) == key["scale"]
        assert a[0].tolist() == key["a"]
        assert b[0].tolist() == key["b"]


def test_key_split_bounds_and_minimal_scale():
    """Closed forms: |a| <= 127, |k'' - e(a + b/256)| <= e/256 (<= e/512 unless b
    was clamped), and e is the smallest BF16 value with max|k''|/e <= 127."""
    bits = _rand_bits((300, 128), seed=5, scale=3.0)
    bits[7] = 0                                  # an all-zero key
    bits[8] = _bits(np.where(np.arange(128) == 3, 100.0, 0.0))  # one spike
    bits[9] = _bits(np.full(128, -0.5))          # constant key: rotated = one coordinate
    a, b, e_bits = q8.split_keys(bits)
    rot = q8.rotate(bf16_bits_to_f64(bits))
    e = bf16_bits_to_f64(e_bits)
    assert np.abs(a.astype(int)).max() <= 127
    rec = q8.dequant(a, b, e)
    err = np.abs(rec - rot)
    assert np.all(err <= e[:, None] / 256 + 1e-300)
    unclamped = b != 127
    assert np.all(err[unclamped] <= e[:, None].repeat(128, 1)[unclamped] / 512 * (1 + 1e-12))
    m = np.abs(rot).max(axis=1)
    nz = m > 0
    assert np.all(e[~nz] == 0) and np.all(a[~nz] == 0) and np.all(b[~nz] == 0)
    assert np.all(m[nz] / e[nz] <= 127)
    smaller = bf16_bits_to_f64((e_bits[nz] - 1).astype(np.uint16))   # next BF16 down
    assert np.all(m[nz] / smaller > 127)
    # the key's code depends on that key alone
    a1, b1, e1 = q8.split_keys(bits[40:41])
    assert np.array_equal(a1[0], a[40]) and np.array_equal(b1[0], b[40]) and e1[0] == e_bits[40]


# ------------------------------------------------------------------ Q3 -----
def test_query_split_hand_example():
    """Hand-computed fixture: planes, scale and the refined score vs q.k = 1."""
    fx = json.load(open(os.path.join(GOLDEN, "q8_split_example.json")))
    qf = fx["query"]
    qa, qb, eta = q8.split_queries(_bits(qf["q"])[None, :], qf["sm_scale"])
    assert qa[0].tolist() == qf["qa"] and qb[0].tolist() == qf["qb"]
    assert abs(float(eta[0]) - qf["eta_f64"]) <= 2.0 ** -24 * qf["eta_f64"]
    ka, kb, ke = q8.split_keys(_bits(fx["keys"][0]["k"])[None, :])
    coarse, refine = q8.coarse_and_refine(qa, qb, eta, ka, kb, bf16_bits_to_f64(ke))
    s = coarse[0, 0] + refine[0, 0]
    assert abs(s - qf["refined_score_vs_key0"]) < 1e-6
    assert abs(s - qf["exact_score_vs_key0"]) < 1e-5


def test_query_split_reconstruction():
    """Closed form: q'' = f (qa + qb/256) within f/256 per coordinate, with
    f = max|q''|/127 recovered from eta = log2(e) sm f / D."""
    bits = _rand_bits((40, 64), seed=9)
    bits[3] = 0
    sm = 0.125
    qa, qb, eta = q8.split_queries(bits, sm)
    rot = q8.rotate(bf16_bits_to_f64(bits))
    f = eta.astype(np.float64) * 64 / (math.log2(math.e) * sm)
    rec = f[:, None] * (qa + qb / 256.0)
    tol = np.abs(rot).max(axis=1, keepdims=True) / 127 / 256 * (1 + 1e-5) + 1e-6 * np.abs(rot)
    assert np.all(np.abs(rec - rot) <= tol)
    assert np.abs(qa.astype(int)).max() == 127
    assert np.all(qa[3] == 0) and eta[3] == 0


def test_refine_tau_follows_request_length():
    """tau = kappa + ceil(log2 n) (the request's own length)."""
    assert q8.refine_tau(1, 4.0) == 4.0
    assert q8.refine_tau(2, 4.0) == 5.0
    assert q8.refine_tau(8192, 4.0) == 17.0
    assert q8.refine_tau(8193, 4.0) == 18.0
    assert q8.refine_tau(100000, 0.5) == np.float32(17.5)


# ------------------------------------------------------------- Q4/Q6 -------
def test_scores_equal_dequantized_dot_products():
    """Independent path: coarse = log2(e) sm (f(qa+qb/256)) . (e a) / D and
    coarse + refine = the same with the full code e (a + b/256), up to the FP32
    rounding of eta; both are close to the exact BF16 score."""
    d, sm = 128, 1 / math.sqrt(128)
    kb_ = _rand_bits((50, d), seed=21)
    qb_ = _rand_bits((4, d), seed=22)
    a, b, e_bits = q8.split_keys(kb_)
    qa, qb, eta = q8.split_queries(qb_, sm)
    e = bf16_bits_to_f64(e_bits)
    coarse, refine = q8.coarse_and_refine(qa, qb, eta, a, b, e)
    f = np.abs(q8.rotate(bf16_bits_to_f64(qb_))).max(axis=1) / 127
    qdeq = f[:, None] * (qa + qb / 256.0)
    scale = math.log2(math.e) * sm / d
    want_coarse = scale * (qdeq @ (e[:, None] * a).T)
    want_full = scale * (qdeq @ q8.dequant(a, b, e).T)
    np.testing.assert_allclose(coarse, want_coarse, rtol=2 ** -23, atol=1e-12)
    np.testing.assert_allclose(coarse + refine, want_full, rtol=2 ** -23, atol=1e-12)
    exact = math.log2(math.e) * sm * (bf16_bits_to_f64(qb_) @ bf16_bits_to_f64(kb_).T)
    assert np.abs(coarse + refine - exact).max() < 1e-3
    # the refine term is what plane B adds: a strictly smaller correction
    assert np.abs(coarse + refine - exact).max() < np.abs(coarse - exact).max() / 20


def test_refine_term_closed_form_bound():
    """|refine| <= eta e ||qa + qb/256||_1 / 2, since |b| <= 128 (a sign or
    scale error in the refine term breaks it)."""
    a, b, e_bits = q8.split_keys(_rand_bits((80, 64), seed=31, scale=2.0))
    qa, qb, eta = q8.split_queries(_rand_bits((6, 64), seed=32), 0.125)
    e = bf16_bits_to_f64(e_bits)
    _, refine = q8.coarse_and_refine(qa, qb, eta, a, b, e)
    bound = (eta.astype(np.float64)[:, None] * e[None, :]
             * np.abs(qa + qb / 256.0).sum(axis=1)[:, None] / 2)
    assert np.all(np.abs(refine) <= bound * (1 + 1e-12))
    assert np.abs(refine).max() > 1e-3 * bound.max()   # not vacuous


# ------------------------------------------------------------------ Q5 -----
def _wl(seed=0, lens=(300, 513), heads=8, kv=2, d=64, spikes=6, sinks=2, paged=True):
    return make_custom(batch=len(lens), heads=heads, kv_heads=kv, dim=d, lens=list(lens),
                       paged=paged, spike_count=spikes, alpha_spike=3.0, n_sink=sinks,
                       alpha_sink=6.0, seed=seed)


def _q8_inputs(wl, kappa):
    planes = q8.split_keys(host_bits(wl.k))
    qa, qb, eta = q8.split_queries(host_bits(wl.q), wl.sm_scale)
    lens = wl.flat.seq_lens_host
    tau = np.array([q8.refine_tau(n, kappa) for n in lens], dtype=np.float32)
    return planes, qa, qb, eta, tau


def _run(wl, planes, qa, qb, eta, tau, z, T, splits=1, level=0, **kw):
    lv = _adapt.level_args(wl.levels[level])
    return q8.decode_level_q8(qa, qb, eta, planes, host_bits(wl.v), num_kv_heads=wl.num_kv_heads,
                              page_size=wl.page_size, z=z, T=T, tau=tau, num_splits=splits,
                              **lv, **kw)


@pytest.mark.parametrize("T", [INF, 16.0, 6.0])
@pytest.mark.parametrize("kappa", [-INF, 2.0, INF])
def test_gate_invariants(T, kappa):
    """refine implies live; kappa = +inf refines every live key; T = inf makes
    every key live; the bits are the same for every row of a GQA group; every
    counted key has x >= -T and every cut key x < -T."""
    wl = _wl(seed=1)
    planes, qa, qb, eta, tau = _q8_inputs(wl, kappa)
    z = _adapt.estimate(_adapt.oracle_inputs(wl))
    _, _, info = _run(wl, planes, qa, qb, eta, tau, z, T, want_scores=True)
    group = wl.num_heads // wl.num_kv_heads
    for (seq, g), (rows, xc, x, live, ref) in info.items():
        assert not np.any(ref & ~live)
        if math.isinf(kappa) and kappa > 0:
            assert np.array_equal(ref, live)
        if math.isinf(kappa) and kappa < 0:
            assert not ref.any()
        if math.isinf(T):
            assert live.all()
        assert np.all(live == live[0]) and np.all(ref == ref[0])   # one request: one group
        assert len(rows) == group
        if not math.isinf(T):
            assert np.all(live == (xc >= -T).any(axis=0))
            assert np.all((x < -T) | live)
        assert np.array_equal(x != xc, ref & (x != xc))              # only refined keys move


def test_gates_follow_request_not_batch():
    """Cascade level with stacked rows of several requests: each request's
    partials equal those of its rows scanned alone (gates do not depend on the
    batch)."""
    wl = make_cascade(requests=3, heads=4, kv_heads=1, dim=64, prefix_len=160, suffix_len=48,
                      seed=4)
    planes, qa, qb, eta, tau = _q8_inputs(wl, 1.0)
    z = _adapt.estimate(_adapt.oracle_inputs(wl))
    lv = _adapt.level_args(wl.levels[0])
    full_a, full_l = _run(wl, planes, qa, qb, eta, tau, z, 8.0, splits=2)
    for r in range(3):
        one = dict(lv)
        one["row_indptr"] = np.array([0, 1])
        one["row_req"] = np.array([r])
        pa, pl = q8.decode_level_q8(qa, qb, eta, planes, host_bits(wl.v),
                                    num_kv_heads=1, page_size=wl.page_size, z=z, T=8.0, tau=tau,
                                    num_splits=2, **one)
        assert np.array_equal(pa[:, r], full_a[:, r]) and np.array_equal(pl[:, r], full_l[:, r])


# ------------------------------------------------------------------ Q7 -----
@pytest.mark.parametrize("d,paged", [(64, True), (128, True), (64, False)])
def test_dense_full_refine_equals_library_softmax_on_codes(d, paged):
    """Library routine: at T = inf with every key refined the output is softmax
    attention over the dequantized rotated operands (torch SDPA in FP64), and it
    stays close to softmax over the original BF16 operands."""
    wl = _wl(seed=2, d=d, paged=paged, lens=(200, 77))
    planes, qa, qb, eta, tau = _q8_inputs(wl, INF)
    z = np.full((2, wl.num_heads), 3.25)
    pa, pl = _run(wl, planes, qa, qb, eta, tau, z, INF, splits=3)
    o, _ = combine(pa, pl)
    oi = _adapt.oracle_inputs(wl)
    group = wl.num_heads // wl.num_kv_heads
    for r, n in enumerate(wl.flat.seq_lens_host):
        for h in range(wl.num_heads):
            g = h // group
            a = q8._gather_raw(planes[0], r, g, n, oi["flat"]["block_table"], wl.page_size)
            b = q8._gather_raw(planes[1], r, g, n, oi["flat"]["block_table"], wl.page_size)
            e = bf16_bits_to_f64(q8._gather_raw(planes[2][..., None], r, g, n,
                                                oi["flat"]["block_table"], wl.page_size)[:, 0])
            kdeq = q8.dequant(a, b, e)
            f = float(eta[r, h]) * d / (math.log2(math.e) * wl.sm_scale)
            qdeq = f * (qa[r, h] + qb[r, h] / 256.0)
            vals = bf16_bits_to_f64(q8._gather_raw(oi["v_bits"], r, g, n,
                                                   oi["flat"]["block_table"], wl.page_size))
            want = torch.nn.functional.scaled_dot_product_attention(
                torch.from_numpy(qdeq)[None, None, None], torch.from_numpy(kdeq)[None, None],
                torch.from_numpy(vals)[None, None], scale=wl.sm_scale / d)[0, 0, 0].numpy()
            np.testing.assert_allclose(o[r, h], want, rtol=0, atol=1e-9 * np.abs(want).max() + 1e-12)
            qo = bf16_bits_to_f64(oi["q_bits"][r, h])
            ko = bf16_bits_to_f64(q8._gather_raw(oi["k_bits"], r, g, n,
                                                 oi["flat"]["block_table"], wl.page_size))
            plain = torch.nn.functional.scaled_dot_product_attention(
                torch.from_numpy(qo)[None, None, None], torch.from_numpy(ko)[None, None],
                torch.from_numpy(vals)[None, None], scale=wl.sm_scale)[0, 0, 0].numpy()
            assert np.abs(o[r, h] - plain).max() < 2e-3 * max(1.0, np.abs(plain).max())


@pytest.mark.parametrize("T,kappa", [(INF, 0.0), (12.0, 3.0), (5.0, -INF), (INF, INF)])
def test_partials_add_over_splits(T, kappa):
    """Additivity: the splits' partials add up to the one-split pair at any
    depth and refine threshold (every decision is per key)."""
    wl = _wl(seed=3, lens=(700, 130))
    planes, qa, qb, eta, tau = _q8_inputs(wl, kappa)
    z = _adapt.estimate(_adapt.oracle_inputs(wl))
    a1, l1 = _run(wl, planes, qa, qb, eta, tau, z, T, splits=1)
    a5, l5 = _run(wl, planes, qa, qb, eta, tau, z, T, splits=5)
    np.testing.assert_allclose(a5.sum(axis=0), a1[0], rtol=1e-12, atol=1e-14)
    np.testing.assert_allclose(l5.sum(axis=0), l1[0], rtol=1e-12, atol=1e-14)


def test_huge_finite_depth_equals_dense():
    """A depth above every |x| keeps every key live: same as T = inf."""
    wl = _wl(seed=6)
    planes, qa, qb, eta, tau = _q8_inputs(wl, 2.0)
    z = _adapt.estimate(_adapt.oracle_inputs(wl))
    ad, ld = _run(wl, planes, qa, qb, eta, tau, z, INF, splits=2)
    ah, lh = _run(wl, planes, qa, qb, eta, tau, z, 1e30, splits=2)
    assert np.array_equal(ad, ah) and np.array_equal(ld, lh)


def test_imposed_mode_reproduces_own_decisions():
    """Imposed decisions taken from FP32 copies of the oracle's own scores give
    the own-mode partials wherever no score sits within FP32 rounding of -T or
    -tau (here: none does)."""
    wl = _wl(seed=7)
    planes, qa, qb, eta, tau = _q8_inputs(wl, 2.0)
    z = _adapt.estimate(_adapt.oracle_inputs(wl))
    T = 9.0
    pa, pl, info = _run(wl, planes, qa, qb, eta, tau, z, T, want_scores=True)
    b_, h = wl.q.shape[:2]
    n_max = max(wl.flat.seq_lens_host)
    ixc = np.zeros((b_, h, n_max), dtype=np.float32)
    ix = np.zeros((b_, h, n_max), dtype=np.float32)
    for (seq, g), (rows, xc, x, live, ref) in info.items():
        for k, (r, hh) in enumerate(rows):
            ixc[r, hh, :xc.shape[1]] = xc[k]
            ix[r, hh, :x.shape[1]] = x[k]
        assert np.abs(np.abs(xc) - T).min() > 1e-4
    pa2, pl2 = _run(wl, planes, qa, qb, eta, tau, z, T, imposed=(ixc, ix))
    assert np.array_equal(pa, pa2) and np.array_equal(pl, pl2)


# --------------------------------------------------------------- estimate -
def test_estimate_on_coarse_scores_is_exact_lse_when_short():
    """Closed form: for n <= 192 the estimate is log2 sum 2^coarse."""
    wl = _wl(seed=8, lens=(150, 192))
    planes, qa, qb, eta, _ = _q8_inputs(wl, 0.0)
    oi = _adapt.oracle_inputs(wl)
    z = q8.estimate_level_q8(qa, qb, eta, planes, num_kv_heads=wl.num_kv_heads,
                             page_size=wl.page_size, seq_lens=oi["flat"]["seq_lens"],
                             block_table=oi["flat"]["block_table"])
    group = wl.num_heads // wl.num_kv_heads
    for r, n in enumerate(wl.flat.seq_lens_host):
        for h in range(wl.num_heads):
            g = h // group
            bt = oi["flat"]["block_table"]
            a = q8._gather_raw(planes[0], r, g, n, bt, wl.page_size)
            e = bf16_bits_to_f64(q8._gather_raw(planes[2][..., None], r, g, n, bt,
                                                wl.page_size)[:, 0])
            f = float(eta[r, h]) * 64 / (math.log2(math.e) * wl.sm_scale)
            s = (math.log2(math.e) * wl.sm_scale / 64) * ((e[:, None] * a) @ (
                f * (qa[r, h] + qb[r, h] / 256.0)))
            want = float(np.logaddexp2.reduce(s))
            assert abs(z[r, h] - want) < 1e-5


# ------------------------------------------------------ 8-bit values -------
def test_e4m3_table_matches_torch():
    """Library routine: torch's float8_e4m3fn decoding of all 256 codes."""
    ref = torch.arange(256, dtype=torch.uint8).view(torch.float8_e4m3fn).double().numpy()
    ours = q8.e4m3_table()
    nan = np.isnan(ref)
    assert np.array_equal(np.isnan(ours), nan)
    assert np.array_equal(ours[~nan], ref[~nan])


def test_e4m3_encode_matches_torch_rounding():
    """Library routine: torch's round-to-nearest-even cast to float8_e4m3fn on
    random magnitudes, every code's value and every midpoint (ties); beyond
    448 the writer saturates (reading) where torch gives NaN."""
    g = torch.Generator().manual_seed(0)
    x = torch.cat([torch.randn(20000, generator=g) * s for s in (1e-3, 0.1, 3.0, 60.0)])
    vals = torch.from_numpy(q8.e4m3_table()[:0x7F]).float()
    mids = (vals[1:] + vals[:-1]) / 2
    x = torch.cat([x, vals, -vals, mids, -mids]).double()
    x = x[x.abs() <= 448]
    want = x.float().to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    got = q8.e4m3_encode(x.numpy())
    neg_zero = (want == 0x80) & (got == 0)   # -0 encodes as +0 here
    assert np.array_equal(got[~neg_zero], want[~neg_zero])
    assert q8.e4m3_encode(np.array([449.0, 1e9, -500.0])).tolist() == [0x7E, 0x7E, 0xFE]


def test_two_value_planes_are_lossless():
    """Brute force over every finite BF16 value: 2^e (p + r/16) gives it back
    exactly when |v 2^-e| <= 448 (and at least 2^-6, the normal E4M3 range)."""
    bits = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16)
    v = bf16_bits_to_f64(bits)
    for e in (-3, 0, 4):
        y = v * 2.0 ** -e
        ok = np.isfinite(v) & (np.abs(y) <= 448) & (np.abs(y) >= 2.0 ** -6)
        p, r = q8.split_values(bits[ok], e)
        assert np.array_equal(q8.dequant_values(p, r, e), v[ok])
        # plane 1 alone is within half an E4M3 step (relative 2^-4)
        err = np.abs(q8.dequant_values(p, r, e, refined=False) - v[ok])
        assert np.all(err <= np.abs(v[ok]) * 2.0 ** -4 + 1e-300)


@pytest.mark.parametrize("T", [INF, 8.0])
def test_value_planes_fully_refined_equal_bf16_values(T):
    """With every live key's second value plane read (kappa_v = +inf), the
    8-bit-value decode equals the BF16-value decode (the planes are exact
    here); with none read, it differs by at most plane 1's rounding."""
    wl = _wl(seed=9)
    planes, qa, qb, eta, tau = _q8_inputs(wl, 0.0)
    z = _adapt.estimate(_adapt.oracle_inputs(wl))
    vb = host_bits(wl.v)
    vmax = float(np.abs(bf16_bits_to_f64(vb)).max())
    e = int(np.ceil(np.log2(vmax / 448.0)))
    p, r = q8.split_values(vb, e)
    lv = _adapt.level_args(wl.levels[0])
    args = dict(num_kv_heads=wl.num_kv_heads, page_size=wl.page_size, z=z, T=T, tau=tau,
                num_splits=2, **lv)
    a0, l0 = q8.decode_level_q8(qa, qb, eta, planes, vb, **args)
    tinf = np.full_like(tau, np.inf)
    a1, l1 = q8.decode_level_q8(qa, qb, eta, planes, vb, values8=(p, r, e), tau_v=tinf, **args)
    small = (np.abs(bf16_bits_to_f64(vb)) < 2.0 ** (e - 6)).any()
    if not small:
        assert np.array_equal(a0, a1)
    np.testing.assert_allclose(a1, a0, rtol=1e-12, atol=1e-12 * np.abs(a0).max())
    assert np.array_equal(l0, l1)
    a2, _ = q8.decode_level_q8(qa, qb, eta, planes, vb, values8=(p, r, e),
                               tau_v=np.full_like(tau, -np.inf), **args)
    o0, _ = combine(a0, l0)
    o2, _ = combine(a2, l0)
    assert np.abs(o2 - o0).max() <= 2.0 ** -4 * vmax * 1.01
    assert np.abs(o2 - o0).max() > 0


def test_refine_v_gate_invariants():
    """refine_v implies live; it follows the coarse scores per GQA group."""
    wl = _wl(seed=10)
    planes, qa, qb, eta, tau = _q8_inputs(wl, 0.0)
    z = _adapt.estimate(_adapt.oracle_inputs(wl))
    _, _, info = _run(wl, planes, qa, qb, eta, tau, z, 8.0, want_scores=True)
    group = wl.num_heads // wl.num_kv_heads
    for (seq, g), (rows, xc, x, live, ref) in info.items():
        tv = np.full(len(rows), 3.0)
        lv_, rv = q8.gate_bits(xc, np.repeat(np.arange(len(rows) // group), group), 8.0, tv)
        assert np.array_equal(lv_, live)
        assert not np.any(rv & ~live)
        assert np.array_equal(rv[0], live[0] & (xc >= -3.0).any(axis=0))


# ------------------------------------------------------------------ Q9 -----
def test_stacked_operands_are_torch_fp16_of_the_exact_codes():
    """Library routine: the stacked level's FP16 keys and queries are torch's
    round-to-nearest-even FP16 conversion of the exact FP32 values
    e (a + b/256) and qa + qb/256, and stay within FP16's relative rounding
    bound 2^-11 of them (normal range)."""
    bits = _rand_bits((64, 128), seed=21, scale=3.0)
    a, b, e_bits = q8.split_keys(bits)
    k = q8.stack_keys(a, b, e_bits)
    assert k.dtype == np.float16
    exact = q8.dequant(a, b, bf16_bits_to_f64(e_bits))
    assert np.array_equal(exact.astype(np.float32).astype(np.float64), exact)  # exact in FP32
    want = torch.from_numpy(exact.astype(np.float32)).to(torch.float16).numpy()
    assert np.array_equal(k.view(np.uint16), want.view(np.uint16))
    normal = np.abs(exact) >= 2.0 ** -14
    assert np.all(np.abs(k.astype(np.float64) - exact)[normal]
                  <= 2.0 ** -11 * np.abs(exact)[normal])
    qa, qb, _ = q8.split_queries(_rand_bits((8, 128), seed=22), 0.125)
    qh = q8.stack_queries(qa, qb)
    qex = qa.astype(np.float64) + qb.astype(np.float64) / 256.0
    want_q = torch.from_numpy(qex.astype(np.float32)).to(torch.float16).numpy()
    assert np.array_equal(qh.view(np.uint16), want_q.view(np.uint16))


def test_stacked_logit_within_the_stated_bound():
    """The paper's bound for the stacked level's FP16 product: each rounding
    puts the logit within about 2^-11 of |q||k|.  Two roundings (key and
    query) and the Cauchy-Schwarz inequality give
    |eta k^.q^ - eta k''.q~| <= eta 2^-11 (2 + 2^-11) |k''| |q~|, q~ = qa + qb/256,
    against the fully refined two-plane logit (both planes, exact)."""
    wl = _wl(seed=23, d=128, lens=(400,))
    planes, qa, qb, eta, tau = _q8_inputs(wl, INF)
    oi = _adapt.oracle_inputs(wl)
    bt = oi["flat"]["block_table"]
    khat_cache = q8.stack_keys(*planes)
    qh = q8.stack_queries(qa, qb)
    n = wl.flat.seq_lens_host[0]
    G = wl.num_heads // wl.num_kv_heads
    worst = 0.0
    for h in range(wl.num_heads):
        g = h // G
        a = q8._gather_raw(planes[0], 0, g, n, bt, wl.page_size)
        b = q8._gather_raw(planes[1], 0, g, n, bt, wl.page_size)
        e = bf16_bits_to_f64(q8._gather_raw(planes[2][..., None], 0, g, n, bt, wl.page_size)[:, 0])
        kdeq = q8.dequant(a, b, e)
        kh = q8._gather_raw(khat_cache, 0, g, n, bt, wl.page_size).astype(np.float64)
        qt = qa[0, h].astype(np.float64) + qb[0, h].astype(np.float64) / 256.0
        coarse, refine = q8.coarse_and_refine(qa[0, h][None], qb[0, h][None], eta[0, h][None],
                                              a, b, e)
        exact = (coarse + refine)[0]                       # eta e (a + b/256) . q~
        stacked = float(eta[0, h]) * (kh @ qh[0, h].astype(np.float64))
        bound = float(eta[0, h]) * 2.0 ** -11 * (2 + 2.0 ** -11) * \
            np.linalg.norm(kdeq, axis=1) * np.linalg.norm(qt)
        assert np.all(np.abs(stacked - exact) <= bound)
        worst = max(worst, float((np.abs(stacked - exact) / bound).max()))
    assert worst > 0.01  # the FP16 rounding is visible, not zero


@pytest.mark.parametrize("T", [INF, 1.5])
def test_stacked_level_equals_library_softmax_on_fp16_operands(T):
    """Library routine: the stacked level's output is softmax attention (torch
    SDPA, FP64) over the FP16 operands with scale eta ln 2 (base-2 logits), with
    the keys the depth rule cuts removed from the numerator only; at T = inf it
    is plain SDPA.  The cascade prefix of 3 requests x 8 heads stacks 24 rows."""
    wl = make_cascade(requests=3, heads=8, kv_heads=1, dim=64, prefix_len=208, suffix_len=16,
                      seed=24)
    planes, qa, qb, eta, _ = _q8_inputs(wl, 0.0)
    khat = q8.stack_keys(*planes)
    qh = q8.stack_queries(qa, qb)
    lv = _adapt.level_args(wl.levels[0])
    z = np.full((3, 8), 2.5)
    n_cut = 0
    pa, pl = q8.decode_level_q8_stacked(qh, eta, khat, host_bits(wl.v), num_kv_heads=1,
                                        page_size=wl.page_size, z=z, T=T, num_splits=3, **lv)
    o, l = combine(pa, pl)
    n = lv["seq_lens"][0]
    keys = q8._gather_raw(khat, 0, 0, n, lv["block_table"], wl.page_size).astype(np.float64)
    vals = bf16_bits_to_f64(q8._gather_raw(host_bits(wl.v), 0, 0, n, lv["block_table"],
                                           wl.page_size))
    for r in range(3):
        for h in range(8):
            qv = qh[r, h].astype(np.float64)
            sc = float(eta[r, h]) * math.log(2.0)
            if math.isinf(T):
                want = torch.nn.functional.scaled_dot_product_attention(
                    torch.from_numpy(qv)[None, None, None], torch.from_numpy(keys)[None, None],
                    torch.from_numpy(vals)[None, None], scale=sc)[0, 0, 0].numpy()
            else:
                s = float(eta[r, h]) * (keys @ qv)
                cut = s - z[r, h] < -T
                n_cut += int(cut.sum())
                p = torch.softmax(torch.from_numpy(s * math.log(2.0)), dim=0).numpy()
                want = (p * ~cut) @ vals
            np.testing.assert_allclose(o[r, h], want, rtol=0, atol=1e-10 * np.abs(want).max())
            # L is every key's weight against the reference
            np.testing.assert_allclose(l[r, h], np.exp2(float(eta[r, h]) * (keys @ qv)
                                                        - z[r, h]).sum(), rtol=1e-12)
    assert math.isinf(T) or 0 < n_cut < 3 * 8 * n


def test_stacked_level_partials_add_over_splits():
    """Additivity over splits, and each request's rows give the same partials
    scanned alone (the stacked level has no group gate)."""
    wl = make_cascade(requests=3, heads=4, kv_heads=1, dim=64, prefix_len=336, suffix_len=16,
                      seed=25)
    planes, qa, qb, eta, _ = _q8_inputs(wl, 0.0)
    khat = q8.stack_keys(*planes)
    qh = q8.stack_queries(qa, qb)
    lv = _adapt.level_args(wl.levels[0])
    z = _adapt.estimate(_adapt.oracle_inputs(wl))
    kw = dict(num_kv_heads=1, page_size=wl.page_size, z=z, T=6.0)
    a1, l1 = q8.decode_level_q8_stacked(qh, eta, khat, host_bits(wl.v), num_splits=1, **kw, **lv)
    a4, l4 = q8.decode_level_q8_stacked(qh, eta, khat, host_bits(wl.v), num_splits=4, **kw, **lv)
    np.testing.assert_allclose(a4.sum(0), a1[0], rtol=1e-12, atol=1e-15)
    np.testing.assert_allclose(l4.sum(0), l1[0], rtol=1e-12)
    one = dict(lv)
    one["row_indptr"] = np.array([0, 1])
    one["row_req"] = np.array([1])
    a_one, _ = q8.decode_level_q8_stacked(qh, eta, khat, host_bits(wl.v), num_splits=4, **kw,
                                          **one)
    assert np.array_equal(a_one[:, 1], a4[:, 1])
