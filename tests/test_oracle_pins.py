"""Pins of the FP64 oracle against facts other than itself (CPU only).

Each test names what fixes the expected value: a hand-computed fixture, a
textbook or library routine, a closed form, or an invariant of
Proposition 1.
"""

import json
import math
import os

import numpy as np
import pytest
import scipy.special
import torch

import oracle
from tests import _adapt
from workloads import host_bits, make_config, make_custom

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
INF = float("inf")


def _T(v):
    return INF if v == "inf" else float(v)


# ------------------------------------------------------------------ O1 -----
def test_bf16_decode_matches_torch_every_pattern():
    """Library routine: torch's own BF16 -> FP64 conversion, all 65536 patterns."""
    bits = np.arange(65536, dtype=np.uint32).astype(np.uint16)
    ours = oracle.bf16_bits_to_f64(bits)
    ref = torch.from_numpy(bits.view(np.int16).copy()).view(torch.bfloat16).double().numpy()
    nan = np.isnan(ref)
    assert np.array_equal(np.isnan(ours), nan)
    assert np.array_equal(ours[~nan], ref[~nan])


@pytest.mark.parametrize("cfg", [1, 2, 4, 5])
def test_gather_reproduces_logical_cache(cfg):
    """The paged gather returns the generator's logical K/V rows (before paging)."""
    wl = make_config(cfg, seed=3, batch=2, seq_len=200 if cfg != 5 else 64, keep_logical=True)
    oi = _adapt.oracle_inputs(wl)
    for li, lv in enumerate(oi["levels"]):
        for seq, n in enumerate(lv["seq_lens"]):
            for g in range(wl.num_kv_heads):
                got = oracle.gather(oi["k_bits"], seq, g, n, lv["block_table"], wl.page_size)
                if cfg == 5:
                    break
                want = wl.logical_k[seq, g, :n].double().numpy()
                assert np.array_equal(got, want)
    fl = oi["flat"]
    for r, n in enumerate(fl["seq_lens"]):
        for g in range(wl.num_kv_heads):
            got = oracle.gather(oi["v_bits"], r, g, n, fl["block_table"], wl.page_size)
            assert np.array_equal(got, wl.logical_v[r, g, :n].double().numpy())


# ------------------------------------------------------------- O4/O5 -------
def test_hand_worked_fold_fixture():
    """Hand-computed exact example of Eq. (fold) with the depth rule."""
    with open(os.path.join(GOLDEN, "fold_worked_example.json")) as f:
        fx = json.load(f)
    s = np.array([fx["scores"]])
    v = np.array(fx["values"])
    x = s - fx["z"]
    for case in fx["cases"]:
        T = _T(case["T"])
        live = oracle.live_mask(x, T)
        assert live[0].tolist() == case["live"]
        a, l = oracle.fold(x, live, v)
        assert a[0].tolist() == case["A"]
        assert l[0] == case["L"]
    r2 = fx["group_row2"]
    x2 = np.array([r2["scores"]]) - r2["z"]
    lives = np.concatenate([oracle.live_mask(x, r2["T"]), oracle.live_mask(x2, r2["T"])])
    key, page = oracle.read_gates(lives, 5)
    assert key.tolist() == r2["key_bits_or"]
    assert page.tolist() == r2["page_bits"]


def test_exact_scores_and_threshold_tie():
    """Integer scores built from BF16-exact operands (sm_scale = ln 2 gives s = q.k).

    A key sitting exactly on x = -T is live; one binade below is cut.
    """
    d = 64
    q = np.zeros((1, d))
    q[0, 0] = 1.0
    k = np.zeros((6, d))
    k[:, 0] = [10.0, -6.0, -7.0, 2.0, 10.0, -40.0]
    s = oracle.scores(q, k, math.log(2.0))
    assert s[0].tolist() == [10.0, -6.0, -7.0, 2.0, 10.0, -40.0]
    x = s - 10.0
    assert oracle.live_mask(x, 16.0)[0].tolist() == [True, True, False, True, True, False]
    assert oracle.live_mask_imposed(x.astype(np.float32), 16.0)[0].tolist() == \
        [True, True, False, True, True, False]


def test_split_interleave_hand_table():
    """Tiles of 64 keys go round-robin to splits (hand-written table)."""
    owner = oracle.split_of_key(300, 4)
    tiles = [owner[t * 64] for t in range(5)]
    assert tiles == [0, 1, 2, 3, 0]
    assert (owner[:64] == 0).all() and (owner[256:] == 0).all() and (owner[64:128] == 1).all()
    assert (oracle.split_of_key(300, 1) == 0).all()


# ------------------------------------------------------------- P1 ----------
def _textbook_softmax_attention(q, k, v, sm_scale):
    """Natural-log softmax with max subtraction, via scipy.special.softmax."""
    logits = (q @ k.T) * sm_scale
    p = scipy.special.softmax(logits, axis=-1)
    return p @ v


def _sdpa_fp64(q, k, v, sm_scale):
    qt = torch.from_numpy(q)[None, None]
    kt = torch.from_numpy(k)[None, None]
    vt = torch.from_numpy(v)[None, None]
    return torch.nn.functional.scaled_dot_product_attention(qt, kt, vt, scale=sm_scale)[0, 0].numpy()


@pytest.mark.parametrize("splits", [1, 4])
def test_dense_equals_softmax_config1(splits):
    """Prop. 1(ii): at T = inf the fold is softmax attention, for the estimated Z."""
    wl = make_config(1)
    oi = _adapt.oracle_inputs(wl)
    z = _adapt.estimate(oi)
    o, _, _, _ = _adapt.decode(oi, z, INF, [splits])
    q = oracle.bf16_bits_to_f64(oi["q_bits"])
    for g in range(4):
        k = oracle.gather(oi["k_bits"], 0, g, 512, None, 0)
        v = oracle.gather(oi["v_bits"], 0, g, 512, None, 0)
        ref = _textbook_softmax_attention(q[0, g:g + 1], k, v, wl.sm_scale)[0]
        ref2 = _sdpa_fp64(q[0, g:g + 1], k, v, wl.sm_scale)[0]
        scale = np.abs(ref).max()
        assert np.abs(o[0, g] - ref).max() <= 1e-12 * scale
        assert np.abs(o[0, g] - ref2).max() <= 1e-12 * scale


@pytest.mark.parametrize("seed", range(4))
def test_dense_equals_softmax_random_tiny(seed):
    """Prop. 1(ii) on random ragged GQA shapes, splits 1-5, any finite Z."""
    rng = np.random.default_rng(seed)
    hkv = int(rng.integers(1, 3))
    group = int(rng.choice([1, 2, 4]))
    d = int(rng.choice([64, 128]))
    lens = [int(x) for x in rng.integers(1, 400, size=3)]
    wl = make_custom(batch=3, heads=hkv * group, kv_heads=hkv, dim=d, lens=lens,
                     spike_count=3, n_sink=2, seed=seed)
    oi = _adapt.oracle_inputs(wl)
    z = rng.normal(0.0, 20.0, size=(3, hkv * group))
    o, _, _, _ = _adapt.decode(oi, z, INF, [int(rng.integers(1, 6))])
    q = oracle.bf16_bits_to_f64(oi["q_bits"])
    for r in range(3):
        for h in range(hkv * group):
            g = h // group
            k = oracle.gather(oi["k_bits"], r, g, lens[r], oi["flat"]["block_table"], 16)
            v = oracle.gather(oi["v_bits"], r, g, lens[r], oi["flat"]["block_table"], 16)
            ref = _sdpa_fp64(q[r, h:h + 1], k, v, wl.sm_scale)[0]
            assert np.abs(o[r, h] - ref).max() <= 1e-12 * np.abs(ref).max()


# ------------------------------------------------------------- P2 ----------
@pytest.mark.parametrize("delta", [-60.0, -7.3, 0.0, 5.0, 60.0])
def test_shift_invariance(delta):
    """Proof of Prop. 1(ii): A and L scale by 2^-delta, the quotient is unchanged."""
    wl = make_custom(batch=2, heads=4, kv_heads=2, dim=64, lens=[300, 77], spike_count=4,
                     n_sink=1, seed=11)
    oi = _adapt.oracle_inputs(wl)
    z = _adapt.estimate(oi)
    o0, l0, a0, _ = _adapt.decode(oi, z, INF, [3])
    o1, l1, a1, _ = _adapt.decode(oi, z + delta, INF, [3])
    assert np.allclose(o1, o0, rtol=1e-12, atol=1e-14)
    assert np.allclose(l1 * 2.0 ** delta, l0, rtol=1e-12, atol=0)
    assert np.allclose(a1 * 2.0 ** delta, a0, rtol=1e-12, atol=1e-12 * np.abs(a0).max())


# ------------------------------------------------------------- P3 ----------
@pytest.mark.parametrize("T", [INF, 16.0, 6.0, 1.0])
def test_additivity_over_random_partitions(T):
    """Prop. 1(i): F(I)+F(J) = F(I u J) for disjoint sets, at any depth."""
    rng = np.random.default_rng(5)
    n, d = 700, 64
    x = rng.normal(-3.0, 4.0, size=(3, n))
    v = rng.normal(size=(n, d))
    live = oracle.live_mask(x, T)
    a_all, l_all = oracle.fold(x, live, v)
    for parts in (2, 5, 31):
        lab = rng.integers(0, parts, size=n)
        a_sum = np.zeros_like(a_all)
        l_sum = np.zeros_like(l_all)
        for p in rng.permutation(parts):
            m = lab == p
            a, l = oracle.fold(x[:, m], live[:, m], v[m])
            a_sum += a
            l_sum += l
        assert np.allclose(a_sum, a_all, rtol=1e-12, atol=1e-12)
        assert np.allclose(l_sum, l_all, rtol=1e-12, atol=0)
    perm = rng.permutation(n)
    a_p, l_p = oracle.fold(x[:, perm], live[:, perm], v[perm])
    assert np.allclose(a_p, a_all, rtol=1e-12, atol=1e-12) and np.allclose(l_p, l_all, rtol=1e-12)


@pytest.mark.parametrize("T", [INF, 16.0])
def test_split_count_invariance(T):
    """Split-KV is a grouping of one sum: every split count gives the same output."""
    wl = make_config(1)
    oi = _adapt.oracle_inputs(wl)
    z = _adapt.estimate(oi)
    outs = [_adapt.decode(oi, z, T, [s])[0] for s in (1, 3, 4, 8, 16)]
    for o in outs[1:]:
        assert np.allclose(o, outs[0], rtol=1e-12, atol=1e-14)


# ------------------------------------------------------------- P4/P5/P6 ----
@pytest.mark.parametrize("T", [24.0, 16.0, 12.0, 4.0])
def test_mass_kept_and_truncation_bound(T):
    """Depth rule keeps cut mass in L (L(T) = L(inf) for fixed Z); every cut key
    weighs < 2^-T relative to Z; the output error obeys the truncation bound."""
    wl = make_config(2, batch=1, seq_len=1000)
    oi = _adapt.oracle_inputs(wl)
    z = _adapt.estimate(oi)
    o_inf, l_inf, _, _ = _adapt.decode(oi, z, INF, [4])
    o_t, l_t, _, _ = _adapt.decode(oi, z, T, [4])
    assert np.array_equal(l_t, l_inf)
    q = oracle.bf16_bits_to_f64(oi["q_bits"])
    fl = oi["flat"]
    for h in range(32):
        g = h // 4
        k = oracle.gather(oi["k_bits"], 0, g, 1000, fl["block_table"], 16)
        v = oracle.gather(oi["v_bits"], 0, g, 1000, fl["block_table"], 16)
        s = oracle.scores(q[0, h:h + 1], k, wl.sm_scale)[0]
        x = s - z[0, h]
        live = oracle.live_mask(x, T)
        assert (np.exp2(x[~live]) < 2.0 ** -T).all()
        assert (np.exp2(x[live]) >= 2.0 ** -T).all()
        diag = oracle.row_diagnostics(s, z[0, h], T, v)
        err = np.abs(o_t[0, h] - o_inf[0, h]).max()
        assert err <= diag["bound_T"] * (1 + 1e-9) + 1e-15


# ------------------------------------------------------------- P7 ----------
def _lse_merge(o1, l1, o2, l2):
    """Eq. (lse-merge), natural log, evaluated stably by comparing l and l'."""
    m = np.maximum(l1, l2)
    e1, e2 = np.exp(l1 - m), np.exp(l2 - m)
    return (e1[..., None] * o1 + e2[..., None] * o2) / (e1 + e2)[..., None], m + np.log(e1 + e2)


def _online_softmax(s, v, tile=64):
    """Textbook online softmax over tiles: running max m, rescale A and L."""
    m = np.full(s.shape[0], -np.inf)
    a = np.zeros((s.shape[0], v.shape[1]))
    l = np.zeros(s.shape[0])
    for t0 in range(0, s.shape[1], tile):
        st = s[:, t0:t0 + tile]
        m2 = np.maximum(m, st.max(axis=1))
        scale = np.exp2(m - m2)
        p = np.exp2(st - m2[:, None])
        a = a * scale[:, None] + p @ v[t0:t0 + tile]
        l = l * scale + p.sum(axis=1)
        m = m2
    return a / l[:, None]


def test_additive_combine_equals_lse_merge_and_online_softmax():
    wl = make_config(2, batch=2, seq_len=1500)
    oi = _adapt.oracle_inputs(wl)
    z = _adapt.estimate(oi)
    o, _, pa, pl = _adapt.decode(oi, z, INF, [5])
    # per-split (o_s, natural-log lse_s), merged pairwise with Eq. (lse-merge)
    om, lm = None, None
    for s in range(5):
        os_ = pa[s] / pl[s][..., None]
        ls = (np.log2(pl[s]) + z) * math.log(2.0)
        om, lm = (os_, ls) if om is None else _lse_merge(om, lm, os_, ls)
    assert np.allclose(om, o, rtol=1e-11, atol=1e-13)
    q = oracle.bf16_bits_to_f64(oi["q_bits"])
    fl = oi["flat"]
    for r in range(2):
        for g in range(8):
            k = oracle.gather(oi["k_bits"], r, g, 1500, fl["block_table"], 16)
            v = oracle.gather(oi["v_bits"], r, g, 1500, fl["block_table"], 16)
            s = oracle.scores(q[r, 4 * g:4 * g + 4], k, wl.sm_scale)
            assert np.allclose(_online_softmax(s, v), o[r, 4 * g:4 * g + 4], rtol=1e-11,
                               atol=1e-13)


# ------------------------------------------------------------- P8 ----------
@pytest.mark.parametrize("cfg", [1, 2, 3, 4, 5])
def test_prop1_range_condition_every_row(cfg):
    """Prop. 1(iii) holds on every row with the estimated reference.

    The left side m - Z + log2(n nu) and L = 2^(lse - Z) are formed here
    from the generator's logical cache (before paging) with torch in FP64
    and torch's logsumexp, independently of the oracle's gather, scores and
    diagnostics; the oracle's O9 figures must agree with them."""
    wl = make_config(cfg, batch=2 if cfg != 1 else None, seq_len=2048 if cfg != 1 else None,
                     keep_logical=True)
    oi = _adapt.oracle_inputs(wl)
    z = _adapt.estimate(oi)
    q = oracle.bf16_bits_to_f64(oi["q_bits"])
    fl = oi["flat"]
    group = wl.group
    qt = wl.q.double()
    log2e = 1.0 / math.log(2.0)
    for r, n in enumerate(fl["seq_lens"]):
        for h in range(wl.num_heads):
            g = h // group
            kl = wl.logical_k[r, g, :n].double()
            vl = wl.logical_v[r, g, :n].double()
            s_ind = (kl @ qt[r, h]) * (wl.sm_scale * log2e)
            m_ind = float(s_ind.max())
            nu_ind = max(1.0, float(vl.abs().max()))
            lhs_ind = m_ind - float(z[r, h]) + math.log2(n * nu_ind)
            lse_ind = float(torch.logsumexp(s_ind * math.log(2.0), dim=0)) * log2e
            assert lhs_ind < 127.0
            k = oracle.gather(oi["k_bits"], r, g, n, fl["block_table"], wl.page_size)
            v = oracle.gather(oi["v_bits"], r, g, n, fl["block_table"], wl.page_size)
            s = oracle.scores(q[r, h:h + 1], k, wl.sm_scale)[0]
            d = oracle.row_diagnostics(s, z[r, h], INF, v)
            assert abs(d["prop1_lhs"] - lhs_ind) <= 1e-9 * max(1.0, abs(lhs_ind))
            assert abs(d["lse"] - lse_ind) <= 1e-9 * max(1.0, abs(lse_ind))
            assert abs(d["headroom"] - (lse_ind - float(z[r, h]))) <= 1e-9 * max(1.0, abs(lse_ind))
            l_ind = 2.0 ** (lse_ind - float(z[r, h]))
            assert abs(d["L"] - l_ind) <= 1e-9 * l_ind
            assert CERT_OK(l_ind)


# ------------------------------------------------------------- O9 ----------
def _row_diag_fixture():
    with open(os.path.join(GOLDEN, "row_diagnostics_example.json")) as f:
        return json.load(f)


@pytest.mark.parametrize("row", [0, 1])
def test_row_diagnostics_hand_computed(row):
    """Hand-computed fixture (exact binary fractions): every O9 figure --
    m, lse, headroom, the Prop. 1(iii) left side, L, the cut mass, the
    truncation bound and the live fraction -- at several depths, ties on
    the threshold included."""
    fx = _row_diag_fixture()
    s = np.array(fx["scores"], dtype=np.float64)
    rw = fx["rows"][row]
    v = np.array(rw["values"], dtype=np.float64)
    for case in rw["cases"]:
        d = oracle.row_diagnostics(s, rw["z"], _T(case["T"]), v)
        want = dict(rw["common"])
        want.update({k: case[k] for k in ("w_cut", "bound_T", "live_frac")})
        for key, val in want.items():
            assert d[key] == pytest.approx(val, rel=1e-15, abs=1e-300), (rw["name"], case["T"], key)


def test_row_diagnostics_fixture_is_what_its_derivation_says():
    """The fixture's own arithmetic, redone in exact rationals: sum 2^s = 16,
    L = 2^(lse - Z), the cut sets on the ties, and nu over every key."""
    from fractions import Fraction as Fr

    fx = _row_diag_fixture()
    s = [int(x) for x in fx["scores"]]
    tot = sum(Fr(2) ** e for e in s)
    assert tot == 16
    for rw in fx["rows"]:
        z = int(rw["z"])
        w = [Fr(2) ** (e - z) for e in s]
        assert sum(w) == Fr(rw["common"]["L"]) == Fr(2) ** (4 - z)
        vals = [[Fr(x) for x in row] for row in rw["values"]]
        nu = max(Fr(1), max(abs(x) for row in vals for x in row))
        lhs = max(s) - z + math.log2(len(s) * nu)
        assert lhs == rw["common"]["prop1_lhs"]
        for case in rw["cases"]:
            T = _T(case["T"])
            cut = [i for i, e in enumerate(s) if not (math.isinf(T) or e - z >= -T)]
            wc = sum((w[i] for i in cut), Fr(0))
            assert wc == Fr(case["w_cut"])
            vmax = max((max(abs(x) for x in vals[i]) for i in cut), default=Fr(0))
            assert wc / sum(w) * vmax == Fr(case["bound_T"])
            assert Fr(len(s) - len(cut), len(s)) == Fr(case["live_frac"])


def CERT_OK(l):
    return oracle.CERT_LO <= l <= oracle.CERT_HI


def test_certificate_fires_on_forced_bad_reference_and_rerun_recovers():
    """Section 3 certificate: Z far above the LSE underflows L below 2^-1, Z far
    below overflows it past 2^100; decoding again with Z = lse recovers."""
    wl = make_config(1)
    oi = _adapt.oracle_inputs(wl)
    z = _adapt.estimate(oi)
    o_ref, l_ref, _, _ = _adapt.decode(oi, z, INF, [1])
    lse, cert = oracle.lse_and_cert(z, l_ref, o_ref)
    assert (cert == 0).all()
    for shift, bit in ((140.0, 1), (-130.0, 2)):
        zb = z + shift
        o, l, _, _ = _adapt.decode(oi, zb, INF, [1])
        lse_b, cert_b = oracle.lse_and_cert(zb, l, o)
        assert ((cert_b & bit) != 0).all()
        assert np.allclose(lse_b, lse, rtol=0, atol=1e-9)
        o2, l2, _, _ = _adapt.decode(oi, lse_b, INF, [1])
        assert np.allclose(o2, o_ref, rtol=1e-12, atol=1e-14)
        assert np.allclose(l2, 1.0, rtol=1e-9)


def test_empty_row_is_nan_with_cert_bit():
    """An empty key set has L = 0: the quotient is NaN and certificate bit 2 is set."""
    a = np.zeros((1, 1, 1, 4))
    l = np.zeros((1, 1, 1))
    o, lsum = oracle.combine(a, l)
    assert np.isnan(o).all()
    _, cert = oracle.lse_and_cert(np.zeros((1, 1)), lsum, o)
    assert cert[0, 0] & 4 and cert[0, 0] & 1


# ------------------------------------------------------------- P9 ----------
@pytest.mark.parametrize("n", [1, 2, 64, 191, 192])
def test_estimator_exact_for_short_rows(n):
    """n <= 192: the estimate is the exact base-2 LSE (scipy.special.logsumexp)."""
    rng = np.random.default_rng(n)
    s = rng.normal(0.0, 30.0, size=n)
    want = scipy.special.logsumexp(s * math.log(2.0)) / math.log(2.0)
    assert abs(oracle.estimate_z(s) - want) <= 1e-12 * max(1.0, abs(want))


@pytest.mark.parametrize("n", [193, 320, 1000, 8192, 131072])
def test_estimator_constant_scores_closed_form(n):
    """All scores equal c: Z = c + log2(n) in closed form."""
    s = np.full(n, 7.25)
    assert abs(oracle.estimate_z(s) - (7.25 + math.log2(n))) < 1e-12


def _influential(s):
    """Keys whose score moves Z when pushed 8 binades up or down (beyond the
    whole spread of s, so a trimmed centre crosses to the other trimmed end and
    changes which centres are kept)."""
    z0 = oracle.estimate_z(s)
    hit = []
    for j in range(s.shape[0]):
        for d in (8.0, -8.0):
            s2 = s.copy()
            s2[j] += d
            if oracle.estimate_z(s2) != z0:
                hit.append(j)
                break
    return hit


def test_estimator_reads_hand_listed_keys_n320():
    """Brute force: perturbing key j changes Z iff j is in the hand-derived sample."""
    with open(os.path.join(GOLDEN, "estimator_n320.json")) as f:
        fx = json.load(f)
    n = fx["n"]
    want = {0} | set(range(257, 320)) | set(range(1, 256, 2))
    rng = np.random.default_rng(0)
    s = rng.normal(0.0, 0.5, size=n)
    assert set(_influential(s)) == want
    # increasing ramp: centre b has rank b, so only strata 8..119 survive the trim
    # and a small nudge is visible only on the kept centres (odd keys 17..239)
    ramp = 0.001 * np.arange(n)
    z0 = oracle.estimate_z(ramp)
    small = set()
    for j in range(n):
        s2 = ramp.copy()
        s2[j] += 1e-4
        if oracle.estimate_z(s2) != z0:
            small.add(j)
    assert small == {0} | set(range(257, 320)) | set(range(17, 240, 2))
    exact, centres, r = oracle.estimator_keys(n)
    assert r == fx["r"] and len(exact) == 64 and len(centres) == 128


@pytest.mark.parametrize("n", [193, 777, 5000])
def test_estimator_samples_one_centre_per_stratum(n):
    """Brute force on other lengths: 192 influential keys, sink and the last 63
    among them, and the 128 others spread one per 1/128 of the middle range."""
    rng = np.random.default_rng(n)
    s = rng.normal(0.0, 0.5, size=n)
    hit = _influential(s)
    assert len(hit) == 192
    assert hit[0] == 0 and hit[-63:] == list(range(n - 63, n))
    mid = np.array(hit[1:-63])
    r = n - 64
    b = np.arange(128)
    # the b-th sampled middle key sits inside the b-th 1/128 of keys 1..n-64
    assert (mid - 1 >= b * r / 128 - 1).all() and (mid - 1 <= (b + 1) * r / 128).all()


def test_estimator_trim_closed_forms():
    """Up to 8 huge centre weights are trimmed away; a 9th survives in the mean;
    a huge exact key (the sink) enters the sum exactly."""
    n = 4160
    r = n - 64
    _, centres, _ = oracle.estimator_keys(n)
    for k in (1, 8):
        s = np.zeros(n)
        s[centres[:k] if k == 1 else centres[::16][:k]] = 30.0
        assert abs(oracle.estimate_z(s) - math.log2(64 + r)) < 1e-12
    s = np.zeros(n)
    s[centres[::14][:9]] = 30.0
    want = math.log2(64 + r * (111 + 2.0 ** 30) / 112)
    assert abs(oracle.estimate_z(s) - want) < 1e-12
    s = np.zeros(n)
    s[0] = 40.0
    assert abs(oracle.estimate_z(s) - math.log2(2.0 ** 40 + 63 + r)) < 1e-12
    s = np.zeros(n)
    non_sampled = sorted(set(range(1, n - 63)) - set(centres.tolist()))[5]
    s[non_sampled] = 40.0
    assert abs(oracle.estimate_z(s) - math.log2(64 + r)) < 1e-12


# ------------------------------------------------------------- P12 ---------
def test_batch_invariance_fixed_split():
    """A request's partials depend only on its own keys: alone == in the batch."""
    wl = make_config(2, batch=3, seq_len=700)
    oi = _adapt.oracle_inputs(wl)
    z = _adapt.estimate(oi)
    o, _, _, _ = _adapt.decode(oi, z, 16.0, [4])
    one = dict(oi)
    one["q_bits"] = oi["q_bits"][1:2]
    lv = dict(oi["levels"][0])
    lv["seq_lens"] = lv["seq_lens"][1:2]
    lv["block_table"] = lv["block_table"][1:2]
    one["levels"] = [lv]
    o1, _, _, _ = _adapt.decode(one, z[1:2], 16.0, [4])
    assert np.array_equal(o1[0], o[1])
