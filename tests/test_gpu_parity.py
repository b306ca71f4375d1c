"""Parity of the HIP path (through the C ABI) with the FP64 oracle.

Bars: output per row max-abs error <= 1e-2 * |o_i|_inf (at T = inf, and at
finite T with the kernel's own verdicts imposed on the oracle); read gates
bit-exact against the oracle's rule applied to the kernel's exported FP32
x values; |Z_gpu - Z_oracle| <= 1e-3 binades; L(T) == L(inf) for a fixed Z.
"""

import math

import numpy as np
import pytest
import torch

import oracle
from tests import _adapt, _gpu
from workloads import host_bits, make_cascade, make_config, make_custom

pytestmark = pytest.mark.gpu
INF = float("inf")
TOL = 1e-2


@pytest.fixture(scope="module", autouse=True)
def _device():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2609_33410_amd as F
    F.load_library()  # raises if the HIP library is not built: never a silent fallback


def _z_parity(wl, oi, res, rows=None):
    zo = _adapt.estimate(oi, rows=rows)
    zg = res["z"].double().numpy()
    if rows is None:
        diff = np.abs(zg - zo).max()
    else:
        diff = max(abs(zg[r, h] - zo[r, h]) for r, h in rows)
    print(f"  Z parity: max |dZ| = {diff:.3e} binades")
    assert diff <= 1e-3


def _gate_check(wl, oi, res, T):
    """Key/page read bits equal the FP32 rule on the exported x, ORed per read group."""
    G = wl.group
    for li, lv in enumerate(oi["levels"]):
        dbg = res["dbg"][li]
        x = dbg["x"].numpy()
        R = dbg["R"]
        for seq, n in enumerate(lv["seq_lens"]):
            if lv["row_indptr"] is None:
                reqs = [seq]
            else:
                reqs = list(lv["row_req"][lv["row_indptr"][seq]:lv["row_indptr"][seq + 1]])
            for g in range(wl.num_kv_heads):
                rows = [(int(r), g * G + hh) for r in reqs for hh in range(G)]
                for u in range((len(rows) + R - 1) // R):
                    grp = rows[u * R:(u + 1) * R]
                    xs = np.stack([x[r, h, :n] for r, h in grp])
                    assert np.isfinite(xs).all(), "x export must cover every key"
                    live = oracle.live_mask_imposed(xs, T)
                    key, page = oracle.read_gates(live, n)
                    kg = dbg["kg"][seq, g, u, :n].numpy().astype(bool)
                    pg = dbg["pg"][seq, g, u, :(n + 15) // 16].numpy().astype(bool)
                    assert np.array_equal(kg, key), f"key gates differ (level {li} seq {seq} head {g})"
                    assert np.array_equal(pg, page), f"page gates differ (level {li} seq {seq} head {g})"


def _x_check(wl, oi, res, z64, chunks=None):
    """The exported x equals the oracle's s - Z to FP32 rounding (on the listed
    (kv sequence, kv head) chunks, or all)."""
    q = oracle.bf16_bits_to_f64(oi["q_bits"])
    G = wl.group
    worst = 0.0
    for li, lv in enumerate(oi["levels"]):
        x = res["dbg"][li]["x"].numpy()
        for seq, n in enumerate(lv["seq_lens"]):
            if lv["row_indptr"] is None:
                reqs = [seq]
            else:
                reqs = list(lv["row_req"][lv["row_indptr"][seq]:lv["row_indptr"][seq + 1]])
            for g in range(wl.num_kv_heads):
                if chunks is not None and (seq, g) not in chunks:
                    continue
                keys = oracle.gather(oi["k_bits"], seq, g, n, lv["block_table"], wl.page_size)
                for r in reqs:
                    hs = [g * G + hh for hh in range(G)]
                    s = oracle.scores(q[r, hs], keys, wl.sm_scale)
                    ref = s - z64[r, hs][:, None]
                    err = np.abs(x[r, hs, :n] - ref) / np.maximum(1.0, np.abs(s))
                    worst = max(worst, float(err.max()) if n else 0.0)
    print(f"  x parity: max rel err = {worst:.3e}")
    assert worst <= 1e-5


def _full_parity(wl, T, splits=None, own_mode=True, check_gates=True):
    oi = _adapt.oracle_inputs(wl)
    res = _gpu.run(wl, T, splits=splits, debug=True)
    _z_parity(wl, oi, res)
    z64 = res["z"].double().numpy()
    splits = res["splits"]
    imposed = [d["x"].numpy() for d in res["dbg"]]
    o_imp, l_imp, pa, pl = _adapt.decode(oi, z64, T, splits, imposed=imposed)
    err = _gpu.row_errors(res["out"].numpy(), o_imp)
    ok_rows = l_imp > 0
    print(f"  {wl.name} T={T} S={splits}: max row err (imposed) = {err[ok_rows].max():.3e}, "
          f"rel l2 = {_gpu.rel_l2(res['out'].numpy()[ok_rows], o_imp[ok_rows]):.3e}")
    assert (err[ok_rows] <= TOL).all()
    # partial sums per slot: L is a sum of positive terms, compare tightly
    gl = res["part_L"].double().numpy()
    cov = pl > 0
    assert np.allclose(gl[cov], pl[cov], rtol=2e-5, atol=0)
    assert (gl[~cov] == 0).all()
    if check_gates:
        _x_check(wl, oi, res, z64)
        _gate_check(wl, oi, res, T)
    if own_mode and not math.isinf(T):
        o_own, l_own, _, _ = _adapt.decode(oi, z64, T, splits)
        err_own = _gpu.row_errors(res["out"].numpy(), o_own)
        # stated bound: TOL plus 2 * 2^-T * N_flip * max|v| / L for keys whose
        # FP64 and FP32 verdicts differ
        flips = _flip_counts(wl, oi, res, z64, T)
        vmax = float(np.abs(oracle.bf16_bits_to_f64(oi["v_bits"])).max())
        bound = TOL + 2.0 * 2.0 ** -T * flips * vmax / np.maximum(l_own, 1e-300) \
            / np.maximum(np.abs(o_own).max(axis=-1), 1e-300)
        print(f"  own-mode max row err = {err_own[ok_rows].max():.3e}, flips = {int(flips.sum())}")
        assert (err_own[ok_rows] <= bound[ok_rows]).all()
    return res, oi


def _flip_counts(wl, oi, res, z64, T, chunks=None):
    q = oracle.bf16_bits_to_f64(oi["q_bits"])
    b, h = z64.shape
    flips = np.zeros((b, h))
    G = wl.group
    for li, lv in enumerate(oi["levels"]):
        x = res["dbg"][li]["x"].numpy()
        for seq, n in enumerate(lv["seq_lens"]):
            reqs = [seq] if lv["row_indptr"] is None else \
                list(lv["row_req"][lv["row_indptr"][seq]:lv["row_indptr"][seq + 1]])
            for g in range(wl.num_kv_heads):
                if chunks is not None and (seq, g) not in chunks:
                    continue
                keys = oracle.gather(oi["k_bits"], seq, g, n, lv["block_table"], wl.page_size)
                for r in reqs:
                    hs = [g * G + hh for hh in range(G)]
                    s = oracle.scores(q[r, hs], keys, wl.sm_scale)
                    own = oracle.live_mask(s - z64[r, hs][:, None], T)
                    imp = oracle.live_mask_imposed(x[r, hs, :n], T)
                    flips[r, hs] += (own != imp).sum(axis=1)
    return flips


# ---------------------------------------------------------------- tiny ------
@pytest.mark.parametrize("splits", [1, 4])
@pytest.mark.parametrize("T", [INF, 16.0])
def test_config1_tiny_mha(splits, T):
    wl = make_config(1, device="cuda")
    _full_parity(wl, T, splits=[splits])


@pytest.mark.parametrize("splits", [1, 3, 8])
@pytest.mark.parametrize("T", [INF, 16.0, 4.0])
def test_config2_shape_small(splits, T):
    wl = make_config(2, batch=2, seq_len=1000, device="cuda")
    _full_parity(wl, T, splits=[splits])


@pytest.mark.parametrize("d", [64, 128])
@pytest.mark.parametrize("group", [1, 2, 4, 8])
@pytest.mark.parametrize("paged", [True, False])
def test_ragged_edge_lengths(d, group, paged):
    """Empty, single-key, page- and tile-boundary lengths; partial last tiles."""
    lens = [0, 1, 15, 16, 17, 63, 64, 65, 200, 333]
    wl = make_custom(batch=len(lens), heads=2 * group, kv_heads=2, dim=d, lens=lens,
                     paged=paged, spike_count=2, n_sink=1, seed=d + group, device="cuda")
    for T, s in ((INF, 1), (6.0, 3), (16.0, 5)):
        res, oi = _full_parity(wl, T, splits=[s], own_mode=False)
        empty = res["part_L"].sum(0).numpy()[0]
        assert (empty == 0).all()
        assert torch.isnan(res["out"][0]).all()
        assert ((res["cert"][0].numpy() & 5) == 5).all()  # L < 2^-1 and non-finite
        assert (res["cert"][1:].numpy() & 2 == 0).all()


@pytest.mark.parametrize("d", [64, 128])
@pytest.mark.parametrize("splits", [1, 3, 5])
def test_mha_waves_per_workgroup(d, splits):
    """The MHA scan with 8 and 4 waves sharing a split's tiles (chosen from the
    longest sequence per split: 2100 keys give 132 chunks, so S = 1 and 3 take
    8 waves, S = 5 four), sequences dispatched longest first, ragged lengths
    with partial last tiles, an empty and a short sequence; output, slots, x
    and read bits against the oracle."""
    lens = [2100, 1100, 2053, 0, 77]
    wl = make_custom(batch=len(lens), heads=3, kv_heads=3, dim=d, lens=lens, paged=True,
                     spike_count=6, n_sink=1, seed=40 + d + splits, device="cuda")
    for T in (INF, 16.0, 4.0):
        _full_parity(wl, T, splits=[splits], own_mode=not math.isinf(T))


def test_page_size_64_and_dim64_gqa8():
    wl = make_custom(batch=3, heads=16, kv_heads=2, dim=64, lens=[500, 129, 64], page_size=64,
                     spike_count=5, n_sink=4, seed=9, device="cuda")
    for T in (INF, 16.0):
        _full_parity(wl, T, splits=[2])


@pytest.mark.parametrize("d", [64, 128])
@pytest.mark.parametrize("requests,prefix,splits,shallow", [(5, 1488, (3, 2), 6.0),
                                                            (8, 1024, (1, 1), 6.0),
                                                            (12, 2000, (4, 3), 6.0),
                                                            (17, 80, (2, 1), 4.0)])
def test_stacked_rows_cascade(d, requests, prefix, splits, shallow):
    """Prefix levels of more than 32 stacked rows (the stacked-row scan): 40 rows
    (one partial read group), 64 (one full group), 96 (a full and a partial group)
    and 136 (three groups); prefixes ending inside a 64-key tile and fewer tiles
    than splits.  At the shallow depth most 32-key halves of a tile are unread
    while a quarter to half of the rows keep live keys."""
    wl = make_cascade(requests=requests, heads=8, kv_heads=1, dim=d, prefix_len=prefix,
                      suffix_len=48, splits=splits, seed=requests + d, device="cuda")
    for T in (INF, 16.0, shallow):
        _full_parity(wl, T)


@pytest.mark.parametrize("heads,kv_heads,requests", [(4, 2, 2), (8, 2, 2), (4, 1, 2), (2, 1, 3)])
def test_small_stacked_groups(heads, kv_heads, requests):
    """Prefix levels of 4 to 8 stacked rows: the GQA groups (of 2 or 4 rows) of
    two or three requests share the row lanes of one packed chunk, so their
    verdicts, read bits and sums must stay apart."""
    wl = make_cascade(requests=requests, heads=heads, kv_heads=kv_heads, dim=128,
                      prefix_len=720, suffix_len=48, splits=(3, 1),
                      seed=heads + kv_heads + requests, device="cuda")
    for T in (INF, 16.0, 6.0):
        _full_parity(wl, T)


def test_stacked_rows_two_kv_heads():
    """Eight heads on two kv heads with 24 requests: 96 stacked rows per (prefix, kv head)."""
    wl = make_cascade(requests=24, heads=8, kv_heads=2, dim=128, prefix_len=784, suffix_len=32,
                      splits=(2, 1), seed=3, device="cuda")
    for T in (INF, 6.0):
        _full_parity(wl, T)


# ------------------------------------------------------- invariants ---------
def test_mass_kept_L_independent_of_T():
    wl = make_config(2, batch=2, seq_len=3000, device="cuda")
    z = _gpu.estimate(wl)
    a = _gpu.run(wl, INF, splits=[4], z=z)
    for T in (24.0, 16.0, 2.0, 0.0):
        b = _gpu.run(wl, T, splits=[4], z=z)
        assert torch.equal(a["part_L"], b["part_L"])


@pytest.mark.parametrize("cfg,T,batch", [(1, INF, None), (1, 16.0, None), (2, INF, 4),
                                         (2, 16.0, 4), (5, 16.0, 4), (5, INF, 12), (5, 6.0, 12),
                                         (5, 2.0, 12)])
def test_debug_exports_do_not_change_results(cfg, T, batch):
    """The kernel variant that exports x and read gates computes the same bits
    as the production variant, so the exported decisions are the production
    kernel's decisions.  Config 5 with 4 requests stacks 32 rows on the prefix;
    with 12 requests, 96 rows (the stacked-row scan, two read groups), whose
    production kernel fetches values with their keys at finite depth while the
    debug variant fetches only the live ones: the same bits."""
    wl = make_config(cfg, device="cuda", batch=batch, seq_len=None if cfg == 1 else 1500)
    z = _gpu.estimate(wl)
    a = _gpu.run(wl, T, z=z, debug=False)
    b = _gpu.run(wl, T, z=z, debug=True)
    assert torch.equal(a["part_A"], b["part_A"]) and torch.equal(a["part_L"], b["part_L"])


def test_repeat_bits_and_batch_invariance():
    wl = make_config(2, batch=4, seq_len=2000, device="cuda")
    z = _gpu.estimate(wl)
    a = _gpu.run(wl, 16.0, splits=[4], z=z)
    b = _gpu.run(wl, 16.0, splits=[4], z=z)
    assert torch.equal(a["out"], b["out"]) and torch.equal(a["part_A"], b["part_A"])
    # request 2 alone (its own q row and table) gives the same bits
    import copy
    one = copy.copy(wl)
    one.q = wl.q[2:3].contiguous()
    lv = copy.copy(wl.levels[0])
    lv.block_table = lv.block_table[2:3].contiguous()
    lv.seq_lens = lv.seq_lens[2:3].contiguous()
    lv.seq_lens_host = lv.seq_lens_host[2:3]
    one.levels = [lv]
    fl = copy.copy(wl.flat)
    fl.block_table, fl.seq_lens, fl.seq_lens_host = lv.block_table, lv.seq_lens, lv.seq_lens_host
    one.flat = fl
    c = _gpu.run(one, 16.0, splits=[4], z=z[2:3].contiguous())
    assert torch.equal(c["out"][0], a["out"][2])
    assert torch.equal(c["z"][0], a["z"][2])


def test_bf16_output_is_rne_of_fp32():
    wl = make_config(2, batch=2, seq_len=777, device="cuda")
    z = _gpu.estimate(wl)
    a = _gpu.run(wl, INF, splits=[3], z=z)
    b = _gpu.run(wl, INF, splits=[3], z=z, out_dtype=torch.bfloat16)
    assert torch.equal(b["out"], a["out"].to(torch.bfloat16))


def test_certificate_forced_bad_reference_and_rerun():
    """Z far above the LSE: L < 2^-1 (bit0); far below: L > 2^100 (bit1); a
    rerun with Z = lse clears the flags and matches the oracle."""
    wl = make_config(1, device="cuda")
    oi = _adapt.oracle_inputs(wl)
    base = _gpu.run(wl, INF, splits=[1])
    assert (base["cert"] == 0).all()
    z = base["z"].cuda()
    # +140 binades flushes every FP32 weight (L = 0): the flag fires, but lse is
    # -inf and cannot seed a rerun.  lse + 20 and lse - 110 keep L representable.
    bad = _gpu.run(wl, INF, splits=[1], z=(z + 140.0).contiguous())
    assert ((bad["cert"].numpy() & 1) != 0).all()
    lse = base["lse"].cuda()
    for shift, bit in ((20.0, 1), (-110.0, 2)):
        bad = _gpu.run(wl, INF, splits=[1], z=(lse + shift).contiguous())
        assert ((bad["cert"].numpy() & bit) != 0).all()
        rerun = _gpu.run(wl, INF, splits=[1], z=bad["lse"].cuda().contiguous())
        assert (rerun["cert"] == 0).all()
        o_ref, _, _, _ = _adapt.decode(oi, rerun["z"].double().numpy(), INF, [1])
        assert (_gpu.row_errors(rerun["out"].numpy(), o_ref) <= TOL).all()


# ------------------------------------------------- full-size, sampled ------
def _sampled(wl, T, chunks, check_gates=False, own_mode=False):
    """Full-size run on the GPU; the oracle recomputes the sampled
    (kv sequence, kv head) chunks of a flat workload one by one.

    With ``check_gates`` the kernel's debug exports are taken: the key and page
    read bits of EVERY chunk of the call must equal the FP32 rule applied to
    the exported x (bit-exact), and the exported x of the sampled chunks must
    equal the oracle's s - Z.  With ``own_mode`` (finite T) the sampled rows
    are also held to the stated bound against the oracle's own FP64
    decisions: the 1e-2 row bar plus 2 * 2^-T * N_flip * max|v| / L."""
    debug = check_gates or own_mode
    res = _gpu.run(wl, T, debug=debug)
    oi = _adapt.oracle_inputs(wl)
    G = wl.group
    rows = [(r, g * G + hh) for r, g in chunks for hh in range(G)]
    _z_parity(wl, oi, res, rows=rows)
    z64 = res["z"].double().numpy()
    lv = oi["levels"][0]
    S = res["splits"][0]
    x = res["dbg"][0]["x"].numpy() if debug else None
    pa, pl = oracle.decode_level(oi["q_bits"], oi["k_bits"], oi["v_bits"],
                                 num_kv_heads=wl.num_kv_heads, page_size=wl.page_size,
                                 sm_scale=wl.sm_scale, z=z64, T=T, num_splits=S,
                                 chunks=chunks, imposed_x=x, **lv)
    o_ref, l_ref = oracle.combine(pa, pl)
    ri = np.array([r for r, _ in rows])
    hi = np.array([h for _, h in rows])
    err = _gpu.row_errors(res["out"].numpy()[ri, hi], o_ref[ri, hi])
    print(f"  {wl.name} T={T}: sampled rows {len(rows)}, max row err = {err.max():.3e}")
    assert (err <= TOL).all()
    gl = res["part_L"].double().numpy()[:, ri, hi]
    assert np.allclose(gl, pl[:, ri, hi], rtol=2e-5, atol=0)
    if check_gates:
        _gate_check(wl, oi, res, T)
        _x_check(wl, oi, res, z64, chunks=chunks)
    if own_mode and not math.isinf(T):
        pa_o, pl_o = oracle.decode_level(oi["q_bits"], oi["k_bits"], oi["v_bits"],
                                         num_kv_heads=wl.num_kv_heads, page_size=wl.page_size,
                                         sm_scale=wl.sm_scale, z=z64, T=T, num_splits=S,
                                         chunks=chunks, **lv)
        o_own, l_own = oracle.combine(pa_o, pl_o)
        flips = _flip_counts(wl, oi, res, z64, T, chunks=chunks)
        vmax = float(np.abs(oracle.bf16_bits_to_f64(oi["v_bits"])).max())
        scale = np.maximum(np.abs(o_own[ri, hi]).max(axis=-1), 1e-300)
        bound = TOL + 2.0 * 2.0 ** -T * flips[ri, hi] * vmax / np.maximum(l_own[ri, hi], 1e-300) \
            / scale
        err_own = _gpu.row_errors(res["out"].numpy()[ri, hi], o_own[ri, hi])
        print(f"  own-mode max row err = {err_own.max():.3e}, flips = {int(flips[ri, hi].sum())}, "
              f"min bound = {bound.min():.3e}")
        assert (err_own <= bound).all()
    return res


@pytest.mark.parametrize("T", [INF, 16.0])
def test_config2_full_size_sampled(T):
    """One (request, kv head) chunk of every request; at T = 16 the read bits of
    the whole call bit-exact and the own-mode stated bound."""
    wl = make_config(2, device="cuda")
    _sampled(wl, T, chunks=[(r, (3 * r) % 8) for r in range(16)],
             check_gates=not math.isinf(T), own_mode=not math.isinf(T))


@pytest.mark.parametrize("T", [INF, 24.0, 16.0, 12.0])
def test_config3_full_size_sampled(T):
    """Every configured depth of the Qwen3-8B-shaped 32K decode."""
    wl = make_config(3, device="cuda")
    _sampled(wl, T, chunks=[(0, 0), (3, 5), (7, 7)], check_gates=not math.isinf(T),
             own_mode=not math.isinf(T))


@pytest.mark.parametrize("T", [INF, 16.0])
def test_config4_full_size_sampled(T):
    """The MHA 64K-128K decode (ragged, 32 splits): sampled rows of every
    request; at T = 16 the read bits of the whole call bit-exact and the
    own-mode stated bound."""
    wl = make_config(4, device="cuda")
    _sampled(wl, T, chunks=[(0, 0), (1, 17), (2, 9), (3, 31)],
             check_gates=not math.isinf(T), own_mode=not math.isinf(T))


@pytest.mark.parametrize("T", [INF, 16.0])
def test_config5_cascade_full(T):
    """Prefix level (1 kv sequence x 512 stacked rows) + suffix level, added."""
    wl = make_config(5, device="cuda")
    res = _gpu.run(wl, T, debug=False)
    oi = _adapt.oracle_inputs(wl)
    rows = [(r, h) for r in (0, 31, 63) for h in range(8)]
    _z_parity(wl, oi, res, rows=rows)
    z64 = res["z"].double().numpy()
    o_ref, l_ref, pa, pl = _adapt.decode(oi, z64, T, res["splits"])
    err = _gpu.row_errors(res["out"].numpy(), o_ref)
    print(f"  cascade T={T}: max row err = {err.max():.3e}")
    assert (err <= TOL).all()
    assert np.allclose(res["part_L"].double().numpy(), pl, rtol=2e-5, atol=0)
