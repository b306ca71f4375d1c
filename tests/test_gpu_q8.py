"""Parity of the two-plane INT8 key path (through the C ABI) with the FP64 oracle.

Bars: cache codes, query codes, eta and tau bit-exact; |Z_gpu - Z_oracle| <=
1e-3 binades; output per row max-abs error <= 1e-2 * |o_i|_inf with the
kernel's FP32 decisions imposed on the oracle, and within that plus the
stated flip bound in the oracle's own FP64 decisions; value-row, page and
plane-B read bits bit-exact against the oracle's group rule applied to the
kernel's exported FP32 coarse scores.
"""

import math

import numpy as np
import pytest
import torch

from oracle import bf16_bits_to_f64, combine
from oracle import q8_oracle as q8
from tests import _adapt, _gpu, _gpu_q8
import paper_2609_33410_amd as F
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


def _oracle_planes(wl, pages=None):
    """The oracle's own codes of the stored keys (all pages, or only ``pages``
    of a paged cache; the other entries stay zero)."""
    kb = host_bits(wl.k) if pages is None else None
    if pages is None:
        return q8.split_keys(kb)
    shape = tuple(wl.k.shape)
    a = np.zeros(shape, dtype=np.int8)
    b = np.zeros(shape, dtype=np.int8)
    e = np.zeros(shape[:-1], dtype=np.uint16)
    idx = torch.as_tensor(sorted(pages), dtype=torch.long, device=wl.k.device)
    sub = host_bits(wl.k.index_select(0, idx))
    pa, pb, pe = q8.split_keys(sub)
    a[idx.cpu().numpy()], b[idx.cpu().numpy()], e[idx.cpu().numpy()] = pa, pb, pe
    return a, b, e


def _gpu_planes(keys):
    return (keys.plane_a.cpu().numpy(), keys.plane_b.cpu().numpy(),
            keys.scale.cpu().numpy().view(np.uint16))


def _query_codes(wl, kappa):
    qa, qb, eta = q8.split_queries(host_bits(wl.q), wl.sm_scale)
    tau = np.array([q8.refine_tau(n, kappa) for n in wl.flat.seq_lens_host], dtype=np.float32)
    return qa, qb, eta, tau


def _check_query_codes(res, qa, qb, eta, tau):
    planes = res["planes"].numpy()
    assert np.array_equal(planes[:, :, 0], qa) and np.array_equal(planes[:, :, 1], qb)
    assert np.array_equal(res["eta"].numpy().view(np.uint32), eta.view(np.uint32))
    assert np.array_equal(res["tau"].numpy().view(np.uint32), tau.view(np.uint32))


def _rows_of(lv, seq, g, group):
    reqs = [seq] if lv["row_indptr"] is None else \
        [int(r) for r in lv["row_req"][lv["row_indptr"][seq]:lv["row_indptr"][seq + 1]]]
    return [(r, g * group + hh) for r in reqs for hh in range(group)]


def _gate_check(wl, oi, res, T, tau):
    """Read bits equal the oracle's group rule on the exported FP32 coarse x,
    ORed over each read group."""
    G = wl.group
    for li, lv in enumerate(oi["levels"]):
        dbg = res["dbg"][li]
        xc = dbg["xc_out"].numpy()
        R = dbg["R"]
        for seq, n in enumerate(lv["seq_lens"]):
            for g in range(wl.num_kv_heads):
                rows = _rows_of(lv, seq, g, G)
                for u in range((len(rows) + R - 1) // R):
                    grp = rows[u * R:(u + 1) * R]
                    xs = np.stack([xc[r, h, :n] for r, h in grp])
                    assert np.isfinite(xs).all(), "xc export must cover every key"
                    blocks = np.array([k // G for k in range(len(grp))])
                    live, ref = q8.gate_bits(xs, blocks, T, tau[[r for r, _ in grp]], f32=True)
                    vkey, vpage, bkey = q8.q8_read_gates(live, ref, n)
                    kg = dbg["key_gate_out"][seq, g, u, :n].numpy().astype(bool)
                    pg = dbg["page_gate_out"][seq, g, u, :(n + 15) // 16].numpy().astype(bool)
                    rg = dbg["refine_gate_out"][seq, g, u, :n].numpy().astype(bool)
                    where = f"level {li} seq {seq} head {g} group {u}"
                    assert np.array_equal(kg, vkey), "value-row bits differ: " + where
                    assert np.array_equal(pg, vpage), "page bits differ: " + where
                    assert np.array_equal(rg, bkey), "plane-B bits differ: " + where


def _decode_oracle(wl, oi, planes, qa, qb, eta, tau, z64, T, splits, imposed=None):
    pa_all, pl_all = [], []
    for li, lv in enumerate(oi["levels"]):
        imp = None if imposed is None else imposed[li]
        pa, pl = q8.decode_level_q8(qa, qb, eta, planes, oi["v_bits"],
                                    num_kv_heads=wl.num_kv_heads, page_size=wl.page_size, z=z64,
                                    T=T, tau=tau, num_splits=splits[li], imposed=imp, **lv)
        pa_all.append(pa)
        pl_all.append(pl)
    pa = np.concatenate(pa_all)
    pl = np.concatenate(pl_all)
    o, l = combine(pa, pl)
    return o, l, pa, pl


def _own_flips(wl, oi, planes, qa, qb, eta, tau, z64, T, res):
    """Per row: keys whose FP64 cut (x >= -T) and refine bit differ from the
    kernel's FP32 decisions; returns (cut flips, refine flips)."""
    b, h = z64.shape
    cut = np.zeros((b, h))
    ref_f = np.zeros((b, h))
    for li, lv in enumerate(oi["levels"]):
        _, _, info = q8.decode_level_q8(qa, qb, eta, planes, oi["v_bits"],
                                        num_kv_heads=wl.num_kv_heads, page_size=wl.page_size,
                                        z=z64, T=T, tau=tau, num_splits=1, want_scores=True, **lv)
        xg = res["dbg"][li]["x_out"].numpy()
        xcg = res["dbg"][li]["xc_out"].numpy()
        for (seq, g), (rows, xc, x, live, ref) in info.items():
            n = xc.shape[1]
            ri = np.array([r for r, _ in rows])
            hi = np.array([hh for _, hh in rows])
            blocks = np.repeat(np.arange(len(rows) // wl.group), wl.group)
            _, ref_g = q8.gate_bits(xcg[ri, hi, :n], blocks, T, tau[ri], f32=True)
            if not math.isinf(T):
                cut[ri, hi] += ((x >= -T) != (xg[ri, hi, :n] >= np.float32(-T))).sum(axis=1)
            ref_f[ri, hi] += (ref != ref_g).sum(axis=1)
    return cut, ref_f


def _full_parity(wl, T, kappa=0.0, splits=None, own_mode=True):
    oi = _adapt.oracle_inputs(wl)
    planes = _oracle_planes(wl)
    qa, qb, eta, tau = _query_codes(wl, kappa)
    zo = q8.estimate_level_q8(qa, qb, eta, planes, num_kv_heads=wl.num_kv_heads,
                              page_size=wl.page_size, seq_lens=oi["flat"]["seq_lens"],
                              block_table=oi["flat"]["block_table"])
    # the estimator takes GQA groups of up to 16 rows; larger groups get the
    # oracle's estimate as their declared reference
    z_in = torch.from_numpy(zo).float().cuda() if wl.group > 16 else None
    res, keys = _gpu_q8.run(wl, T, kappa=kappa, splits=splits, debug=True, z=z_in)
    for got, want, nm in zip(_gpu_planes(keys), planes, ("plane A", "plane B", "scale")):
        assert np.array_equal(got, want), nm + " codes differ from the oracle's"
    _check_query_codes(res, qa, qb, eta, tau)
    z64 = res["z"].double().numpy()
    dz = np.abs(z64 - zo).max()
    assert dz <= 1e-3, f"Z differs by {dz:.3e} binades"
    splits = res["splits"]
    imposed = [(d["xc_out"].numpy(), d["x_out"].numpy()) for d in res["dbg"]]
    o_imp, l_imp, pa, pl = _decode_oracle(wl, oi, planes, qa, qb, eta, tau, z64, T, splits,
                                          imposed=imposed)
    ok_rows = l_imp > 0
    err = _gpu.row_errors(res["out"].numpy(), o_imp)
    print(f"  q8 {wl.name} T={T} kappa={kappa} S={splits}: max row err (imposed) = "
          f"{err[ok_rows].max() if ok_rows.any() else 0:.3e}, dZ = {dz:.2e}")
    assert (err[ok_rows] <= TOL).all()
    gl = res["part_L"].double().numpy()
    cov = pl > 0
    assert np.allclose(gl[cov], pl[cov], rtol=2e-5, atol=0)
    assert (gl[~cov] == 0).all()
    _gate_check(wl, oi, res, T, tau)
    if own_mode:
        o_own, l_own, _, _ = _decode_oracle(wl, oi, planes, qa, qb, eta, tau, z64, T, splits)
        err_own = _gpu.row_errors(res["out"].numpy(), o_own)
        cut, ref_f = _own_flips(wl, oi, planes, qa, qb, eta, tau, z64, T, res)
        vmax = float(np.abs(bf16_bits_to_f64(oi["v_bits"])).max())
        # stated bound: a key whose cut differs carries weight about 2^-T, one
        # whose refine bit differs about 2^-tau (relative to 2^Z), and moves
        # the output by at most twice its weight times max|v| over L
        w_cut = 0.0 if math.isinf(T) else 2.0 ** -T
        tau_rows = np.repeat(tau[:, None], z64.shape[1], axis=1).astype(np.float64)
        w_ref = np.where(np.isfinite(tau_rows), 2.0 ** -np.where(np.isfinite(tau_rows),
                                                                 tau_rows, 0.0), 0.0)
        moved = 2.0 * (cut * w_cut + ref_f * w_ref) * vmax / np.maximum(l_own, 1e-300)
        bound = TOL + moved / np.maximum(np.abs(o_own).max(axis=-1), 1e-300)
        print(f"  own-mode max row err = {err_own[ok_rows].max():.3e}, "
              f"cut flips = {int(cut.sum())}, refine flips = {int(ref_f.sum())}")
        assert (err_own[ok_rows] <= bound[ok_rows]).all()
    return res, oi


# ---------------------------------------------------------------- writer ----
def test_paged_writer_appends_and_skips():
    """The writer through a paged view: every valid (sequence, position) gets
    the oracle's code at its page slot; tokens past a sequence's capacity, of
    an unknown sequence or on an invalid page id leave the cache untouched."""
    import paper_2609_33410_amd as F
    wl = make_custom(batch=3, heads=8, kv_heads=2, dim=128, lens=[40, 17, 64], spike_count=2,
                     n_sink=1, seed=5, device="cuda")
    fl = wl.flat
    bt = fl.block_table.clone()
    bt[2, 1] = 10 ** 6  # an invalid page id: writes there are skipped
    kv = F.kv_view(wl.k, None, fl.seq_lens, num_kv_heads=2, max_seq_len=fl.max_seq_len,
                   block_table=bt)
    keys = F.q8_empty_keys(wl.k)
    for t in (keys.plane_a, keys.plane_b):
        t.fill_(0x33)
    keys.scale.fill_(0x3333)
    seqs, poss = [], []
    for r, n in enumerate(fl.seq_lens_host):
        seqs += [r] * n
        poss += list(range(n))
    seqs += [0, 7, -1, 1]
    poss += [fl.block_table.shape[1] * 16, 0, 3, -2]      # past capacity / bad seq / bad pos
    n_tok = len(seqs)
    # token t carries the logical key of (seq, pos) when valid, noise otherwise
    g = torch.Generator(device="cpu").manual_seed(1)
    k_src = torch.randn(n_tok, 2, 128, generator=g).to(torch.bfloat16)
    logical = torch.zeros(3, 2, 64, 128, dtype=torch.bfloat16)
    for t in range(n_tok - 4):
        logical[seqs[t], :, poss[t]] = k_src[t]
    F.fold_q8_write_keys(kv, k_src.cuda(), torch.tensor(seqs, dtype=torch.int32).cuda(),
                         torch.tensor(poss, dtype=torch.int32).cuda(), keys)
    torch.cuda.synchronize()
    ga, gb, ge = _gpu_planes(keys)
    table = bt.cpu().numpy()
    written = np.zeros(ga.shape[:3], dtype=bool)
    for r, n in enumerate(fl.seq_lens_host):
        a, b, e = q8.split_keys(host_bits(logical[r, :, :n]))
        for j in range(n):
            page = int(table[r, j // 16])
            if page >= ga.shape[0]:
                continue
            written[page, :, j % 16] = True
            assert np.array_equal(ga[page, :, j % 16], a[:, j])
            assert np.array_equal(gb[page, :, j % 16], b[:, j])
            assert np.array_equal(ge[page, :, j % 16], e[:, j])
    assert (ga[~written] == 0x33).all() and (gb[~written] == 0x33).all()
    assert (ge[~written] == 0x3333).all()


# ---------------------------------------------------------------- tiny ------
@pytest.mark.parametrize("splits", [1, 4])
@pytest.mark.parametrize("T", [INF, 16.0])
def test_q8_config1_tiny_mha(splits, T):
    wl = make_config(1, device="cuda")
    _full_parity(wl, T, splits=[splits])


@pytest.mark.parametrize("kappa", [0.0, -INF, INF, -6.0])
@pytest.mark.parametrize("T", [INF, 16.0, 4.0])
def test_q8_config2_shape_small(kappa, T):
    wl = make_config(2, batch=2, seq_len=1000, device="cuda")
    _full_parity(wl, T, kappa=kappa, splits=[3])


@pytest.mark.parametrize("d", [64, 128])
@pytest.mark.parametrize("group", [1, 4, 16, 32])
@pytest.mark.parametrize("paged", [True, False])
def test_q8_ragged_edge_lengths(d, group, paged):
    """Empty, single-key, page- and tile-boundary lengths; partial last tiles;
    GQA groups from 1 to 32 rows (32: a read group of two 16-row blocks)."""
    lens = [0, 1, 15, 16, 17, 63, 64, 65, 200, 333]
    wl = make_custom(batch=len(lens), heads=2 * group, kv_heads=2, dim=d, lens=lens,
                     paged=paged, spike_count=2, n_sink=1, seed=d + group, device="cuda")
    for T, s, kappa in ((INF, 1, 0.0), (6.0, 3, 0.0), (16.0, 5, -4.0)):
        res, _ = _full_parity(wl, T, kappa=kappa, splits=[s], own_mode=False)
        assert (res["part_L"].sum(0).numpy()[0] == 0).all()
        assert torch.isnan(res["out"][0]).all()


@pytest.mark.parametrize("d", [64, 128])
@pytest.mark.parametrize("splits", [1, 3, 5])
def test_q8_mha_ragged_longest_first(d, splits):
    """MHA (one row per kv sequence and head: the VALU two-plane scan) over
    ragged lengths dispatched longest first, several splits and depths."""
    wl = make_custom(batch=5, heads=4, kv_heads=4, dim=d, lens=[2100, 1100, 2053, 0, 77],
                     spike_count=6, n_sink=1, seed=d + splits, device="cuda")
    for T, kappa in ((INF, 0.0), (16.0, -4.0), (6.0, 2.0)):
        _full_parity(wl, T, kappa=kappa, splits=[splits])


@pytest.mark.parametrize("requests,prefix,splits", [(5, 1488, (3, 2)), (3, 80, (2, 1))])
def test_q8_cascade_stacked_rows(requests, prefix, splits):
    """Shared-prefix levels: 40 and 24 stacked rows of 8-head GQA groups in
    read groups of 32 (gates per request, read bits per read group)."""
    wl = make_cascade(requests=requests, heads=8, kv_heads=1, dim=128, prefix_len=prefix,
                      suffix_len=48, splits=splits, seed=requests, device="cuda")
    for T in (INF, 16.0, 6.0):
        _full_parity(wl, T)


@pytest.mark.parametrize("heads,kv_heads,requests", [(4, 2, 2), (8, 2, 2), (2, 1, 3)])
def test_q8_small_stacked_groups(heads, kv_heads, requests):
    """Prefix levels of 4 to 8 stacked rows: two or three requests' GQA groups
    share the row lanes of one packed chunk; the refine and value verdicts are
    per group, the read bits per read group."""
    wl = make_cascade(requests=requests, heads=heads, kv_heads=kv_heads, dim=128,
                      prefix_len=720, suffix_len=48, splits=(3, 1),
                      seed=heads + kv_heads + requests, device="cuda")
    for T in (INF, 16.0, 6.0):
        _full_parity(wl, T)


@pytest.mark.parametrize("d,group,paged,thresholds", [(128, 4, True, "both"), (128, 8, True, "tau"),
                                                      (64, 2, False, "none"), (128, 16, True, "both"),
                                                      (64, 1, True, "tau")])
def test_q8_front_equals_split_then_estimate(d, group, paged, thresholds):
    """The fused front writes the same query codes, eta, thresholds and Z, bit
    for bit, as the query split followed by the coarse-logit estimate
    (ragged lengths, an empty request, 16-row groups)."""
    lens = [0, 1, 17, 191, 192, 193, 700, 2049]
    wl = make_custom(batch=len(lens), heads=2 * group, kv_heads=2, dim=d, lens=lens, paged=paged,
                     spike_count=3, n_sink=1, seed=d + group, device="cuda")
    keys = _gpu_q8.encode_cache(wl)
    _, flat = _gpu_q8.level_views(wl, keys)
    req = wl.flat.seq_lens if thresholds != "none" else None
    kappa, kappa_v = -3.5, 1.25
    a = F.q8_empty_query(wl.q)
    b = F.q8_empty_query(wl.q)
    for t in (a.planes, b.planes):
        t.fill_(0x33)
    for t in (a.eta, a.tau, a.tau_v, b.eta, b.tau, b.tau_v):
        t.fill_(float("nan"))
    if thresholds == "tau":
        a.tau_v = b.tau_v = None
    F.fold_q8_split_query(wl.q, wl.sm_scale, a, req_lens=req, kappa=kappa, kappa_v=kappa_v)
    za = torch.empty(wl.batch, wl.num_heads, dtype=torch.float32, device="cuda")
    F.fold_q8_ref_estimate(flat, keys, a, za)
    zb = torch.full_like(za, float("nan"))
    F.fold_q8_front(flat, keys, wl.q, wl.sm_scale, b, zb, req_lens=req, kappa=kappa,
                    kappa_v=kappa_v)
    torch.cuda.synchronize()
    assert torch.equal(a.planes, b.planes)
    assert torch.equal(a.eta, b.eta)
    assert torch.equal(za, zb)
    if req is not None:
        assert torch.equal(a.tau, b.tau)
        if a.tau_v is not None:
            assert torch.equal(a.tau_v, b.tau_v)


def test_q8_front_rejects_bad_arguments():
    wl = make_config(2, batch=2, seq_len=300, device="cuda")
    keys = _gpu_q8.encode_cache(wl)
    _, flat = _gpu_q8.level_views(wl, keys)
    qq = F.q8_empty_query(wl.q)
    z = torch.empty(wl.batch, wl.num_heads, dtype=torch.float32, device="cuda")
    with pytest.raises(F.FoldError):
        F.fold_q8_front(flat, keys, wl.q, float("nan"), qq, z)
    with pytest.raises(F.FoldError):
        F.fold_q8_front(flat, keys, wl.q, wl.sm_scale, qq, z, kappa=float("nan"))


# ------------------------------------------------------- invariants ---------
@pytest.mark.parametrize("cfg", [2, 4])
@pytest.mark.parametrize("T", [INF, 16.0])
def test_q8_debug_exports_do_not_change_results(T, cfg):
    """Config 2 (GQA, the packed scan) and config 4 shrunk (MHA, the VALU scan
    with one row per read group)."""
    wl = make_config(cfg, batch=4 if cfg == 2 else 3, seq_len=1500 if cfg == 2 else 3000,
                     device="cuda")
    a, keys = _gpu_q8.run(wl, T, debug=False)
    z = a["z"].cuda()
    b, _ = _gpu_q8.run(wl, T, z=z, keys=keys, debug=True)
    assert torch.equal(a["part_A"], b["part_A"]) and torch.equal(a["part_L"], b["part_L"])


def test_q8_repeat_bits():
    wl = make_config(2, batch=3, seq_len=2000, device="cuda")
    a, keys = _gpu_q8.run(wl, 16.0, splits=[4])
    b, _ = _gpu_q8.run(wl, 16.0, splits=[4], keys=keys)
    assert torch.equal(a["out"], b["out"]) and torch.equal(a["part_A"], b["part_A"])


def test_q8_close_to_exact_softmax_at_full_refine():
    """kappa = +inf refines every key: the output is softmax attention over the
    two-plane codes, within 1e-3 of softmax over the BF16 operands here."""
    wl = make_config(2, batch=2, seq_len=3000, device="cuda")
    res, _ = _gpu_q8.run(wl, INF, kappa=INF, splits=[4])
    oi = _adapt.oracle_inputs(wl)
    o_ref, _, _, _ = _adapt.decode(oi, res["z"].double().numpy(), INF, [1])
    err = _gpu.row_errors(res["out"].numpy(), o_ref)
    print(f"  q8 vs BF16 softmax: max row err = {err.max():.3e}")
    assert err.max() < 1e-3


# ------------------------------------------------- full-size, sampled ------
def _sampled(cfg, T, chunks, kappa=0.0):
    wl = make_config(cfg, device="cuda")
    res, keys = _gpu_q8.run(wl, T, kappa=kappa)
    oi = _adapt.oracle_inputs(wl)
    lv = oi["levels"][0]
    bt = lv["block_table"]
    pages = set()
    for r, g in chunks:
        n = lv["seq_lens"][r]
        pages |= {int(p) for p in bt[r, :(n + 15) // 16]}
    planes = _oracle_planes(wl, pages)
    ga, gb, ge = _gpu_planes(keys)
    idx = np.array(sorted(pages))
    assert np.array_equal(ga[idx], planes[0][idx]) and np.array_equal(gb[idx], planes[1][idx])
    assert np.array_equal(ge[idx], planes[2][idx])
    qa, qb, eta, tau = _query_codes(wl, kappa)
    _check_query_codes(res, qa, qb, eta, tau)
    G = wl.group
    rows = [(r, g * G + hh) for r, g in chunks for hh in range(G)]
    zo = q8.estimate_level_q8(qa, qb, eta, planes, num_kv_heads=wl.num_kv_heads,
                              page_size=wl.page_size, seq_lens=oi["flat"]["seq_lens"],
                              block_table=oi["flat"]["block_table"], rows=rows)
    z64 = res["z"].double().numpy()
    assert max(abs(z64[r, h] - zo[r, h]) for r, h in rows) <= 1e-3
    pa, pl = q8.decode_level_q8(qa, qb, eta, planes, oi["v_bits"], num_kv_heads=wl.num_kv_heads,
                                page_size=wl.page_size, z=z64, T=T, tau=tau,
                                num_splits=res["splits"][0], chunks=chunks, **lv)
    o_ref, _ = combine(pa, pl)
    ri = np.array([r for r, _ in rows])
    hi = np.array([h for _, h in rows])
    err = _gpu.row_errors(res["out"].numpy()[ri, hi], o_ref[ri, hi])
    print(f"  q8 {wl.name} T={T}: sampled rows {len(rows)}, max row err = {err.max():.3e}")
    assert (err <= TOL).all()
    gl = res["part_L"].double().numpy()[:, ri, hi]
    assert np.allclose(gl, pl[:, ri, hi], rtol=2e-5, atol=0)


@pytest.mark.parametrize("T", [INF, 16.0])
def test_q8_config2_full_size_sampled(T):
    _sampled(2, T, chunks=[(0, 0), (5, 3), (15, 7)])


@pytest.mark.parametrize("T", [INF, 12.0])
def test_q8_config3_full_size_sampled(T):
    _sampled(3, T, chunks=[(0, 0), (7, 7)])


@pytest.mark.parametrize("T", [INF, 16.0])
def test_q8_config4_full_size_sampled(T):
    _sampled(4, T, chunks=[(0, 0), (3, 31)])
