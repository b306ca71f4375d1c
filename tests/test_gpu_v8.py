"""Parity of 8-bit values (two E4M3 planes) on the GPU with the FP64 oracle.

Bars: value-plane codes bit-exact; outputs within 1e-2 of the row's inf-norm
with the kernel's FP32 decisions imposed (and within the stated flip bound in
the oracle's own decisions); second-value-plane read bits bit-exact against
the oracle's group rule on the exported coarse scores.
"""

import math

import numpy as np
import pytest
import torch

import paper_2609_33410_amd as F
from oracle import bf16_bits_to_f64, combine
from oracle import q8_oracle as q8
from tests import _adapt, _gpu, _gpu_q8
from workloads import host_bits, make_cascade, make_config, make_custom

pytestmark = pytest.mark.gpu
INF = float("inf")
TOL = 1e-2


@pytest.fixture(scope="module", autouse=True)
def _device():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    F.load_library()


def _planes_of(vals):
    return vals.plane_p.cpu().numpy(), vals.plane_r.cpu().numpy()


def test_value_writer_codes():
    """Whole cache through the writer: the oracle's E4M3 codes bit for bit, at
    the cache's own scale and at a scale that saturates part of it."""
    wl = make_config(2, batch=2, seq_len=700, device="cuda")
    for e in (None, -9):
        vals = _gpu_q8.encode_values(wl, e)
        torch.cuda.synchronize()
        gp, gr = _planes_of(vals)
        p, r = q8.split_values(host_bits(wl.v), vals.scale_exp)
        assert np.array_equal(gp, p) and np.array_equal(gr, r)
        if e == -9:  # 448 * 2^-9 = 0.875
            assert ((gp & 0x7F) == 0x7E).any()   # saturated codes present


def test_paged_value_writer_appends_and_skips():
    """The value writer through a paged view: every valid (sequence, position)
    gets the oracle's codes at its page slot; tokens past capacity, of an
    unknown sequence or on an invalid page id leave the planes untouched."""
    wl = make_custom(batch=3, heads=8, kv_heads=2, dim=128, lens=[40, 17, 64], seed=5,
                     device="cuda")
    fl = wl.flat
    bt = fl.block_table.clone()
    bt[2, 1] = 10 ** 6
    kv = F.kv_view(wl.k, wl.v, fl.seq_lens, num_kv_heads=2, max_seq_len=fl.max_seq_len,
                   block_table=bt)
    vals = F.v8_empty_values(wl.v, -4)
    vals.plane_p.fill_(0x33)
    vals.plane_r.fill_(0x33)
    seqs, poss = [], []
    for r, n in enumerate(fl.seq_lens_host):
        seqs += [r] * n
        poss += list(range(n))
    seqs += [0, 7, -1, 1]
    poss += [fl.block_table.shape[1] * 16, 0, 3, -2]
    n_tok = len(seqs)
    g = torch.Generator(device="cpu").manual_seed(2)
    v_src = (4 * torch.randn(n_tok, 2, 128, generator=g)).to(torch.bfloat16)
    logical = torch.zeros(3, 2, 64, 128, dtype=torch.bfloat16)
    for t in range(n_tok - 4):
        logical[seqs[t], :, poss[t]] = v_src[t]
    F.fold_v8_write_values(kv, v_src.cuda(), torch.tensor(seqs, dtype=torch.int32).cuda(),
                           torch.tensor(poss, dtype=torch.int32).cuda(), vals)
    torch.cuda.synchronize()
    gp, gr = _planes_of(vals)
    table = bt.cpu().numpy()
    written = np.zeros(gp.shape[:3], dtype=bool)
    for r, n in enumerate(fl.seq_lens_host):
        p, q = q8.split_values(host_bits(logical[r, :, :n]), -4)
        for j in range(n):
            page = int(table[r, j // 16])
            if page >= gp.shape[0]:
                continue
            written[page, :, j % 16] = True
            assert np.array_equal(gp[page, :, j % 16], p[:, j])
            assert np.array_equal(gr[page, :, j % 16], q[:, j])
    assert (gp[~written] == 0x33).all() and (gr[~written] == 0x33).all()


def _imposed_v8(wl, oi, res, vals, T, keys_planes):
    qa, qb, eta = q8.split_queries(host_bits(wl.q), wl.sm_scale)
    tau = res["tau"].numpy()
    tau_v = res["tau_v"].numpy()
    z64 = res["z"].double().numpy()
    p, r = q8.split_values(host_bits(wl.v), vals.scale_exp)
    pa_all, pl_all = [], []
    for li, lv in enumerate(oi["levels"]):
        d = res["dbg"][li]
        pa, pl = q8.decode_level_q8(qa, qb, eta, keys_planes, oi["v_bits"],
                                    num_kv_heads=wl.num_kv_heads, page_size=wl.page_size,
                                    z=z64, T=T, tau=tau, num_splits=res["splits"][li],
                                    imposed=(d["xc_out"].numpy(), d["x_out"].numpy()),
                                    values8=(p, r, vals.scale_exp), tau_v=tau_v, **lv)
        pa_all.append(pa), pl_all.append(pl)
    return combine(np.concatenate(pa_all), np.concatenate(pl_all))


def _refine_v_bits_check(wl, oi, res):
    G = wl.group
    tau_v = res["tau_v"].numpy()
    for li, lv in enumerate(oi["levels"]):
        d = res["dbg"][li]
        xc = d["xc_out"].numpy()
        R = d["R"]
        for seq, n in enumerate(lv["seq_lens"]):
            reqs = [seq] if lv["row_indptr"] is None else \
                [int(x) for x in lv["row_req"][lv["row_indptr"][seq]:lv["row_indptr"][seq + 1]]]
            for g in range(wl.num_kv_heads):
                rows = [(rr, g * G + hh) for rr in reqs for hh in range(G)]
                for u in range((len(rows) + R - 1) // R):
                    grp = rows[u * R:(u + 1) * R]
                    xs = np.stack([xc[rr, hh, :n] for rr, hh in grp])
                    blocks = np.array([k // G for k in range(len(grp))])
                    T = res["T"]
                    _, rv = q8.gate_bits(xs, blocks, T, tau_v[[rr for rr, _ in grp]], f32=True)
                    want = rv.any(axis=0) if len(grp) else np.zeros(n, bool)
                    got = d["refine_v_gate_out"][seq, g, u, :n].numpy().astype(bool)
                    assert np.array_equal(got, want), f"refine-V bits: level {li} seq {seq} g {g}"


def _v8_parity(wl, T, kappa_v=0.0, splits=None):
    oi = _adapt.oracle_inputs(wl)
    vals = _gpu_q8.encode_values(wl)
    res, keys = _gpu_q8.run(wl, T, splits=splits, debug=True, values=vals, kappa_v=kappa_v)
    res["T"] = T
    keys_planes = (keys.plane_a.cpu().numpy(), keys.plane_b.cpu().numpy(),
                   keys.scale.cpu().numpy().view(np.uint16))
    want_planes = q8.split_keys(host_bits(wl.k))
    assert all(np.array_equal(a, b) for a, b in zip(keys_planes, want_planes))
    o_ref, l_ref = _imposed_v8(wl, oi, res, vals, T, want_planes)
    ok = l_ref > 0
    err = _gpu.row_errors(res["out"].numpy(), o_ref)
    print(f"  v8 {wl.name} T={T} kappa_v={kappa_v}: max row err (imposed) = "
          f"{err[ok].max() if ok.any() else 0:.3e}")
    assert (err[ok] <= TOL).all()
    _refine_v_bits_check(wl, oi, res)
    return res, keys, vals


@pytest.mark.parametrize("kappa_v", [0.0, -INF, INF, 4.0])
@pytest.mark.parametrize("T", [INF, 16.0, 5.0])
def test_v8_config2_shape_small(T, kappa_v):
    wl = make_config(2, batch=2, seq_len=1000, device="cuda")
    _v8_parity(wl, T, kappa_v, splits=[3])


@pytest.mark.parametrize("d", [64, 128])
@pytest.mark.parametrize("group", [1, 8])
def test_v8_ragged(d, group):
    lens = [0, 1, 17, 64, 65, 333]
    wl = make_custom(batch=len(lens), heads=2 * group, kv_heads=2, dim=d, lens=lens,
                     spike_count=2, n_sink=1, seed=d + group, device="cuda")
    for T in (INF, 6.0):
        _v8_parity(wl, T, splits=[2])


@pytest.mark.parametrize("splits", [1, 4])
def test_v8_mha_ragged_longest_first(splits):
    """MHA with 8-bit values (the VALU two-plane scan) over ragged lengths."""
    wl = make_custom(batch=5, heads=4, kv_heads=4, dim=128, lens=[2100, 1100, 2053, 0, 77],
                     spike_count=6, n_sink=1, seed=40 + splits, device="cuda")
    for T, kv in ((INF, 0.0), (16.0, -4.0), (5.0, 4.0)):
        _v8_parity(wl, T, kappa_v=kv, splits=[splits])


def test_v8_cascade_groups_keep_their_own_values():
    """Stacked rows of three requests share read groups: each row's second
    value plane counts only where its own GQA group set refine-V."""
    wl = make_cascade(requests=5, heads=8, kv_heads=1, dim=128, prefix_len=496, suffix_len=48,
                      splits=(2, 1), seed=11, device="cuda")
    for T in (INF, 8.0):
        _v8_parity(wl, T, kappa_v=-4.0)


def test_v8_full_refine_equals_bf16_values():
    """kappa_v = +inf reads every live key's second plane; the planes are
    lossless here, so the output equals the two-plane-key path over BF16
    values up to FP32 summation order."""
    wl = make_config(2, batch=2, seq_len=2000, device="cuda")
    vals = _gpu_q8.encode_values(wl)
    a, keys = _gpu_q8.run(wl, 16.0, splits=[4], kappa_v=INF, values=vals)
    b, _ = _gpu_q8.run(wl, 16.0, splits=[4], kappa_v=INF, keys=keys, z=a["z"].cuda())
    err = _gpu.row_errors(a["out"].numpy(), b["out"].double().numpy())
    print(f"  v8 vs BF16 values: max row err = {err.max():.2e}")
    # exact for |v 2^-e| >= 2^-6; below, the residual plane keeps 2^-13 2^e
    assert err.max() < 1e-4


@pytest.mark.parametrize("cfg", [2, 4])
def test_v8_debug_exports_do_not_change_results(cfg):
    wl = make_config(cfg, batch=3, seq_len=1500 if cfg == 2 else 3000, device="cuda")
    vals = _gpu_q8.encode_values(wl)
    a, keys = _gpu_q8.run(wl, 16.0, values=vals)
    b, _ = _gpu_q8.run(wl, 16.0, values=vals, keys=keys, z=a["z"].cuda(), debug=True)
    assert torch.equal(a["part_A"], b["part_A"]) and torch.equal(a["part_L"], b["part_L"])


def _on_pages(fn, t, pages, outs):
    """fn over the stored rows of the listed pages only; other entries zero."""
    idx = torch.as_tensor(sorted(pages), dtype=torch.long, device=t.device)
    sub = fn(host_bits(t.index_select(0, idx)))
    full = []
    for arr, (shape, dtype) in zip(sub, outs):
        z = np.zeros(shape, dtype=dtype)
        z[idx.cpu().numpy()] = arr
        full.append(z)
    return full


def _on_chunk_pages(fn, t, chunks, bt, seq_lens, outs):
    """fn over the stored rows of each chunk's pages at the chunk's kv head
    only (the rows its scan reads); other entries zero."""
    full = [np.zeros(shape, dtype=dtype) for shape, dtype in outs]
    for seq, g in chunks:
        pg = sorted({int(x) for x in bt[seq, :(seq_lens[seq] + 15) // 16]})
        idx = torch.as_tensor(pg, dtype=torch.long, device=t.device)
        sub = fn(host_bits(t.index_select(0, idx)[:, g:g + 1].contiguous()))
        for dst, arr in zip(full, sub):
            dst[np.array(pg), g:g + 1] = arr
    return full


@pytest.mark.parametrize("cfg,chunks", [(2, [(0, 0), (5, 3), (15, 7)]),
                                        (3, [(0, 0), (7, 7)]),
                                        (4, [(0, 5), (2, 30)])])
@pytest.mark.parametrize("T", [INF, 16.0])
def test_v8_full_size_sampled(cfg, chunks, T):
    """Full-size workloads 2 (16 x 8192 keys, GQA), 3 (8 x 32768, 16 splits)
    and 4 (MHA, 64K-128K ragged, 32 splits): sampled (request, kv head)
    chunks against the oracle's own FP64 decisions, within the row bar; the
    sampled chunks' key and value codes bit-exact."""
    wl = make_config(cfg, device="cuda")
    vals = _gpu_q8.encode_values(wl)
    res, keys = _gpu_q8.run(wl, T, values=vals)
    oi = _adapt.oracle_inputs(wl)
    lv = oi["levels"][0]
    bt = lv["block_table"]
    shp = tuple(wl.k.shape)
    planes = _on_chunk_pages(q8.split_keys, wl.k, chunks, bt, lv["seq_lens"],
                             [(shp, np.int8), (shp, np.int8), (shp[:-1], np.uint16)])
    p, r = _on_chunk_pages(lambda b: q8.split_values(b, vals.scale_exp), wl.v, chunks, bt,
                           lv["seq_lens"], [(shp, np.uint8), (shp, np.uint8)])
    gp, gr = _planes_of(vals)
    ga = keys.plane_a.cpu().numpy()
    for seq, g in chunks:
        idx = np.array(sorted({int(x) for x in bt[seq, :(lv["seq_lens"][seq] + 15) // 16]}))
        assert np.array_equal(gp[idx, g], p[idx, g]) and np.array_equal(gr[idx, g], r[idx, g])
        assert np.array_equal(ga[idx, g], planes[0][idx, g])
    qa, qb, eta = q8.split_queries(host_bits(wl.q), wl.sm_scale)
    tau = np.array([q8.refine_tau(n, 0.0) for n in wl.flat.seq_lens_host], dtype=np.float32)
    assert np.array_equal(res["tau_v"].numpy(), tau)
    G = wl.group
    rows = [(rq, g * G + hh) for rq, g in chunks for hh in range(G)]
    pa, pl = q8.decode_level_q8(qa, qb, eta, planes, oi["v_bits"], num_kv_heads=wl.num_kv_heads,
                                page_size=wl.page_size, z=res["z"].double().numpy(), T=T,
                                tau=tau, num_splits=res["splits"][0], chunks=chunks,
                                values8=(p, r, vals.scale_exp), tau_v=tau, **lv)
    o_ref, _ = combine(pa, pl)
    ri = np.array([rr for rr, _ in rows])
    hi = np.array([hh for _, hh in rows])
    err = _gpu.row_errors(res["out"].numpy()[ri, hi], o_ref[ri, hi])
    print(f"  v8 {wl.name} T={T}: sampled rows {len(rows)}, max row err = {err.max():.3e}")
    assert (err <= TOL).all()
