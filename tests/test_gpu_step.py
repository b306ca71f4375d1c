"""The decode step around the scan on the GPU, against the step oracle.

Bars: appended cache rows and gathered draft rows bit-exact; certified
outputs within 1e-2 of the row's inf-norm of exact softmax with the rerun
counts of the reading (out-of-window rows once, non-finite L stepping 64
binades); draft columns within 1e-2 of the oracle's masked fold with the
kernel's references.
"""

import math

import numpy as np
import pytest
import torch

import paper_2609_33410_amd as F
from oracle import bf16_bits_to_f64, gather
from oracle import step_oracle as st
from tests import _adapt, _gpu, _gpu_q8
from workloads import chain_parents, host_bits, make_custom, make_drafts

pytestmark = pytest.mark.gpu
INF = float("inf")
TOL = 1e-2


@pytest.fixture(scope="module", autouse=True)
def _device():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    F.load_library()


# ---------------------------------------------------------------- append ---
@pytest.mark.parametrize("paged", [True, False])
def test_append_kv_matches_oracle(paged):
    wl = make_custom(batch=3, heads=8, kv_heads=2, dim=128, lens=[40, 17, 64], paged=paged,
                     seed=5, device="cuda")
    fl = wl.flat
    bt = fl.block_table.clone() if paged else None
    if paged:
        bt[2, 1] = 10 ** 6                        # writes to this page are skipped
    kv = F.kv_view(wl.k, wl.v, fl.seq_lens, num_kv_heads=2, max_seq_len=fl.max_seq_len,
                   block_table=bt)
    cap = bt.shape[1] * 16 if paged else fl.max_seq_len
    seqs = [0, 1, 2, 2, 0, 7, -1, 1]
    poss = [39, 3, 20, 63, cap, 0, 3, -2]         # the last four are skipped
    g = torch.Generator(device="cpu").manual_seed(3)
    ks = torch.randn(len(seqs), 2, 128, generator=g).to(torch.bfloat16).cuda()
    vs = torch.randn(len(seqs), 2, 128, generator=g).to(torch.bfloat16).cuda()
    kc, vc = wl.k.clone(), wl.v.clone()
    F.fold_append_kv(kv, ks, vs, torch.tensor(seqs, dtype=torch.int32).cuda(),
                     torch.tensor(poss, dtype=torch.int32).cuda(), kc, vc)
    torch.cuda.synchronize()
    btn = None if bt is None else bt.cpu().numpy()
    for src, cache, got in ((ks, wl.k, kc), (vs, wl.v, vc)):
        want = st.append_tokens(host_bits(cache), host_bits(src), seqs, poss, btn,
                                16 if paged else 0)
        assert np.array_equal(host_bits(got), want)
    # one side only
    kc2 = wl.k.clone()
    F.fold_append_kv(kv, ks, None, torch.tensor(seqs, dtype=torch.int32).cuda(),
                     torch.tensor(poss, dtype=torch.int32).cuda(), kc2, None)
    torch.cuda.synchronize()
    assert torch.equal(kc2, kc)


# ------------------------------------------------------------- certificate -
def _exact(wl, oi):
    """FP64 base-2 log-sum-exp and softmax output of every row."""
    b, h = wl.q.shape[:2]
    G = wl.group
    lse = np.zeros((b, h))
    out = np.zeros((b, h, wl.head_dim))
    for r, n in enumerate(oi["flat"]["seq_lens"]):
        for g in range(wl.num_kv_heads):
            keys = gather(oi["k_bits"], r, g, n, oi["flat"]["block_table"], wl.page_size)
            vals = gather(oi["v_bits"], r, g, n, oi["flat"]["block_table"], wl.page_size)
            for hh in range(g * G, (g + 1) * G):
                s = (keys @ bf16_bits_to_f64(oi["q_bits"][r, hh])) * wl.sm_scale
                m = s.max()
                w = np.exp(s - m)
                lse[r, hh] = (m + math.log(w.sum())) / math.log(2.0)
                out[r, hh] = (w @ vals) / w.sum()
    return lse, out


@pytest.mark.parametrize("T", [INF, 16.0])
def test_certified_decode_recovers_bad_references(T):
    """Rows with references far from the truth: inside the window untouched;
    outside but with a finite L, one rerun; L = 0 (delta = 300: 300, 236,
    172 give L = 0, 108 a finite L, then l) four reruns; L = inf (delta =
    -200: -200, -136 overflow, -72 inside the window) two reruns.  Final
    outputs equal the oracle's decode with the final references (and exact
    softmax at T = inf)."""
    wl = make_custom(batch=2, heads=8, kv_heads=2, dim=128, lens=[700, 333], spike_count=4,
                     n_sink=1, seed=12, device="cuda")
    oi = _adapt.oracle_inputs(wl)
    lse, o_exact = _exact(wl, oi)
    deltas = np.array([[0.0, 0.6, 2.5, -60.0, 300.0, -200.0, -110.0, 30.0],
                       [-0.4, 1.8, 40.0, 300.0, -200.0, 0.2, -3.0, 8.0]])
    z0 = torch.tensor(lse + deltas, dtype=torch.float32, device="cuda")
    levels, _ = _gpu.kv_views(wl)
    out, zf, reruns, cert = F.fold_certified_decode(levels, wl.q, z0, T, [2], wl.sm_scale)
    torch.cuda.synchronize()
    want = np.where((deltas >= -100.0) & (deltas <= 1.0), 0, 1)
    want[deltas == 300.0] = 4
    want[deltas == -200.0] = 2
    got = reruns.cpu().numpy()
    print(f"  certificate T={T}: reruns {got.tolist()}")
    assert np.array_equal(got, want)
    assert not cert.cpu().numpy().any()
    zf = zf.cpu().double().numpy()
    # the final outputs against the oracle's decode with the final references
    o_ref, _, _, _ = _adapt.decode(oi, zf, T, [1])
    err = _gpu.row_errors(out.cpu().numpy(), o_ref)
    print(f"  certificate T={T}: max row err = {err.max():.3e}")
    assert (err <= TOL).all()
    if math.isinf(T):
        assert (_gpu.row_errors(out.cpu().numpy(), o_exact) <= TOL).all()
    assert np.array_equal(zf[want == 0], z0.cpu().double().numpy()[want == 0])
    one = want == 1
    assert np.abs(zf[one] - lse[one]).max() < 1e-3


def test_certified_decode_leaves_good_rows_bitwise():
    """Rows inside the window are never decoded differently: the certified
    output equals a plain decode's bit for bit where no row is flagged."""
    wl = make_custom(batch=2, heads=4, kv_heads=1, dim=64, lens=[500, 90], seed=2, device="cuda")
    z = _gpu.estimate(wl)
    levels, _ = _gpu.kv_views(wl)
    out, _, _, _, _ = F.fold_decode(levels, wl.q, z, 16.0, [2], wl.sm_scale)
    out2, z2, reruns, cert = F.fold_certified_decode(levels, wl.q, z, 16.0, [2], wl.sm_scale)
    torch.cuda.synchronize()
    if not reruns.any():
        assert torch.equal(out, out2) and torch.equal(z, z2)


# ------------------------------------------------------------------ drafts -
def _run_drafts(dw, T, splits=2, bf16=True):
    wl = dw.wl
    fl = wl.flat
    dv = F.fold_draft_views(wl.k, wl.v, fl.block_table, fl.seq_lens_host,
                            dw.col_indptr.cpu().tolist(), dw.parent.cpu().tolist(),
                            dw.spare_pages, num_kv_heads=wl.num_kv_heads)
    z = torch.empty(dw.num_cols, wl.num_heads, dtype=torch.float32, device="cuda")
    F.fold_ref_estimate(dv.estimate, F.q_view(dw.q), wl.sm_scale, z)
    out, pa, pl, _, _ = F.fold_decode([dv.committed, dv.ancestors], dw.q, z, T, [splits, 1],
                                      wl.sm_scale)
    torch.cuda.synchronize()
    return dv, z, out


def _oracle_drafts(dw, z, T):
    wl = dw.wl
    fl = wl.flat
    a, l = st.decode_drafts(host_bits(dw.q), host_bits(wl.k), host_bits(wl.v),
                            num_kv_heads=wl.num_kv_heads, page_size=wl.page_size,
                            sm_scale=wl.sm_scale, seq_lens=fl.seq_lens_host,
                            block_table=fl.block_table.cpu().numpy(),
                            col_indptr=dw.col_indptr.cpu().tolist(),
                            parent=dw.parent.cpu().tolist(), z=z, T=T)
    with np.errstate(invalid="ignore"):
        return a / l[..., None]


def _check_gathered_rows(dw):
    """Spare pages hold each column's ancestor rows, bit for bit."""
    wl = dw.wl
    kb, vb = host_bits(wl.k), host_bits(wl.v)
    bt = wl.flat.block_table.cpu().numpy()
    sp = dw.spare_pages.cpu().numpy()
    ind = dw.col_indptr.cpu().tolist()
    par = dw.parent.cpu().tolist()
    for r, n in enumerate(wl.flat.seq_lens_host):
        m = ind[r + 1] - ind[r]
        for c in range(m):
            vis = st.draft_visible(n, m, par[ind[r]:ind[r + 1]], c)
            for i, pos in enumerate(vis[vis >= n - m]):
                src = (bt[r, pos // 16], pos % 16)
                dst = (sp[ind[r] + c, i // 16], i % 16)
                for arr in (kb, vb):
                    assert np.array_equal(arr[dst[0], :, dst[1]], arr[src[0], :, src[1]])


@pytest.mark.parametrize("shape", ["chain2", "chain4", "tree8", "wide"])
@pytest.mark.parametrize("T", [INF, 16.0])
def test_draft_columns_match_masked_oracle(shape, T):
    if shape == "chain2":
        parents, heads, kvh, d = [chain_parents(2)] * 3, 8, 2, 128
    elif shape == "chain4":
        parents, heads, kvh, d = [chain_parents(4), chain_parents(4), []], 8, 2, 64
    elif shape == "tree8":
        parents, heads, kvh, d = [[-1, 0, 0, 1, 1, 2, 2, 3], chain_parents(3)], 8, 2, 128
    else:  # 8 columns x G = 8: 64 stacked rows on the committed level
        parents, heads, kvh, d = [[-1, 0, 0, 1, 2, 3, 3, -1]], 8, 1, 128
    committed = [700, 333, 90][:len(parents)]
    dw = make_drafts(committed=committed, parents=parents, heads=heads, kv_heads=kvh, dim=d,
                     spike_count=3, n_sink=1, seed=len(shape), device="cuda")
    dv, z, out = _run_drafts(dw, T)
    _check_gathered_rows(dw)
    o_ref = _oracle_drafts(dw, z.cpu().double().numpy(), T)
    err = _gpu.row_errors(out.cpu().numpy(), o_ref)
    print(f"  drafts {shape} T={T}: columns {dw.num_cols}, max row err = {err.max():.3e}")
    assert (err <= TOL).all()


def test_drafts_equal_per_column_plain_decodes_for_chains():
    """A chain's column c is a plain decode of its request truncated at
    n0 + c + 1 keys: the two-level draft decode agrees with it at T = inf."""
    dw = make_drafts(committed=[400], parents=[chain_parents(4)], heads=8, kv_heads=2, dim=128,
                     spike_count=2, seed=3, device="cuda")
    dv, z, out = _run_drafts(dw, INF)
    wl = dw.wl
    for c in range(4):
        n = 400 + c + 1
        sl = torch.tensor([n], dtype=torch.int32, device="cuda")
        kv = F.kv_view(wl.k, wl.v, sl, num_kv_heads=2, max_seq_len=n,
                       block_table=wl.flat.block_table)
        o1, _, _, _, _ = F.fold_decode([kv], dw.q[c:c + 1].contiguous(), z[c:c + 1].contiguous(),
                                       INF, [1], wl.sm_scale)
        torch.cuda.synchronize()
        err = _gpu.row_errors(out[c:c + 1].cpu().numpy(), o1.cpu().double().numpy())
        assert err.max() < 1e-5


def test_q8_draft_columns_close_to_exact():
    """Two-plane keys: the same layout over the key planes, scale and BF16
    values; with every key refined the columns are within 2e-3 of the
    masked softmax over BF16 operands."""
    dw = make_drafts(committed=[600, 200], parents=[chain_parents(3), [-1, 0, 0, 1]], heads=8,
                     kv_heads=2, dim=128, spike_count=3, seed=9, device="cuda")
    wl = dw.wl
    keys = _gpu_q8.encode_cache(wl)
    fl = wl.flat
    d = wl.head_dim
    dv = F.fold_draft_views(None, wl.v, fl.block_table, fl.seq_lens_host,
                            dw.col_indptr.cpu().tolist(), dw.parent.cpu().tolist(),
                            dw.spare_pages, num_kv_heads=2, layout=keys.plane_a,
                            extra=[(keys.plane_a, d), (keys.plane_b, d), (keys.scale, 2)])
    qq = F.q8_empty_query(dw.q)
    col_req = dv.keep[1].cpu().tolist()          # each column's request
    req_lens = torch.tensor([fl.seq_lens_host[r] for r in col_req], dtype=torch.int32,
                            device="cuda")
    F.fold_q8_split_query(dw.q, wl.sm_scale, qq, req_lens=req_lens, kappa=INF)
    z = torch.empty(dw.num_cols, wl.num_heads, dtype=torch.float32, device="cuda")
    F.fold_q8_ref_estimate(dv.estimate, keys, qq, z)
    b, h = z.shape
    pa = torch.empty(3, b, h, d, device="cuda")
    pl = torch.empty(3, b, h, device="cuda")
    F.fold_q8_decode_split(dv.committed, keys, qq, z, INF, 2, 0, pa, pl)
    F.fold_q8_decode_split(dv.ancestors, keys, qq, z, INF, 1, 2, pa, pl)
    out = torch.empty(b, h, d, device="cuda")
    F.fold_combine(pa, pl, out)
    torch.cuda.synchronize()
    o_ref = _oracle_drafts(dw, z.cpu().double().numpy(), INF)
    err = _gpu.row_errors(out.cpu().numpy(), o_ref)
    print(f"  q8 drafts: max row err vs BF16 masked softmax = {err.max():.3e}")
    assert err.max() < 2e-3
