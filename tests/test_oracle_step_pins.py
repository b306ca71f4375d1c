"""Pins of the step oracle (append, certified decode, draft columns) against
what the paper and the mathematics fix: the generator's logical cache,
torch SDPA with an explicit boolean mask, truncated plain decodes, and
hand-computed rerun sequences."""

import math

import numpy as np
import pytest
import torch

from oracle import bf16_bits_to_f64, combine, decode_level, gather, scores
from oracle import step_oracle as st
from tests import _adapt
from workloads import chain_parents, host_bits, make_custom, make_drafts

INF = float("inf")


# ---------------------------------------------------------------- append ---
def test_append_round_trip_through_logical_cache():
    """Zero each request's last token in the pages, append it back from the
    logical cache: the pages are restored bit for bit; invalid tokens (bad
    sequence, position past the table, negative position, page id out of
    range) change nothing."""
    wl = make_custom(batch=3, heads=4, kv_heads=2, dim=64, lens=[40, 17, 64], seed=3)
    bt = wl.flat.block_table.numpy()
    kb = host_bits(wl.k)
    lens = wl.flat.seq_lens_host
    damaged = kb.copy()
    for r, n in enumerate(lens):
        damaged[bt[r, (n - 1) // 16], :, (n - 1) % 16] = 0
    src = np.stack([host_bits(wl.logical_k[r, :, n - 1]) for r, n in enumerate(lens)])
    back = st.append_tokens(damaged, src, list(range(3)), [n - 1 for n in lens], bt, 16)
    assert np.array_equal(back, kb)
    bt_bad = bt.copy()
    bt_bad[2, 0] = 10 ** 6
    junk = np.full((4, 2, 64), 0x3F80, dtype=np.uint16)
    same = st.append_tokens(kb, junk, [7, 0, 1, 2], [0, bt.shape[1] * 16, -1, 3], bt_bad, 16)
    assert np.array_equal(same, kb)


def test_append_contiguous_cache():
    wl = make_custom(batch=2, heads=2, kv_heads=1, dim=64, lens=[5, 9], paged=False, seed=1)
    kb = host_bits(wl.k)
    src = np.full((3, 1, 64), 0x4000, dtype=np.uint16)
    out = st.append_tokens(kb, src, [0, 1, 1], [4, 8, 9], None, 0)   # position 9: past the view
    assert (out[0, :, 4] == 0x4000).all() and (out[1, :, 8] == 0x4000).all()
    out[0, :, 4] = kb[0, :, 4]
    out[1, :, 8] = kb[1, :, 8]
    assert np.array_equal(out, kb)


# ------------------------------------------------------------- certificate -
def _exact_lse2(wl, oi):
    """Base-2 log-sum-exp of every row over all its keys (torch logsumexp)."""
    b, h = wl.q.shape[:2]
    G = wl.group
    out = np.zeros((b, h))
    for r, n in enumerate(oi["flat"]["seq_lens"]):
        for g in range(wl.num_kv_heads):
            keys = gather(oi["k_bits"], r, g, n, oi["flat"]["block_table"], wl.page_size)
            for hh in range(g * G, (g + 1) * G):
                q = bf16_bits_to_f64(oi["q_bits"][r, hh])
                s = torch.from_numpy(keys @ q) * wl.sm_scale
                out[r, hh] = float(torch.logsumexp(s, 0)) / math.log(2.0)
    return out


def _sdpa(wl):
    q = wl.q.double().unsqueeze(2)                      # [B, H, 1, D]
    k = wl.logical_k.double().repeat_interleave(wl.group, dim=1)
    v = wl.logical_v.double().repeat_interleave(wl.group, dim=1)
    n = wl.flat.seq_lens_host
    outs = []
    for r in range(wl.batch):
        outs.append(torch.nn.functional.scaled_dot_product_attention(
            q[r:r + 1], k[r:r + 1, :, :n[r]], v[r:r + 1, :, :n[r]], scale=wl.sm_scale)[0, :, 0])
    return torch.stack(outs).numpy()


def test_certified_decode_reruns_out_of_window_rows_once():
    """Rows whose first L = 2^-delta lies outside [2^-1, 2^100] are decoded
    once more with Z = l (then L = 1); rows inside are untouched.  Final
    outputs equal torch SDPA in FP64."""
    wl = make_custom(batch=2, heads=8, kv_heads=2, dim=64, lens=[300, 77], spike_count=3,
                     n_sink=1, seed=9)
    oi = _adapt.oracle_inputs(wl)
    lse = _exact_lse2(wl, oi)
    deltas = np.array([0.0, 0.9, 1.5, -50.0, -101.0, 300.0, -0.5, 2.0] * 2).reshape(2, 8)
    z0 = lse + deltas

    def dec(z):
        o, l, _, _ = _adapt.decode(oi, z, INF, [1])
        return o, l

    o, zf, reruns, cert = st.certified_decode(dec, z0)
    want = np.where((2.0 ** -deltas >= 0.5) & (2.0 ** -deltas <= 2.0 ** 100), 0, 1)
    assert np.array_equal(reruns, want)
    assert not cert.any()
    np.testing.assert_allclose(zf[want == 1], lse[want == 1], atol=1e-9)
    assert np.array_equal(zf[want == 0], z0[want == 0])
    np.testing.assert_allclose(o, _sdpa(wl), rtol=0, atol=1e-12)


def test_certified_decode_steps_when_lse_is_not_finite():
    """A decode whose L is formed in FP32 underflows to 0 or overflows to
    infinity: Z moves 64 binades towards the truth per rerun, then takes l.
    delta = 300: 300 -> 236 -> 172 -> 108 (L = 2^-108 > 0, l finite) -> 0:
    four reruns.  delta = -200: L = 2^200 = inf -> -136 (inf) -> -72:
    L = 2^72 is inside the window, two reruns, final Z = l - 72."""
    lse = np.array([[3.0, -7.0, 11.0]])
    z0 = lse + np.array([[300.0, -200.0, 0.25]])
    o_true = np.array([[[1.0, 2.0], [3.0, 4.0], [5.0, 6.0]]])

    def dec(z):
        with np.errstate(over="ignore", under="ignore"):
            l = np.exp2((lse - z).astype(np.float32)).astype(np.float64)
        return o_true.copy(), l

    o, zf, reruns, cert = st.certified_decode(dec, z0)
    assert reruns.tolist() == [[4, 2, 0]]
    assert not cert.any()
    assert zf[0, 0] == lse[0, 0] and zf[0, 1] == lse[0, 1] - 72.0 and zf[0, 2] == z0[0, 2]


def test_certified_decode_gives_up_after_max_reruns():
    def dec(z):
        return np.full((1, 2), np.nan), np.ones(1)

    _, _, reruns, cert = st.certified_decode(dec, np.zeros(1), max_reruns=3)
    assert reruns.tolist() == [3] and cert.tolist() == [4]


def test_certify_bits_match_the_window():
    z = np.zeros(5)
    l = np.array([0.5, 0.4999, 2.0 ** 100, 2.0 ** 100 * 1.0001, 1.0])
    o = np.ones((5, 3))
    o[4, 1] = np.inf
    _, cert, nxt = st.certify(z, l, o)
    assert cert.tolist() == [0, 1, 0, 2, 4]
    assert nxt[0] == 0 and nxt[2] == 0 and nxt[4] == 0.0
    assert nxt[1] == pytest.approx(math.log2(0.4999))


# ------------------------------------------------------------------ drafts -
def _mask_sdpa(dw):
    """torch SDPA (FP64) of every draft column with an explicit boolean mask
    over its request's keys."""
    wl = dw.wl
    out = np.zeros(tuple(dw.q.shape))
    par = dw.parent.tolist()
    ind = dw.col_indptr.tolist()
    for r, n in enumerate(wl.flat.seq_lens_host):
        c0, c1 = ind[r], ind[r + 1]
        m = c1 - c0
        k = wl.logical_k[r, :, :n].double().repeat_interleave(wl.group, dim=0)[None]
        v = wl.logical_v[r, :, :n].double().repeat_interleave(wl.group, dim=0)[None]
        for c in range(m):
            mask = torch.zeros(n, dtype=torch.bool)
            mask[:n - m] = True
            t = c
            while t >= 0:               # walk to the root, marking the path
                mask[n - m + t] = True
                t = par[c0 + t]
            q = dw.q[c0 + c].double()[None, :, None]
            o = torch.nn.functional.scaled_dot_product_attention(
                q, k, v, attn_mask=mask[None, None, None], scale=wl.sm_scale)
            out[c0 + c] = o[0, :, 0].numpy()
    return out


def _draft_oracle(dw, z, T):
    wl = dw.wl
    fl = wl.flat
    return st.decode_drafts(host_bits(dw.q), host_bits(wl.k), host_bits(wl.v),
                            num_kv_heads=wl.num_kv_heads, page_size=wl.page_size,
                            sm_scale=wl.sm_scale, seq_lens=fl.seq_lens_host,
                            block_table=fl.block_table.numpy(),
                            col_indptr=dw.col_indptr.tolist(), parent=dw.parent.tolist(),
                            z=z, T=T)


@pytest.mark.parametrize("tree", [False, True])
def test_drafts_equal_masked_sdpa(tree):
    parents = ([[-1, 0, 0, 1, 2, 2], [-1, -1, 1]] if tree
               else [chain_parents(4), chain_parents(2)])
    dw = make_drafts(committed=[50, 21], parents=parents, heads=8, kv_heads=2, dim=64,
                     spike_count=2, seed=4)
    z = np.full(tuple(dw.q.shape[:2]), 3.0)
    a, l = _draft_oracle(dw, z, INF)
    o = a / l[..., None]
    np.testing.assert_allclose(o, _mask_sdpa(dw), rtol=0, atol=1e-12)


@pytest.mark.parametrize("T", [INF, 4.0])
def test_chain_column_equals_truncated_plain_decode(T):
    """Column c of a chain sees exactly the first n0 + c + 1 keys: the plain
    decode of a view truncated there gives the same pair."""
    m = 5
    dw = make_drafts(committed=[70], parents=[chain_parents(m)], heads=4, kv_heads=1, dim=64,
                     spike_count=3, seed=5)
    wl = dw.wl
    z = np.random.default_rng(0).normal(4.0, 1.0, size=tuple(dw.q.shape[:2]))
    a, l = _draft_oracle(dw, z, T)
    qb = host_bits(dw.q)
    for c in range(m):
        pa, pl = decode_level(qb[c:c + 1], host_bits(wl.k), host_bits(wl.v), num_kv_heads=1,
                              page_size=16, sm_scale=wl.sm_scale, seq_lens=[70 + c + 1],
                              block_table=wl.flat.block_table.numpy(), z=z[c:c + 1], T=T,
                              num_splits=1)
        np.testing.assert_allclose(a[c], pa[0, 0], rtol=1e-13, atol=0)
        np.testing.assert_allclose(l[c], pl[0, 0], rtol=1e-13, atol=0)


def test_drafts_split_into_committed_and_ancestor_levels():
    """Proposition 1(i): the committed keys with every column stacked, plus
    each column's ancestors, add up to the masked pair."""
    parents = [[-1, 0, 1, 0], [-1, 0]]
    dw = make_drafts(committed=[33, 64], parents=parents, heads=4, kv_heads=2, dim=64,
                     seed=6)
    wl = dw.wl
    z = np.full(tuple(dw.q.shape[:2]), 2.0)
    for T in (INF, 3.0):
        a, l = _draft_oracle(dw, z, T)
        ind = dw.col_indptr.tolist()
        pa, pl = decode_level(host_bits(dw.q), host_bits(wl.k), host_bits(wl.v),
                              num_kv_heads=2, page_size=16, sm_scale=wl.sm_scale,
                              seq_lens=dw.committed, block_table=wl.flat.block_table.numpy(),
                              row_indptr=ind, row_req=list(range(dw.num_cols)), z=z, T=T,
                              num_splits=1)
        a2, l2 = pa[0].copy(), pl[0].copy()
        qf = bf16_bits_to_f64(host_bits(dw.q))
        for r, n in enumerate(wl.flat.seq_lens_host):
            m = ind[r + 1] - ind[r]
            for c in range(m):
                vis = st.draft_visible(n, m, parents[r], c)
                anc = vis[vis >= n - m]
                for g in range(2):
                    keys = gather(host_bits(wl.k), r, g, n, wl.flat.block_table.numpy(), 16)
                    vals = gather(host_bits(wl.v), r, g, n, wl.flat.block_table.numpy(), 16)
                    hs = np.arange(2 * g, 2 * g + 2)
                    x = scores(qf[ind[r] + c, hs], keys[anc], wl.sm_scale) - z[ind[r] + c, hs][:, None]
                    live = np.ones(x.shape, bool) if math.isinf(T) else x >= -T
                    a2[ind[r] + c, hs] += (np.exp2(x) * live) @ vals[anc]
                    l2[ind[r] + c, hs] += np.exp2(x).sum(axis=1)
        np.testing.assert_allclose(a2, a, rtol=1e-12, atol=1e-300)
        np.testing.assert_allclose(l2, l, rtol=1e-12, atol=0)
        o, _ = combine(a[None], l[None])
        assert np.isfinite(o).all()


def test_draft_parent_cycle_is_rejected():
    with pytest.raises(ValueError):
        st.draft_visible(10, 3, [1, 2, 0], 0)
