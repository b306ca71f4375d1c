"""Pins of the oracle's cut-key value model (the request mean as the value of
every cut key; Section 4, "Depth as a dial"), CPU only."""

import math

import numpy as np
import pytest
import torch

import oracle
from tests import _adapt
from workloads import host_bits, make_cascade, make_custom

INF = float("inf")


def _wl(seed=0, lens=(300, 517), heads=8, kv=2, d=64, paged=True):
    return make_custom(batch=len(lens), heads=heads, kv_heads=kv, dim=d, lens=list(lens),
                       paged=paged, spike_count=6, alpha_spike=3.0, n_sink=2, alpha_sink=6.0,
                       seed=seed)


def _means(oi, wl):
    fl = oi["flat"]
    return np.stack([np.stack([oracle.value_mean(oi["v_bits"], r, g, n, fl["block_table"],
                                                 wl.page_size)
                               for g in range(wl.num_kv_heads)])
                     for r, n in enumerate(fl["seq_lens"])])


def _decode_model(oi, wl, z, T, splits, mean):
    pa, pl, pc = [], [], []
    for lv, s in zip(oi["levels"], splits):
        a, l, c = oracle.decode_level(oi["q_bits"], oi["k_bits"], oi["v_bits"],
                                      num_kv_heads=wl.num_kv_heads, page_size=wl.page_size,
                                      sm_scale=wl.sm_scale, z=z, T=T, num_splits=s,
                                      with_cut=True, **lv)
        pa.append(a), pl.append(l), pc.append(c)
    pa, pl, pc = np.concatenate(pa), np.concatenate(pl), np.concatenate(pc)
    return oracle.combine(pa, pl, pc, mean, wl.num_kv_heads), (pa, pl, pc)


def test_mean_matches_closed_form():
    """Closed form: values v_j = j * u over j < n have mean (n-1)/2 * u."""
    n, d = 37, 8
    u = np.arange(1, d + 1, dtype=np.float32) / 8      # exact in BF16
    rows = np.stack([j * u for j in range(n)]).astype(np.float32)
    bits = (rows.view(np.uint32) >> 16).astype(np.uint16)[None, None]  # [1, 1, n, d]
    got = oracle.value_mean(bits, 0, 0, n, None, 0)
    np.testing.assert_allclose(got, (n - 1) / 2 * u, rtol=1e-12)
    assert np.array_equal(oracle.value_mean(bits, 0, 0, 0, None, 0), np.zeros(d))


def test_running_mean_equals_batch_mean():
    """The running update from an empty mean reproduces the batch mean."""
    rng = np.random.default_rng(0)
    rows = rng.standard_normal((50, 16))
    mu = np.zeros(16)
    for k, r in enumerate(rows):
        mu = oracle.running_mean(mu, k, r)
    np.testing.assert_allclose(mu, rows.mean(axis=0), rtol=1e-12, atol=1e-14)


@pytest.mark.parametrize("T", [0.0, 4.0, 16.0])
def test_constant_values_make_the_model_exact(T):
    """Closed form: when every value row equals one vector c, the model's
    stand-in is exact, so the output is c at any depth."""
    wl = _wl(seed=1)
    c = torch.linspace(-1, 1, wl.head_dim).to(torch.bfloat16)
    wl.v = c.expand_as(wl.v).contiguous()
    oi = _adapt.oracle_inputs(wl)
    z = _adapt.estimate(oi)
    (o, l), _ = _decode_model(oi, wl, z, T, [3], _means(oi, wl))
    want = c.double().numpy()
    ok = l > 0
    assert np.allclose(o[ok], want, rtol=0, atol=1e-12)
    # without the model the cut mass is lost: the output shrinks towards zero
    o0, _ = oracle.combine(*_decode_model(oi, wl, z, T, [3], _means(oi, wl))[1][:2])
    if T < 16:
        assert np.abs(o0[ok] - want).max() > 1e-3


@pytest.mark.parametrize("T", [2.0, 8.0])
def test_model_equals_softmax_with_cut_values_replaced(T):
    """Library routine: the model's output is softmax attention (torch SDPA,
    FP64) over values in which each row's cut keys carry the request mean."""
    wl = _wl(seed=2, lens=(200, 90))
    oi = _adapt.oracle_inputs(wl)
    z = _adapt.estimate(oi)
    mean = _means(oi, wl)
    (o, _), _ = _decode_model(oi, wl, z, T, [2], mean)
    q = oracle.bf16_bits_to_f64(oi["q_bits"])
    fl = oi["flat"]
    group = wl.num_heads // wl.num_kv_heads
    for r, n in enumerate(fl["seq_lens"]):
        for h in range(wl.num_heads):
            g = h // group
            keys = oracle.gather(oi["k_bits"], r, g, n, fl["block_table"], wl.page_size)
            vals = oracle.gather(oi["v_bits"], r, g, n, fl["block_table"], wl.page_size)
            s = oracle.scores(q[r, h][None], keys, wl.sm_scale)[0]
            cut = ~oracle.live_mask(s - z[r, h], T)
            v2 = vals.copy()
            v2[cut] = mean[r, g]
            want = torch.nn.functional.scaled_dot_product_attention(
                torch.from_numpy(q[r, h])[None, None, None], torch.from_numpy(keys)[None, None],
                torch.from_numpy(v2)[None, None], scale=wl.sm_scale)[0, 0, 0].numpy()
            np.testing.assert_allclose(o[r, h], want, rtol=1e-9, atol=1e-12)


def test_model_is_additive_and_void_at_infinite_depth():
    """The cut masses add over splits like L; at T = inf they are zero."""
    wl = _wl(seed=3)
    oi = _adapt.oracle_inputs(wl)
    z = _adapt.estimate(oi)
    _, (pa1, pl1, pc1) = _decode_model(oi, wl, z, 6.0, [1], _means(oi, wl))
    _, (pa5, pl5, pc5) = _decode_model(oi, wl, z, 6.0, [5], _means(oi, wl))
    np.testing.assert_allclose(pc5.sum(0), pc1[0], rtol=1e-12, atol=1e-300)
    assert pc1.max() > 0
    # cut + live = all: L - Lcut is the live mass, never negative
    assert (pl1 - pc1 >= -1e-12 * pl1).all()
    _, (_, _, pci) = _decode_model(oi, wl, z, INF, [3], _means(oi, wl))
    assert not pci.any()


def test_model_cascade_uses_request_means():
    """A cascade's cut masses over both levels times the request mean equal the
    flat decode of prefix ++ suffix with the same model (per-key rule)."""
    wl = make_cascade(requests=3, heads=4, kv_heads=1, dim=64, prefix_len=160, suffix_len=48,
                      seed=5)
    oi = _adapt.oracle_inputs(wl)
    z = _adapt.estimate(oi)
    mean = _means(oi, wl)
    (o_c, _), _ = _decode_model(oi, wl, z, 5.0, [2, 1], mean)
    flat = dict(oi)
    flat["levels"] = [oi["flat"]]
    (o_f, _), _ = _decode_model(flat, wl, z, 5.0, [3], mean)
    np.testing.assert_allclose(o_c, o_f, rtol=1e-10, atol=1e-13)


# ------------------------------------------------------------ block model --
def _block_means(oi, wl, level=None):
    """{(kv seq, kv head): [ceil(n / 64), D]} block means of a level's view."""
    lv = oi["flat"] if level is None else level
    return {(r, g): oracle.block_means(oi["v_bits"], r, g, n, lv["block_table"], wl.page_size)
            for r, n in enumerate(lv["seq_lens"]) for g in range(wl.num_kv_heads)}


def _decode_blocks(oi, wl, z, T, splits, levels=None, means=None):
    """Slots of every level with the block model on, then the combine."""
    levels = oi["levels"] if levels is None else levels
    pa, pl = [], []
    for i, (lv, s) in enumerate(zip(levels, splits)):
        bm = _block_means(oi, wl, lv) if means is None else means[i]
        a, l = oracle.decode_level(oi["q_bits"], oi["k_bits"], oi["v_bits"],
                                   num_kv_heads=wl.num_kv_heads, page_size=wl.page_size,
                                   sm_scale=wl.sm_scale, z=z, T=T, num_splits=s,
                                   block_mean=bm, **lv)
        pa.append(a), pl.append(l)
    pa, pl = np.concatenate(pa), np.concatenate(pl)
    return oracle.combine(pa, pl), (pa, pl)


def test_block_means_closed_form():
    """Closed form: values v_j = j * u have block means (64 t + 31.5) u for
    full blocks and the mean index of the keys held for the partial last one."""
    n, d = 150, 8
    u = (2.0 ** -np.arange(d)).astype(np.float32)  # j * u is exact in BF16 for j < 256
    rows = np.stack([j * u for j in range(n)]).astype(np.float32)
    assert np.array_equal(rows.astype(np.float64),
                          oracle.bf16_bits_to_f64((rows.view(np.uint32) >> 16).astype(np.uint16)))
    bits = (rows.view(np.uint32) >> 16).astype(np.uint16)[None, None]
    got = oracle.block_means(bits, 0, 0, n, None, 0)
    assert got.shape == (3, d)
    for t, centre in enumerate([31.5, 95.5, (128 + 149) / 2]):
        np.testing.assert_allclose(got[t], centre * u, rtol=1e-12)
    assert oracle.block_means(bits, 0, 0, 0, None, 0).shape == (0, d)


def test_block_means_of_a_paged_view_follow_the_block_table():
    """The paged and the contiguous layout of the same logical values give the
    same block means (the table is followed, not the physical order)."""
    wl = _wl(seed=4, lens=(200, 77))
    oi = _adapt.oracle_inputs(wl)
    for r, n in enumerate(oi["flat"]["seq_lens"]):
        for g in range(wl.num_kv_heads):
            want = host_bits(wl.logical_v)[r, g, :n]
            want = oracle.bf16_bits_to_f64(want)
            got = oracle.block_means(oi["v_bits"], r, g, n, oi["flat"]["block_table"],
                                     wl.page_size)
            for t in range(got.shape[0]):
                np.testing.assert_allclose(got[t], want[64 * t:64 * t + 64].mean(axis=0),
                                           rtol=1e-13, atol=1e-15)


@pytest.mark.parametrize("T,splits", [(2.0, 1), (6.0, 3), (0.0, 2)])
def test_block_model_equals_softmax_with_cut_values_replaced(T, splits):
    """Library routine: with the block model the output is softmax attention
    (torch SDPA, FP64) over values in which each row's cut keys carry the mean
    value row of their own 64-key block."""
    wl = _wl(seed=5, lens=(300, 130))
    oi = _adapt.oracle_inputs(wl)
    z = _adapt.estimate(oi)
    (o, _), _ = _decode_blocks(oi, wl, z, T, [splits])
    q = oracle.bf16_bits_to_f64(oi["q_bits"])
    fl = oi["flat"]
    group = wl.num_heads // wl.num_kv_heads
    n_cut = 0
    for r, n in enumerate(fl["seq_lens"]):
        for h in range(wl.num_heads):
            g = h // group
            keys = oracle.gather(oi["k_bits"], r, g, n, fl["block_table"], wl.page_size)
            vals = oracle.gather(oi["v_bits"], r, g, n, fl["block_table"], wl.page_size)
            s = oracle.scores(q[r, h][None], keys, wl.sm_scale)[0]
            cut = ~oracle.live_mask(s - z[r, h], T)
            n_cut += int(cut.sum())
            v2 = vals.copy()
            for j in np.nonzero(cut)[0]:
                t = j // 64
                v2[j] = vals[64 * t:min(n, 64 * t + 64)].mean(axis=0)
            want = torch.nn.functional.scaled_dot_product_attention(
                torch.from_numpy(q[r, h])[None, None, None], torch.from_numpy(keys)[None, None],
                torch.from_numpy(v2)[None, None], scale=wl.sm_scale)[0, 0, 0].numpy()
            np.testing.assert_allclose(o[r, h], want, rtol=1e-9, atol=1e-12)
    assert n_cut > 100


@pytest.mark.parametrize("T", [0.0, 5.0, 16.0])
def test_blockwise_constant_values_make_the_block_model_exact(T):
    """Closed form: when the value rows are constant within every 64-key block
    (and differ between blocks), the block model's stand-in is each cut key's
    own value, so the output is dense softmax at every depth; the request-mean
    model is not exact on the same cache."""
    wl = _wl(seed=6, lens=(300, 200), paged=False)
    n_max = wl.v.shape[2]
    per_block = torch.randn(wl.v.shape[0], wl.v.shape[1], (n_max + 63) // 64, wl.head_dim,
                            generator=torch.Generator().manual_seed(1)).to(torch.bfloat16)
    wl.v = per_block.repeat_interleave(64, dim=2)[:, :, :n_max].contiguous()
    oi = _adapt.oracle_inputs(wl)
    z = _adapt.estimate(oi)
    (o, l), _ = _decode_blocks(oi, wl, z, T, [2])
    (o_dense, _), _ = _decode_blocks(oi, wl, z, INF, [2])
    ok = l > 0
    assert np.allclose(o[ok], o_dense[ok], rtol=0, atol=1e-12)
    (o_mean, _), _ = _decode_model(oi, wl, z, T, [2], _means(oi, wl))
    if T < 16:
        assert np.abs(o_mean[ok] - o_dense[ok]).max() > 1e-3


def test_block_model_is_additive_and_void_at_infinite_depth():
    """Each tile's virtual row belongs to the split that owns the tile: the
    slots of five splits add up to the one slot of a single split, and at
    T = inf the block model changes no slot."""
    wl = _wl(seed=7, lens=(517, 300))
    oi = _adapt.oracle_inputs(wl)
    z = _adapt.estimate(oi)
    _, (pa1, pl1) = _decode_blocks(oi, wl, z, 4.0, [1])
    _, (pa5, pl5) = _decode_blocks(oi, wl, z, 4.0, [5])
    np.testing.assert_allclose(pa5.sum(0), pa1[0], rtol=1e-11, atol=1e-13)
    np.testing.assert_allclose(pl5.sum(0), pl1[0], rtol=1e-12)
    # the virtual rows are what the model adds to the plain scan's slots
    _, (pa0, _, _) = _decode_model(oi, wl, z, 4.0, [5], _means(oi, wl))
    assert np.abs(pa5 - pa0).max() > 1e-6
    _, (pai, _) = _decode_blocks(oi, wl, z, INF, [3])
    _, (pa_plain, _, _) = _decode_model(oi, wl, z, INF, [3], _means(oi, wl))
    assert np.array_equal(pai, pa_plain)


def test_block_model_cascade_equals_flat_when_blocks_align():
    """A cascade whose prefix is a whole number of 64-key blocks has the same
    blocks as the flat prefix ++ suffix view, so the cascade with per-level
    block means equals the flat decode with the flat block means."""
    wl = make_cascade(requests=3, heads=4, kv_heads=1, dim=64, prefix_len=192, suffix_len=80,
                      seed=8)
    oi = _adapt.oracle_inputs(wl)
    z = _adapt.estimate(oi)
    (o_c, _), _ = _decode_blocks(oi, wl, z, 5.0, [2, 1])
    (o_f, _), _ = _decode_blocks(oi, wl, z, 5.0, [3], levels=[oi["flat"]])
    np.testing.assert_allclose(o_c, o_f, rtol=1e-10, atol=1e-13)


def test_running_update_builds_the_block_means():
    """Appending one token at a time with the running update of its block
    (count = position mod 64) reproduces the block means."""
    rng = np.random.default_rng(3)
    rows = rng.standard_normal((150, 16)).astype(np.float32)
    bits = (rows.view(np.uint32) >> 16).astype(np.uint16)
    vals = oracle.bf16_bits_to_f64(bits)
    mu = np.zeros((3, 16))
    for j in range(150):
        mu[j // 64] = oracle.running_mean(mu[j // 64], j % 64, vals[j])
    np.testing.assert_allclose(mu, oracle.block_means(bits[None, None], 0, 0, 150, None, 0),
                               rtol=1e-12, atol=1e-14)
