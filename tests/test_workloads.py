"""The seeded input generator: shapes, reproducibility and planted structure."""

import math

import numpy as np
import torch

from workloads import host_bits, make_config, make_custom


def test_reproducible_and_seed_sensitive():
    a = make_config(1)
    b = make_config(1)
    c = make_config(1, seed=1)
    assert torch.equal(a.k, b.k) and torch.equal(a.q, b.q) and torch.equal(a.v, b.v)
    assert not torch.equal(a.k, c.k)


def test_config1_shapes_and_spikes():
    wl = make_config(1, keep_logical=True)
    assert wl.q.shape == (1, 4, 64) and wl.k.shape == (1, 4, 512, 64)
    assert wl.flat.block_table is None and wl.flat.seq_lens_host == [512]
    u = wl.q.float()[0] / wl.q.float()[0].norm(dim=-1, keepdim=True)
    for h in range(4):
        idx = wl.meta["spikes"][(0, h)]
        assert len(set(idx.tolist())) == 8
        proj = wl.k[0, h].float() @ u[h]
        # planted spikes project ~ 4*sqrt(64) = 32 along q_h; the bulk ~ N(0,1)
        assert (proj[idx] > 24).all()
        rest = np.setdiff1d(np.arange(512), idx.numpy())
        assert proj[rest].abs().max() < 8


def test_paged_table_is_a_permutation():
    wl = make_config(2, batch=3, seq_len=1000)
    bt = wl.flat.block_table
    npg = (1000 + 15) // 16
    used = bt[:, :npg].flatten().tolist()
    assert sorted(used) == list(range(wl.k.shape[0]))
    assert wl.k.shape == (3 * npg, 8, 16, 128)


def test_spike_and_sink_counts_config2_shape():
    wl = make_config(2, batch=2, seq_len=2000)
    for (r, g), idx in wl.meta["spikes"].items():
        assert len(idx) == round(0.01 * 2000)
        assert idx.min() >= 4  # sinks 0..3 are not spike candidates


def test_ragged_lengths_drawn_first_and_in_range():
    wl = make_config(4, batch=4, seq_len=4096)
    lens = wl.flat.seq_lens_host
    assert all(2048 <= n <= 4096 for n in lens)
    assert len(set(lens)) > 1


def test_cascade_views():
    wl = make_config(5, batch=4, seq_len=256)
    pre, suf = wl.levels
    assert pre.num_seqs == 1 and pre.seq_lens_host == [256]
    assert pre.row_req.tolist() == [0, 1, 2, 3] and pre.row_indptr.tolist() == [0, 4]
    assert suf.num_seqs == 4 and suf.seq_lens_host == [16] * 4
    flat = wl.flat.block_table
    assert torch.equal(flat[:, :16], pre.block_table.expand(4, -1))
    assert torch.equal(flat[:, 16:], suf.block_table)


def test_host_bits_roundtrip():
    t = torch.randn(100).to(torch.bfloat16)
    b = host_bits(t)
    assert b.dtype == np.uint16
    back = torch.from_numpy(b.view(np.int16).copy()).view(torch.bfloat16)
    assert torch.equal(back, t)
