"""Both levels of a shared-prefix cascade in one scan launch
(fold_decode_cascade) against the FP64 oracle.

The oracle decodes the prefix level with S splits and the suffix level with
one split per 64-key tile (U splits).  The expected slot s of row (r, h) is
the prefix slot s plus the suffix tiles u whose pair index p * U + u falls to
split s, p being the request's position among the requests of the row's read
group of 64 stacked rows.  Bars: every slot's L within rtol 2e-5 (L holds
every weight, so it does not depend on the verdicts); the output per row
max-abs error <= 1e-2 * |o_i|_inf against the oracle's own FP64 verdicts,
plus 2 * 2^-T * max|v| / L / |o|_inf for every key whose FP64 x lies within
1e-4 of -T (where the kernel's FP32 verdict may differ); at finite T every
slot's cut mass within rtol 2e-5 plus 2^(-T+1e-4) per such key; and the
output against the two-launch path (fold_decode_split per level) within 1e-4
of |o|_inf, since only the slots' summation order differs.
"""

import dataclasses
import math

import numpy as np
import pytest
import torch

import oracle
from tests import _adapt, _gpu
from workloads import make_cascade, make_config

pytestmark = pytest.mark.gpu
INF = float("inf")
TOL = 1e-2
NEAR = 1e-4


@pytest.fixture(scope="module", autouse=True)
def _device():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2609_33410_amd as F
    F.load_library()  # raises if the HIP library is not built: never a silent fallback


def _tiles(n):
    return (n + 63) // 64


def _positions(wl):
    """Position of each row's request among the requests of its read group."""
    pre = wl.levels[0]
    indptr = pre.row_indptr.cpu().numpy()
    req = pre.row_req.cpu().numpy()
    G = wl.num_heads // wl.num_kv_heads
    b = wl.q.shape[0]
    pos = np.full((b, wl.num_heads), -1, dtype=np.int64)
    for seq in range(len(indptr) - 1):
        for p, r in enumerate(req[indptr[seq]:indptr[seq + 1]]):
            for hh in range(G):
                rho = p * G + hh
                for kvh in range(wl.num_kv_heads):
                    pos[r, kvh * G + hh] = p - (64 * (rho // 64)) // G
    return pos


def _expected_slots(wl, pa, pl, S):
    """Compose the oracle's per-level slots (prefix: S splits, suffix: one per
    tile) into the one-launch slots."""
    U = _tiles(wl.levels[1].max_seq_len)
    ea, el = pa[:S].copy(), pl[:S].copy()
    pos = _positions(wl)
    b, h = pl.shape[1:]
    rr, hh = np.meshgrid(np.arange(b), np.arange(h), indexing="ij")
    covered = pos >= 0
    for u in range(U):
        slot = (pos * U + u) % S
        np.add.at(ea, (slot[covered], rr[covered], hh[covered]), pa[S + u][covered])
        np.add.at(el, (slot[covered], rr[covered], hh[covered]), pl[S + u][covered])
    return ea, el


def _near_counts(wl, oi, z64, T):
    """Keys per row whose FP64 x = s - Z lies within NEAR of -T."""
    q = oracle.bf16_bits_to_f64(oi["q_bits"])
    b, h = z64.shape
    near = np.zeros((b, h))
    G = wl.num_heads // wl.num_kv_heads
    for lv in oi["levels"]:
        for seq, n in enumerate(lv["seq_lens"]):
            reqs = [seq] if lv["row_indptr"] is None else \
                list(lv["row_req"][lv["row_indptr"][seq]:lv["row_indptr"][seq + 1]])
            for g in range(wl.num_kv_heads):
                keys = oracle.gather(oi["k_bits"], seq, g, n, lv["block_table"], wl.page_size)
                for r in reqs:
                    hs = [g * G + k for k in range(G)]
                    x = oracle.scores(q[r, hs], keys, wl.sm_scale) - z64[r, hs][:, None]
                    near[r, hs] += (np.abs(x + T) <= NEAR).sum(axis=1)
    return near


def _cascade(wl, T, S, z):
    import paper_2609_33410_amd as F

    levels, _ = _gpu.kv_views(wl)
    qv = F.q_view(wl.q)
    b, h, d = wl.q.shape
    dev = wl.q.device
    part_a = torch.full((S, b, h, d), float("nan"), dtype=torch.float32, device=dev)
    part_l = torch.full((S, b, h), float("nan"), dtype=torch.float32, device=dev)
    part_c = torch.full((S, b, h), float("nan"), dtype=torch.float32, device=dev)
    F.fold_decode_cascade(levels[0], levels[1], qv, wl.sm_scale, z, T, S, 0, part_a, part_l,
                          part_Lcut=part_c)
    out = torch.empty(b, h, d, dtype=torch.float32, device=dev)
    F.fold_combine(part_a, part_l, out)
    torch.cuda.synchronize()
    return out.cpu().numpy(), part_a.cpu().numpy(), part_l.cpu().numpy(), part_c.cpu().numpy()


def _check(wl, T, S, two_launch=True):
    print(f"  {wl.name} rows={wl.q.shape[0] * wl.q.shape[1]} T={T} S={S}", flush=True)
    z = _gpu.estimate(wl)
    z64 = z.double().cpu().numpy()
    oi = _adapt.oracle_inputs(wl)
    out, pa, pl, pc = _cascade(wl, T, S, z)
    assert np.isfinite(pa).all() and np.isfinite(pl).all()
    o_own, l_own, opa, opl = _adapt.decode(oi, z64, T, [S, _tiles(wl.levels[1].max_seq_len)])
    _, el = _expected_slots(wl, opa, opl, S)
    assert np.allclose(pl, el, rtol=2e-5, atol=0)
    err = _gpu.row_errors(out, o_own)
    bound = np.full(err.shape, TOL)
    if not math.isinf(T):
        vmax = float(np.abs(oracle.bf16_bits_to_f64(oi["v_bits"])).max())
        near = _near_counts(wl, oi, z64, T)
        bound = bound + 2.0 * 2.0 ** -T * near * vmax / np.maximum(l_own, 1e-300) \
            / np.maximum(np.abs(o_own).max(axis=-1), 1e-300)
        # cut mass per slot: the oracle's per-level cut slots composed like L;
        # a key within NEAR of -T may sit on either side (weight <= 2^-T+NEAR)
        cuts = [oracle.decode_level(oi["q_bits"], oi["k_bits"], oi["v_bits"],
                                    num_kv_heads=oi["num_kv_heads"], page_size=oi["page_size"],
                                    sm_scale=oi["sm_scale"], z=z64, T=T, num_splits=s_,
                                    with_cut=True, **lv)[2]
                for lv, s_ in zip(oi["levels"], [S, _tiles(wl.levels[1].max_seq_len)])]
        _, ec = _expected_slots(wl, opa, np.concatenate(cuts, axis=0), S)
        slack = 2e-5 * ec + near[None] * 2.0 ** (-T + NEAR)
        assert (np.abs(pc - ec) <= slack).all()
    else:
        assert (pc == 0).all()
    print(f"    max row err = {err.max():.3e}", flush=True)
    assert (err <= bound).all()
    if two_launch and (math.isinf(T) or T >= 16):
        ref = _gpu.run(wl, T, z=z)["out"].numpy()
        d2 = np.abs(out - ref).max(axis=-1) / np.maximum(np.abs(ref).max(axis=-1), 1e-30)
        print(f"    vs two launches: {d2.max():.3e}", flush=True)
        assert (d2 <= 1e-4).all()


@pytest.mark.parametrize("d,requests,heads,kv_heads,prefix,suffix,S", [
    (128, 5, 8, 1, 1488, 48, 3),    # 40 rows: one partial read group
    (64, 8, 8, 1, 1024, 48, 1),     # 64 rows, one split: 16 prefix + 8 suffix tiles
    (128, 12, 8, 1, 2000, 96, 4),   # two read groups; a partial second suffix tile
    (128, 17, 8, 1, 80, 48, 2),     # three groups; suffix tiles among the first five
    (128, 24, 8, 2, 784, 32, 2),    # two kv heads, 96 rows each
    (128, 9, 12, 1, 512, 64, 4),    # G = 12: a request's rows straddle two read groups
])
def test_cascade_matches_oracle(d, requests, heads, kv_heads, prefix, suffix, S):
    wl = make_cascade(requests=requests, heads=heads, kv_heads=kv_heads, dim=d,
                      prefix_len=prefix, suffix_len=suffix, splits=(S, 1),
                      seed=requests + heads + d, device="cuda")
    for T in (INF, 16.0, 6.0):
        _check(wl, T, S)


def test_cascade_ragged_suffixes_and_row_order():
    """Suffix lengths from 0 to 176 keys (a request with no suffix, partial
    chunks) and a prefix row list in permuted request order."""
    wl = make_cascade(requests=10, heads=8, kv_heads=1, dim=128, prefix_len=640,
                      suffix_len=176, splits=(4, 1), seed=7, device="cuda")
    dev = wl.q.device
    lens = [176, 0, 5, 64, 65, 130, 17, 176, 1, 100]
    pre, suf, flat = wl.levels[0], wl.levels[1], wl.flat
    plen = wl.meta["prefix_len"]
    suf = dataclasses.replace(suf, seq_lens=torch.tensor(lens, dtype=torch.int32, device=dev),
                              seq_lens_host=list(lens))
    flens = [plen + n for n in lens]
    flat = dataclasses.replace(flat, seq_lens=torch.tensor(flens, dtype=torch.int32, device=dev),
                               seq_lens_host=flens)
    perm = torch.tensor([3, 7, 0, 9, 1, 5, 2, 8, 6, 4], dtype=torch.int32, device=dev)
    pre = dataclasses.replace(pre, row_req=perm)
    wl = dataclasses.replace(wl, flat=flat, levels=[pre, suf])
    for T in (INF, 16.0, 5.0):
        _check(wl, T, 4)


def test_cascade_two_prefix_sequences():
    """A prefix view of two kv sequences (over the same pages) that serve two
    disjoint request sets, one of them in permuted order: read groups and
    request positions are per prefix sequence."""
    wl = make_cascade(requests=12, heads=8, kv_heads=1, dim=128, prefix_len=1024,
                      suffix_len=96, splits=(4, 1), seed=11, device="cuda")
    dev = wl.q.device
    pre = wl.levels[0]
    bt = pre.block_table.expand(2, -1).contiguous()
    indptr = torch.tensor([0, 5, 12], dtype=torch.int32, device=dev)
    req = torch.tensor([0, 1, 2, 3, 4, 11, 6, 9, 8, 5, 10, 7], dtype=torch.int32, device=dev)
    n = pre.seq_lens_host[0]
    pre = dataclasses.replace(pre, block_table=bt,
                              seq_lens=torch.tensor([n, n], dtype=torch.int32, device=dev),
                              seq_lens_host=[n, n], row_indptr=indptr, row_req=req,
                              max_reqs_per_seq=7)
    wl = dataclasses.replace(wl, levels=[pre, wl.levels[1]])
    for T in (INF, 16.0, 6.0):
        _check(wl, T, 4)


@pytest.mark.parametrize("T", [INF, 16.0])
def test_cascade_workload5_full(T):
    """The 64 x (16384 + 1024)-key cascade with 32 splits: 8 prefix and 4
    suffix tiles per workgroup."""
    wl = make_config(5, device="cuda")
    _check(wl, T, 32, two_launch=True)
