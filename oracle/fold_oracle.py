"""FoldAttention decode: a plain, slow FP64 CPU oracle.

TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the
benchmark's CPU-baseline leg may import or call this module.  The product
path (the HIP library and its Python binding) never touches it, and this
module imports nothing from the product path.

Everything is numpy FP64, computed step by step in the paper's order and
notation:

* O1  gather the keys/values of one (kv sequence, kv head) from the paged
      cache (Section 4, paged cache with a per-request block table);
* O2  base-2 scores ``s_ij = log2(e) * sm_scale * q_i . k_j`` (Section 2,
      online-softmax paragraph; the dot product is formed first, then scaled);
* O3  the reference ``Z_i`` is an input of decode (Eq. fold: it is fixed
      before any key is read); ``estimate_z`` below is the oracle's own
      reading of the estimator of Section 3 ("Choosing the reference");
* O4  depth rule (Section 4, weight-gated reads and depth paragraphs;
      Algorithm 1): ``x_ij = s_ij - Z_i``; a key is live iff ``T`` is
      infinite or ``x_ij >= -T`` (the tie ``x = -T`` is live);
* O5  fold (Eq. fold and the depth paragraph): ``w = 2**x``;
      ``A_i = sum_{live j} w_ij v_j``; ``L_i = sum_{all j} w_ij`` (cut keys
      keep their mass in L but add nothing to A);
* O6  splits (Section 4; Algorithm 1's input list): 64-key tile ``t`` belongs
      to split ``t mod S``;
* O7  combine (Algorithm 1, last step): ``o_i = sum_s A_i^s / sum_s L_i^s``
      over slots in increasing order; a cascade simply has more slots
      (Section 4, value product paragraph);
* O8  read gates: a key is read iff some row of the read group is live on it;
      a 16-key page is read iff one of its keys is (Section 4; Algorithm 1);
* O9  per-row diagnostics (Proposition 1(iii), the certificate window of
      Section 3, the truncation bound, live fractions);
* O10 cut-key value models (Section 4, "Depth as a dial"; Algorithm 1's
      virtual row): the request mean (``value_mean``, ``running_mean``) whose
      weight is a slot's cut mass, and the block model of BF16 values
      (``block_means``; ``decode_level(block_mean=...)``), one virtual row per
      64-key tile carrying the tile's cut mass times the block's mean.

Readings of points the paper leaves open are listed in the design notes of
the repository (score scale, tie at the threshold, cut keys' value, gate
granularity, estimator details, empty rows, combine order).

Parity status: O1-O10 are pinned by the CPU tests (closed forms, textbook and
library softmax, invariants, hand-computed fixtures; O10 against library
softmax over values with the cut keys replaced by their model; O9 by a hand-computed
fixture of exact binary fractions and by an independent FP64 evaluation of
the Proposition 1(iii) left side on every row of every workload).  The estimator's
stratified/trimmed branch (n > 192) is pinned only structurally (exact
cases, which keys it reads, what its trim discards); the paper prints no
value to check it against, so its exact value is "parity unpinned".
"""

from __future__ import annotations

import math
from typing import Dict, Iterable, List, Optional, Sequence, Tuple

import numpy as np

LOG2E = 1.0 / math.log(2.0)
TILE = 64          # keys per tile of the split interleave (Section 4)
PAGE_GATE = 16     # keys per page-gate bit
CERT_LO = 0.5      # certificate window [2^-1, 2^100] on L (Section 3)
CERT_HI = 2.0 ** 100

EST_DEFAULT = {"sink": 1, "recent": 63, "strata": 128, "trim_lo": 8, "trim_hi": 8}


# ---------------------------------------------------------------- O1 -------
def bf16_bits_to_f64(bits: np.ndarray) -> np.ndarray:
    """Exact value of BF16 bit patterns: the bits are the top half of an FP32."""
    b = np.ascontiguousarray(bits, dtype=np.uint16)
    with np.errstate(invalid="ignore"):
        return (b.astype(np.uint32) << np.uint32(16)).view(np.float32).astype(np.float64)


def gather(cache_bits: np.ndarray, seq: int, g: int, n: int,
           block_table: Optional[np.ndarray], page_size: int) -> np.ndarray:
    """Rows 0..n-1 of kv sequence ``seq``, kv head ``g``, as FP64 ``[n, D]``.

    Paged: key j lives in physical page ``block_table[seq, j // P]`` at slot
    ``j % P`` of the page's ``[Hkv, P, D]`` slab.  Contiguous (no table): the
    cache is ``[num_seqs, Hkv, max_len, D]``.
    """
    if n == 0:
        return np.zeros((0, cache_bits.shape[-1]), dtype=np.float64)
    if block_table is None:
        rows = cache_bits[seq, g, :n, :]
    else:
        j = np.arange(n)
        pages = np.asarray(block_table[seq])[j // page_size]
        rows = cache_bits[pages, g, j % page_size, :]
    return bf16_bits_to_f64(rows)


# ---------------------------------------------------------------- O2 -------
def scores(q_rows: np.ndarray, keys: np.ndarray, sm_scale: float) -> np.ndarray:
    """Base-2 scores ``s[i, j] = log2(e) * sm_scale * (q_i . k_j)``, FP64."""
    return (q_rows @ keys.T) * (LOG2E * sm_scale)


# ---------------------------------------------------------------- O4 -------
def live_mask(x: np.ndarray, T: float) -> np.ndarray:
    """Depth rule: live iff T is infinite or x >= -T (the tie is live)."""
    if math.isinf(T):
        return np.ones(x.shape, dtype=bool)
    return x >= -T


def live_mask_imposed(x_f32: np.ndarray, T: float) -> np.ndarray:
    """The same rule evaluated in FP32 on given FP32 ``x`` values."""
    x_f32 = np.asarray(x_f32, dtype=np.float32)
    if math.isinf(T):
        return np.ones(x_f32.shape, dtype=bool)
    return x_f32 >= np.float32(-T)


# ---------------------------------------------------------------- O5 -------
def fold(x: np.ndarray, live: np.ndarray, values: np.ndarray) -> Tuple[np.ndarray, np.ndarray]:
    """``F = (A, L)``: ``A = sum_{live} 2^x v``, ``L = sum_{all} 2^x``."""
    w = np.exp2(x)
    a = (w * live) @ values
    l = w.sum(axis=-1)
    return a, l


# ---------------------------------------------------------------- O6 -------
def split_of_key(n: int, num_splits: int) -> np.ndarray:
    """Split owning each key: tile ``j // 64`` goes to split ``tile % S``."""
    return (np.arange(n) // TILE) % num_splits


# --------------------------------------------------------- cut-key model ---
def value_mean(v_bits: np.ndarray, seq: int, g: int, n: int, block_table, page_size: int
               ) -> np.ndarray:
    """Mean value row of keys 0..n-1 of (seq, g), FP64 (0 for an empty row).

    The request's running mean of Section 4 ("Depth as a dial"): the value
    model that stands in for every cut key."""
    d = v_bits.shape[-1]
    if n == 0:
        return np.zeros(d)
    return gather(v_bits, seq, g, n, block_table, page_size).mean(axis=0)


def running_mean(prev: np.ndarray, count: int, v_new: np.ndarray) -> np.ndarray:
    """Mean of count + 1 rows from the mean of the first count and the new row."""
    return prev + (np.asarray(v_new, dtype=np.float64) - prev) / (count + 1)


def block_means(v_bits: np.ndarray, seq: int, g: int, n: int, block_table, page_size: int
                ) -> np.ndarray:
    """Mean value row of every 64-key block of keys 0..n-1 of (seq, g), FP64
    ``[ceil(n / 64), D]``; the last block averages the keys it holds.

    The mean part of the block model of BF16 values (Section 4, "Depth as a
    dial"): a cut key of block t is modelled by block t's mean value row."""
    vals = gather(v_bits, seq, g, n, block_table, page_size)
    nblk = (n + TILE - 1) // TILE
    out = np.zeros((nblk, v_bits.shape[-1]))
    for t in range(nblk):
        out[t] = vals[t * TILE:(t + 1) * TILE].mean(axis=0)
    return out


# ------------------------------------------------------------ level driver -
def _rows_of(seq: int, g: int, group: int, row_indptr, row_req) -> List[Tuple[int, int]]:
    """(request, head) pairs of the query rows that attend kv seq ``seq``, head ``g``."""
    if row_indptr is None:
        reqs = [seq]
    else:
        reqs = [int(r) for r in row_req[row_indptr[seq]:row_indptr[seq + 1]]]
    return [(r, g * group + hh) for r in reqs for hh in range(group)]


def decode_level(q_bits, k_bits, v_bits, *, num_kv_heads: int, page_size: int,
                 sm_scale: float, seq_lens: Sequence[int], block_table=None,
                 row_indptr=None, row_req=None, z: np.ndarray, T: float, num_splits: int,
                 imposed_x: Optional[np.ndarray] = None,
                 chunks: Optional[Iterable[Tuple[int, int]]] = None,
                 with_cut: bool = False, block_mean=None):
    """Split partials of one scan level (steps O1-O6).

    Returns ``part_A [S, B, H, D]`` and ``part_L [S, B, H]`` (FP64); rows the
    level does not cover stay zero.  ``imposed_x`` ``[B, H, max_len]`` FP32,
    if given, replaces the FP64 live decisions by the FP32 rule applied to
    those values.  ``chunks`` restricts the work to the listed
    ``(kv seq, kv head)`` pairs.  With ``with_cut`` a third array
    ``part_Lcut [S, B, H]`` holds the cut keys' summed weights (the mass the
    value model of Section 4 attaches to its virtual row).  With
    ``block_mean`` (a mapping ``(kv seq, kv head) -> [ceil(n / 64), D]``
    block mean rows, see ``block_means``) the block model of BF16 values is
    on: every 64-key tile ``t`` of a split has one virtual row whose weight is
    the row's summed weight of the tile's cut keys ``c_it`` and whose value is
    the block's mean ``mu_t``, so the split's *A* gains ``sum_t c_it mu_t``
    (Section 4, "Depth as a dial"; Algorithm 1, the tile's virtual row).
    """
    q = bf16_bits_to_f64(q_bits)
    b, h, d = q.shape
    group = h // num_kv_heads
    part_a = np.zeros((num_splits, b, h, d))
    part_l = np.zeros((num_splits, b, h))
    part_c = np.zeros((num_splits, b, h))
    if chunks is None:
        chunks = [(s, g) for s in range(len(seq_lens)) for g in range(num_kv_heads)]
    for seq, g in chunks:
        n = int(seq_lens[seq])
        rows = _rows_of(seq, g, group, row_indptr, row_req)
        if n == 0 or not rows:
            continue
        keys = gather(k_bits, seq, g, n, block_table, page_size)
        vals = gather(v_bits, seq, g, n, block_table, page_size)
        ri = np.array([r for r, _ in rows])
        hi = np.array([hh for _, hh in rows])
        s = scores(q[ri, hi], keys, sm_scale)
        x = s - np.asarray(z, dtype=np.float64)[ri, hi][:, None]
        if imposed_x is None:
            live = live_mask(x, T)
        else:
            live = live_mask_imposed(imposed_x[ri, hi, :n], T)
        owner = split_of_key(n, num_splits)
        for sp in range(num_splits):
            m = owner == sp
            if not m.any():
                continue
            a, l = fold(x[:, m], live[:, m], vals[m])
            if block_mean is not None:
                mu = np.asarray(block_mean[(seq, g)], dtype=np.float64)
                cut_w = np.exp2(x) * ~live
                for t in range(sp, (n + TILE - 1) // TILE, num_splits):
                    c_t = cut_w[:, t * TILE:(t + 1) * TILE].sum(axis=-1)
                    a = a + c_t[:, None] * mu[t][None, :]
            part_a[sp, ri, hi] = a
            part_l[sp, ri, hi] = l
            part_c[sp, ri, hi] = (np.exp2(x[:, m]) * ~live[:, m]).sum(axis=-1)
    if with_cut:
        return part_a, part_l, part_c
    return part_a, part_l


# ---------------------------------------------------------------- O7 -------
def combine(part_a: np.ndarray, part_l: np.ndarray, part_lcut: Optional[np.ndarray] = None,
            mean: Optional[np.ndarray] = None, num_kv_heads: int = 1
            ) -> Tuple[np.ndarray, np.ndarray]:
    """Sum the slots in increasing order and take the quotient ``A / L``.

    With the cut-key value model (``part_lcut [S, B, H]`` and the request
    means ``mean [B, Hkv, D]``), the cut keys of every slot add their summed
    weight times the mean of the row's request and kv head to *A*: a virtual
    row whose weight is the cut mass (Section 4, "Depth as a dial").  The
    term is linear in the cut mass, so adding it per slot or after the slot
    sum is the same value."""
    a = np.zeros(part_a.shape[1:])
    l = np.zeros(part_l.shape[1:])
    for s in range(part_a.shape[0]):
        a = a + part_a[s]
        l = l + part_l[s]
    if part_lcut is not None:
        c = np.zeros(part_lcut.shape[1:])
        for s in range(part_lcut.shape[0]):
            c = c + part_lcut[s]
        b_, h = c.shape
        group = h // num_kv_heads
        mu = np.asarray(mean, dtype=np.float64)[:, np.arange(h) // group, :]  # [B, H, D]
        a = a + c[..., None] * mu
    with np.errstate(invalid="ignore", divide="ignore"):
        o = a / l[..., None]
    return o, l


def lse_and_cert(z: np.ndarray, l: np.ndarray, o: np.ndarray) -> Tuple[np.ndarray, np.ndarray]:
    """Base-2 log-sum-exp ``Z + log2 L`` and certificate bits.

    bit0: L < 2^-1; bit1: L > 2^100; bit2: some output entry is not finite
    (Section 3, certificate paragraph).
    """
    with np.errstate(divide="ignore", invalid="ignore"):
        lse = np.asarray(z, dtype=np.float64) + np.log2(l)
    cert = ((l < CERT_LO).astype(np.uint8)
            | ((l > CERT_HI).astype(np.uint8) << 1)
            | ((~np.isfinite(o).all(axis=-1)).astype(np.uint8) << 2))
    return lse, cert


def decode(q_bits, k_bits, v_bits, *, num_kv_heads, page_size, sm_scale, levels, z, T,
           splits: Sequence[int], imposed_x_per_level=None):
    """Whole decode: every level's partials, concatenated as slots, then O7."""
    pa, pl = [], []
    for li, lv in enumerate(levels):
        ix = None if imposed_x_per_level is None else imposed_x_per_level[li]
        a, l = decode_level(q_bits, k_bits, v_bits, num_kv_heads=num_kv_heads,
                            page_size=page_size, sm_scale=sm_scale, z=z, T=T,
                            num_splits=splits[li], imposed_x=ix, **lv)
        pa.append(a)
        pl.append(l)
    part_a = np.concatenate(pa, axis=0)
    part_l = np.concatenate(pl, axis=0)
    o, l = combine(part_a, part_l)
    return o, l, part_a, part_l


# ---------------------------------------------------------------- O3 -------
def estimator_keys(n: int, p: Dict[str, int] = EST_DEFAULT):
    """Indices the estimator scores for a request of ``n`` keys.

    Returns ``(exact, centres, r)``.  For ``n <= sink + recent + strata`` every
    key is exact and there are no strata.  Otherwise the exact keys are the
    first ``sink`` keys and the last ``recent`` keys, and the ``r`` keys in
    between are cut into ``strata`` contiguous strata
    ``[lo_b, hi_b)`` with ``lo_b = sink + floor(b r / strata)``; stratum b is
    represented by its centre ``floor((lo_b + hi_b - 1) / 2)``.
    """
    sink, recent, strata = p["sink"], p["recent"], p["strata"]
    if n <= sink + recent + strata:
        return np.arange(n), np.zeros(0, dtype=np.int64), 0
    r = n - sink - recent
    exact = np.concatenate([np.arange(sink), np.arange(n - recent, n)])
    b = np.arange(strata)
    lo = sink + (b * r) // strata
    hi = sink + ((b + 1) * r) // strata
    centres = (lo + hi - 1) // 2
    return exact, centres, r


def estimate_z(s_row: np.ndarray, p: Dict[str, int] = EST_DEFAULT) -> float:
    """Reference estimate of one row from its FP64 scores over all n keys.

    Base-2 log-sum-exp of the exact keys plus a trimmed stratified estimate
    of the remaining mass: the centre weights are sorted, the ``trim_lo``
    smallest and ``trim_hi`` largest are dropped, and the rest's mean stands
    for every one of the ``r`` stratified keys (Section 3, "Choosing the
    reference").  Weights are taken relative to the largest sampled score M.
    """
    n = s_row.shape[0]
    if n == 0:
        return 0.0
    exact, centres, r = estimator_keys(n, p)
    sampled = np.concatenate([s_row[exact], s_row[centres]])
    m = sampled.max()
    exact_mass = np.exp2(s_row[exact] - m).sum()
    mass_r = 0.0
    if r > 0:
        u = np.sort(np.exp2(s_row[centres] - m))
        kept = u[p["trim_lo"]:p["strata"] - p["trim_hi"]]
        mass_r = (r / kept.shape[0]) * kept.sum()
    return float(m + math.log2(exact_mass + mass_r))


def estimate_level(q_bits, k_bits, *, num_kv_heads, page_size, sm_scale, seq_lens,
                   block_table=None, p: Dict[str, int] = EST_DEFAULT,
                   rows: Optional[Iterable[Tuple[int, int]]] = None) -> np.ndarray:
    """Z for every (request, head) row of a per-request view: ``[B, H]``."""
    q = bf16_bits_to_f64(q_bits)
    b, h, _ = q.shape
    group = h // num_kv_heads
    z = np.zeros((b, h))
    want = None if rows is None else set(rows)
    for r in range(b):
        n = int(seq_lens[r])
        for g in range(num_kv_heads):
            heads = [g * group + hh for hh in range(group)]
            if want is not None and not any((r, hh) in want for hh in heads):
                continue
            if n == 0:
                continue
            keys = gather(k_bits, r, g, n, block_table, page_size)
            s = scores(q[r, heads], keys, sm_scale)
            for a, hh in enumerate(heads):
                z[r, hh] = estimate_z(s[a], p)
    return z


# ---------------------------------------------------------------- O8 -------
def read_gates(live_rows: np.ndarray, n: int) -> Tuple[np.ndarray, np.ndarray]:
    """Key bits (OR over the read group's rows) and 16-key page bits."""
    key = live_rows.any(axis=0) if live_rows.shape[0] else np.zeros(n, dtype=bool)
    npg = (n + PAGE_GATE - 1) // PAGE_GATE
    pad = np.zeros(npg * PAGE_GATE, dtype=bool)
    pad[:n] = key
    return key, pad.reshape(npg, PAGE_GATE).any(axis=1)


# ---------------------------------------------------------------- O9 -------
def row_diagnostics(s_row: np.ndarray, z: float, T: float, values: np.ndarray) -> Dict[str, float]:
    """Per-row range and truncation figures.

    ``m`` (largest score), ``lse`` (base-2 log-sum-exp), ``headroom`` (lse - Z),
    ``prop1_lhs`` = m - Z + log2(n * nu) which Proposition 1(iii) requires to
    be below 127, ``w_cut`` (cut mass relative to Z), ``bound_T`` = the
    truncation bound (W_cut / L) * max over cut keys of |v|_inf, and
    ``live_frac``.
    """
    n = s_row.shape[0]
    m = float(s_row.max())
    lse = float(m + math.log2(np.exp2(s_row - m).sum()))
    nu = max(1.0, float(np.abs(values).max()))
    x = s_row - z
    live = live_mask(x, T)
    w = np.exp2(x)
    l = float(w.sum())
    cut = ~live
    w_cut = float(w[cut].sum())
    vmax_cut = float(np.abs(values[cut]).max()) if cut.any() else 0.0
    return {"m": m, "lse": lse, "headroom": lse - z, "prop1_lhs": m - z + math.log2(n * nu),
            "L": l, "w_cut": w_cut, "bound_T": (w_cut / l) * vmax_cut if l > 0 else 0.0,
            "live_frac": float(live.mean())}
