"""Two-plane INT8 key cache: a plain, slow FP64 CPU oracle.

TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the
benchmark's CPU-baseline leg may import or call this module.  It imports
nothing from the product path.

What it computes (Section 4, "Cache format", "Weight-gated reads"; Algorithm 1
with BF16 values):

* Q1  rotation: keys and queries are multiplied by the Sylvester Hadamard
      matrix H_D (entries +-1, H H^T = D I).  The orthonormal rotation of the
      paper is H_D / sqrt(D); the factor 1/D of a rotated dot product is moved
      into the query scale, so every rotated coordinate is an exact FP64 sum
      of +-BF16 inputs.
* Q2  key split: k'' = e (a + b/256) with INT8 planes a, b and a BF16 scale e
      per key, e the smallest BF16 value >= max|k''| / 127 (rounded up, so
      plane A never saturates); a = rint(k''/e), b = rint(256 (k''/e - a))
      clamped to [-128, 127].  A key's code depends on that key alone.
* Q3  query split, the same way each step: q'' = f (qa + qb/256) with
      f = max|q''| / 127 and the base-2 score scale eta = log2(e) sm_scale f / D
      rounded once to FP32.
* Q4  coarse score against the fixed reference (plane A only):
      xc_ij = eta_i e_j (a_j . qa_i + (a_j . qb_i) / 256) - Z_i.
* Q5  gates, ORed over the GQA group of the row (the G rows of one request
      that share a kv head): live_j = OR [xc_ij >= -T] (T = inf: all live);
      refine_j = live_j AND OR [xc_ij >= -tau], where tau = kappa +
      ceil(log2 n_r) follows the request's own length n_r.
* Q6  refined score: x_ij = xc_ij + [refine_j] eta_i e_j (b_j . qa_i +
      (b_j . qb_i) / 256) / 256.
* Q7  fold: a key counts for row i iff x_ij >= -T (T = inf: always); w = 2^x;
      A_i = sum of live w v_j, L_i = sum of all w (cut keys keep their mass).
      Splits and combine are those of the BF16 path (64-key tiles, tile t to
      split t mod S, slots added in order).
* Q8  read bits: a value row is read iff live_j holds for some GQA group of
      the read group; a plane-B row iff refine_j does.
* Q9  stacked level (Appendix E, tile layouts: past 64 stacked rows the level
      runs laid out as prefill is, with one FP16 product per logit): each key's
      code rounded once to FP16, k^_j = fp16(e_j (a_j + b_j/256)) (the scale is
      folded in before that one rounding), each row's query codes rounded to
      FP16, q^_i = fp16(qa_i + qb_i/256), and s_ij = eta_i (k^_j . q^_i) in
      FP64 from those FP16 operands; then the depth rule and the fold of the
      BF16 path (no coarse pass and no refine gate: the product already holds
      both planes).

Parity status: Q9 is pinned by torch's FP16 rounding of the same exact
values, by the paper's stated logit bound (within about 2^-11 of |q||k| per
rounding), by library softmax over the FP16 operands and by additivity over
splits.  Q1-Q3 are pinned by closed forms (orthogonality, exact
rational sums, reconstruction bounds, minimality of the rounded-up scale);
Q4-Q7 by the dequantized dot product, by library softmax over the
dequantized operands, by the closed-form refine bound and by additivity over
splits; the estimator on coarse scores shares the BF16 estimator's pins and
its "parity unpinned" status for the stratified branch.
"""

from __future__ import annotations

import math
from typing import Dict, Iterable, Optional, Sequence, Tuple

import numpy as np

from .fold_oracle import (EST_DEFAULT, TILE, bf16_bits_to_f64, estimate_z, fold, gather,
                          live_mask, live_mask_imposed, read_gates, split_of_key)

LOG2E_F64 = float.fromhex("0x1.71547652b82fep+0")   # log2(e) rounded to FP64
QMAX = 127          # plane-A magnitude bound
B_LO, B_HI = -128, 127
FP32_MIN_NORMAL = 2.0 ** -126


# ---------------------------------------------------------------- Q1 -------
def hadamard(d: int) -> np.ndarray:
    """Sylvester Hadamard matrix of order d (a power of two), entries +-1."""
    if d < 1 or d & (d - 1):
        raise ValueError("order must be a power of two")
    h = np.ones((1, 1))
    while h.shape[0] < d:
        h = np.block([[h, h], [h, -h]])
    return h


def rotate(x: np.ndarray) -> np.ndarray:
    """``x @ H_D^T`` over the last axis, FP64 (H is symmetric)."""
    return x @ hadamard(x.shape[-1]).T


# ---------------------------------------------------------------- Q2 -------
def bf16_ceil(t: float) -> float:
    """Smallest BF16 value >= t for t > 0 (8 significant bits, rounded up)."""
    mant, ex = math.frexp(t)            # t = mant * 2^ex, mant in [0.5, 1)
    return math.ldexp(math.ceil(mant * 256.0), ex - 8)


def f64_to_bf16_bits(x: float) -> int:
    """Bits of a value already representable in BF16."""
    return int(np.array([x], dtype=np.float32).view(np.uint32)[0] >> 16)


def split_rows(rot: np.ndarray, scale: np.ndarray):
    """Planes of rows ``rot`` under per-row scales ``scale`` (0 = zero row)."""
    with np.errstate(divide="ignore", invalid="ignore"):
        x = np.where(scale[:, None] > 0, rot / scale[:, None], 0.0)
    a = np.rint(x)
    b = np.clip(np.rint(256.0 * (x - a)), B_LO, B_HI)
    return a.astype(np.int8), b.astype(np.int8)


def split_keys(k_bits: np.ndarray):
    """Key codes of BF16 keys ``[n, D]``: ``(a, b, e_bits)``.

    A key whose scale would fall below the smallest normal FP32 value is
    stored as zero (scale 0, planes 0).
    """
    rot = rotate(bf16_bits_to_f64(k_bits).reshape(-1, k_bits.shape[-1]))
    m = np.abs(rot).max(axis=1)
    e = np.zeros(rot.shape[0])
    for r in range(rot.shape[0]):
        if m[r] >= QMAX * FP32_MIN_NORMAL:
            e[r] = bf16_ceil(m[r] / QMAX)
    a, b = split_rows(rot, e)
    e_bits = np.array([f64_to_bf16_bits(v) for v in e], dtype=np.uint16)
    shape = k_bits.shape
    return a.reshape(shape), b.reshape(shape), e_bits.reshape(shape[:-1])


# ---------------------------------------------------------------- Q3 -------
def split_queries(q_bits: np.ndarray, sm_scale: float):
    """Query codes of BF16 queries ``[..., D]``: ``(qa, qb, eta_f32)``."""
    d = q_bits.shape[-1]
    rot = rotate(bf16_bits_to_f64(q_bits).reshape(-1, d))
    f = np.abs(rot).max(axis=1) / QMAX
    qa, qb = split_rows(rot, f)
    sm = float(np.float32(sm_scale))
    eta = np.array([np.float32(((LOG2E_F64 * sm) * fi) / d) for fi in f], dtype=np.float32)
    shape = q_bits.shape
    return qa.reshape(shape), qb.reshape(shape), eta.reshape(shape[:-1])


def refine_tau(n: int, kappa: float) -> np.float32:
    """Refine threshold of a request of n keys: kappa + ceil(log2 n), FP32."""
    c = (n - 1).bit_length() if n > 0 else 0
    return np.float32(float(np.float32(kappa)) + c)


def dequant(a: np.ndarray, b: np.ndarray, scale: np.ndarray) -> np.ndarray:
    """``scale (a + b / 256)`` in FP64 (the value a code stands for)."""
    return np.asarray(scale, dtype=np.float64)[..., None] * (a.astype(np.float64)
                                                             + b.astype(np.float64) / 256.0)


# ---------------------------------------------------------------- V1/V2 ----
# 8-bit values (Section 4, "Cache format"): two E4M3 planes under a power-of-
# two scale 2^e for the whole cache.  E4M3 here is the OCP "E4M3FN" format:
# sign, 4 exponent bits (bias 7), 3 mantissa bits, subnormals m 2^-9, largest
# finite 448, codes S.1111.111 are NaN and no infinity exists.
E4M3_MAX = 448.0


def e4m3_table() -> np.ndarray:
    """Value of each of the 256 codes (NaN for the two NaN codes)."""
    out = np.zeros(256)
    for c in range(256):
        sgn = -1.0 if c & 0x80 else 1.0
        ex, m = (c >> 3) & 15, c & 7
        if ex == 15 and m == 7:
            out[c] = np.nan
        elif ex == 0:
            out[c] = sgn * m * 2.0 ** -9
        else:
            out[c] = sgn * (1 + m / 8) * 2.0 ** (ex - 7)
    return out


_E4M3 = e4m3_table()
_POS_CODES = np.arange(0x7F)                      # 0 .. 0x7E: the finite non-negative codes
_POS_VALS = _E4M3[_POS_CODES]


def e4m3_encode(x: np.ndarray) -> np.ndarray:
    """Codes of x rounded to the nearest E4M3 value, ties to the even code
    (the one whose mantissa LSB is 0); magnitudes above 448 saturate to 448.
    Nearest-value search over the code table (FP64)."""
    x = np.asarray(x, dtype=np.float64)
    a = np.minimum(np.abs(x), E4M3_MAX)
    i = np.clip(np.searchsorted(_POS_VALS, a), 1, len(_POS_VALS) - 1)
    lo, hi = _POS_VALS[i - 1], _POS_VALS[i]
    pick_hi = (a - lo > hi - a) | ((a - lo == hi - a) & (_POS_CODES[i] % 2 == 0))
    code = np.where(pick_hi, _POS_CODES[i], _POS_CODES[i - 1])
    code = np.where(a == 0, 0, code)
    neg = (x < 0) & (code != 0)
    return (code | (neg.astype(np.int64) << 7)).astype(np.uint8)


def e4m3_decode(codes: np.ndarray) -> np.ndarray:
    return _E4M3[np.asarray(codes, dtype=np.int64)]


def split_values(v_bits: np.ndarray, scale_exp: int):
    """Value planes of BF16 value rows: y = v 2^-e, p = E4M3(y),
    r = E4M3(16 (y - p)); the value stands for 2^e (p + r/16)."""
    y = bf16_bits_to_f64(v_bits) * 2.0 ** -scale_exp
    p = e4m3_encode(y)
    r = e4m3_encode(16.0 * (y - e4m3_decode(p)))
    return p, r


def dequant_values(p: np.ndarray, r: np.ndarray, scale_exp: int, refined=True) -> np.ndarray:
    """2^e (p + [refined] r / 16), FP64."""
    v = e4m3_decode(p)
    if refined is not False:
        v = v + np.where(np.asarray(refined)[..., None] if np.ndim(refined) else refined,
                         e4m3_decode(r) / 16.0, 0.0)
    return v * 2.0 ** scale_exp


# ---------------------------------------------------------------- Q4/Q6 ----
def coarse_and_refine(qa, qb, eta, a, b, e):
    """``(coarse, refine)`` score terms [rows, keys], FP64, before the reference.

    coarse = eta e (a . qa + (a . qb) / 256);
    refine = eta e (b . qa + (b . qb) / 256) / 256.
    The integer dot products are exact in int64.
    """
    qa64, qb64 = qa.astype(np.int64), qb.astype(np.int64)
    a64, b64 = a.astype(np.int64), b.astype(np.int64)
    ee = np.asarray(eta, dtype=np.float64)[:, None] * np.asarray(e, dtype=np.float64)[None, :]
    caa, cab = (qa64 @ a64.T).astype(np.float64), (qb64 @ a64.T).astype(np.float64)
    cba, cbb = (qa64 @ b64.T).astype(np.float64), (qb64 @ b64.T).astype(np.float64)
    return ee * (caa + cab / 256.0), ee * (cba + cbb / 256.0) / 256.0


def gate_bits(xc: np.ndarray, blocks: np.ndarray, T: float, tau: np.ndarray,
              f32: bool = False):
    """Per-row views of the group bits ``(live, refine)`` [rows, keys].

    ``blocks[i]`` names row i's GQA group; ``tau[i]`` its request's refine
    threshold.  With ``f32`` the compares are FP32 on FP32 ``xc``.
    """
    if f32:
        xc = np.asarray(xc, dtype=np.float32)
        neg_t = np.float32(-T)
        neg_tau = (-np.asarray(tau, dtype=np.float32))[:, None]
    else:
        neg_t = -T
        neg_tau = -np.asarray(tau, dtype=np.float64)[:, None]
    row_live = np.ones(xc.shape, dtype=bool) if math.isinf(T) else xc >= neg_t
    row_ref = xc >= neg_tau
    live = np.zeros(xc.shape, dtype=bool)
    ref = np.zeros(xc.shape, dtype=bool)
    for blk in np.unique(blocks):
        sel = blocks == blk
        lv = row_live[sel].any(axis=0)
        live[sel] = lv
        ref[sel] = lv & row_ref[sel].any(axis=0)
    return live, ref


# ---------------------------------------------------------------- Q7 -------
def decode_level_q8(qa, qb, eta, planes, v_bits, *, num_kv_heads: int, page_size: int,
                    seq_lens: Sequence[int], block_table=None, row_indptr=None, row_req=None,
                    z: np.ndarray, T: float, tau: np.ndarray, num_splits: int,
                    imposed: Optional[Tuple[np.ndarray, np.ndarray]] = None,
                    chunks: Optional[Iterable[Tuple[int, int]]] = None,
                    want_scores: bool = False, with_cut: bool = False,
                    values8: Optional[Tuple[np.ndarray, np.ndarray, int]] = None,
                    tau_v: Optional[np.ndarray] = None):
    """Split partials of one level over a two-plane key cache.

    ``qa, qb`` [B, H, D] int8 and ``eta`` [B, H] FP32 are the query codes;
    ``planes = (a, b, e_bits)`` hold the cache in the layout of the BF16 path
    (int8 planes, BF16 scale bits); ``tau`` [B] FP32 is each request's refine
    threshold.  ``imposed = (xc_f32, x_f32)`` [B, H, max_len] replaces the
    FP64 decisions by FP32 decisions on those values: the group bits from the
    coarse scores, each row's own cut from the refined score.
    Returns ``part_A [S, B, H, D]``, ``part_L [S, B, H]``, with ``with_cut``
    also ``part_Lcut [S, B, H]`` (the cut keys' summed weights) and, with
    ``want_scores``, a dict ``(seq, g) -> (rows, xc, x, live, refine)``.

    ``values8 = (p, r, e)`` replaces the BF16 values by two E4M3 planes: key j
    contributes 2^e (p_j + [refine_v_j] r_j / 16), where refine_v_j = live_j
    AND OR over the GQA group of [xc_ij >= -tau_v] (``tau_v`` [B], Algorithm
    1's third verdict bit; imposed mode applies it in FP32 to the given xc).
    """
    pa_, pb_, pe_ = planes
    b_, h, d = qa.shape
    group = h // num_kv_heads
    part_a = np.zeros((num_splits, b_, h, d))
    part_l = np.zeros((num_splits, b_, h))
    part_c = np.zeros((num_splits, b_, h))
    info = {}
    if chunks is None:
        chunks = [(s, g) for s in range(len(seq_lens)) for g in range(num_kv_heads)]
    for seq, g in chunks:
        n = int(seq_lens[seq])
        reqs = [seq] if row_indptr is None else [int(r) for r in
                                                  row_req[row_indptr[seq]:row_indptr[seq + 1]]]
        if n == 0 or not reqs:
            continue
        ri = np.array([r for r in reqs for _ in range(group)])
        hi = np.array([g * group + hh for _ in reqs for hh in range(group)])
        blocks = np.repeat(np.arange(len(reqs)), group)
        a = _gather_raw(pa_, seq, g, n, block_table, page_size)
        bb = _gather_raw(pb_, seq, g, n, block_table, page_size)
        e = bf16_bits_to_f64(_gather_raw(pe_[..., None], seq, g, n, block_table,
                                         page_size)[:, 0])
        if values8 is None:
            vals = gather(v_bits, seq, g, n, block_table, page_size)
        else:
            vp = _gather_raw(values8[0], seq, g, n, block_table, page_size)
            vr = _gather_raw(values8[1], seq, g, n, block_table, page_size)
        coarse, refine = coarse_and_refine(qa[ri, hi], qb[ri, hi], eta[ri, hi], a, bb, e)
        xc = coarse - np.asarray(z, dtype=np.float64)[ri, hi][:, None]
        tau_rows = np.asarray(tau)[ri]
        if imposed is None:
            live, ref = gate_bits(xc, blocks, T, tau_rows)
            x = xc + np.where(ref, refine, 0.0)
            counts = np.ones(x.shape, dtype=bool) if math.isinf(T) else x >= -T
        else:
            ixc = imposed[0][ri, hi, :n]
            ix = imposed[1][ri, hi, :n]
            live, ref = gate_bits(ixc, blocks, T, tau_rows, f32=True)
            x = xc + np.where(ref, refine, 0.0)
            counts = (np.ones(x.shape, dtype=bool) if math.isinf(T)
                      else np.asarray(ix, dtype=np.float32) >= np.float32(-T))
        w = np.exp2(x)
        if values8 is not None:
            tv = np.asarray(tau_v)[ri]
            xsrc = xc if imposed is None else imposed[0][ri, hi, :n]
            _, ref_v = gate_bits(xsrc, blocks, T, tv, f32=imposed is not None)
            # per row its group's bit; one value row per key for every row of
            # a group, so rows of different groups may see different values
            v_rows = [dequant_values(vp, vr, values8[2], ref_v[k]) for k in range(len(ri))]
        owner = split_of_key(n, num_splits)
        for sp in range(num_splits):
            m = owner == sp
            if not m.any():
                continue
            if values8 is None:
                part_a[sp, ri, hi] = (w[:, m] * counts[:, m]) @ vals[m]
            else:
                part_a[sp, ri, hi] = np.stack([(w[k, m] * counts[k, m]) @ v_rows[k][m]
                                               for k in range(len(ri))])
            part_l[sp, ri, hi] = w[:, m].sum(axis=1)
            part_c[sp, ri, hi] = (w[:, m] * ~counts[:, m]).sum(axis=1)
        if want_scores:
            info[(seq, g)] = (list(zip(ri.tolist(), hi.tolist())), xc, x, live, ref)
    out = (part_a, part_l) + ((part_c,) if with_cut else ())
    if want_scores:
        return out + (info,)
    return out


# ---------------------------------------------------------------- Q9 -------
def stack_keys(a: np.ndarray, b: np.ndarray, e_bits: np.ndarray) -> np.ndarray:
    """The stacked level's FP16 keys ``fp16(e (a + b/256))`` of key codes
    ``[..., D]``: the product is exact in FP32 (a 16-bit code times an 8-bit
    scale), rounded once to FP16, nearest even."""
    e = bf16_bits_to_f64(e_bits)[..., None]
    exact = e * (a.astype(np.float64) + b.astype(np.float64) / 256.0)
    return exact.astype(np.float32).astype(np.float16)


def stack_queries(qa: np.ndarray, qb: np.ndarray) -> np.ndarray:
    """The stacked level's FP16 query operand ``fp16(qa + qb/256)`` (the sum is
    exact in FP32, then one rounding to FP16, nearest even)."""
    return (qa.astype(np.float32) + qb.astype(np.float32) / np.float32(256.0)).astype(np.float16)


def decode_level_q8_stacked(qhat, eta, khat, v_bits, *, num_kv_heads: int, page_size: int,
                            seq_lens: Sequence[int], block_table=None, row_indptr=None,
                            row_req=None, z: np.ndarray, T: float, num_splits: int,
                            imposed_x: Optional[np.ndarray] = None,
                            chunks: Optional[Iterable[Tuple[int, int]]] = None):
    """Split partials of a stacked level over the FP16 keys ``khat`` (the
    layout of the BF16 path's key cache): ``s_ij = eta_i (k^_j . q^_i)`` in
    FP64 from the FP16 operands, ``x = s - Z``, the depth rule (or the FP32
    rule on ``imposed_x`` [B, H, max_len]) and the fold, splits and slots of
    the BF16 path.  Returns ``part_A [S, B, H, D]``, ``part_L [S, B, H]``."""
    b_, h, d = qhat.shape
    group = h // num_kv_heads
    part_a = np.zeros((num_splits, b_, h, d))
    part_l = np.zeros((num_splits, b_, h))
    if chunks is None:
        chunks = [(s, g) for s in range(len(seq_lens)) for g in range(num_kv_heads)]
    for seq, g in chunks:
        n = int(seq_lens[seq])
        reqs = [seq] if row_indptr is None else [int(r) for r in
                                                  row_req[row_indptr[seq]:row_indptr[seq + 1]]]
        if n == 0 or not reqs:
            continue
        ri = np.array([r for r in reqs for _ in range(group)])
        hi = np.array([g * group + hh for _ in reqs for hh in range(group)])
        keys = _gather_raw(khat, seq, g, n, block_table, page_size).astype(np.float64)
        vals = gather(v_bits, seq, g, n, block_table, page_size)
        s = np.asarray(eta, dtype=np.float64)[ri, hi][:, None] * (
            qhat[ri, hi].astype(np.float64) @ keys.T)
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
            part_a[sp, ri, hi] = a
            part_l[sp, ri, hi] = l
    return part_a, part_l


def _gather_raw(arr: np.ndarray, seq: int, g: int, n: int, block_table, page_size: int):
    """Rows 0..n-1 of (seq, g) from a cache array, without conversion."""
    if block_table is None:
        return arr[seq, g, :n, :]
    j = np.arange(n)
    pages = np.asarray(block_table[seq])[j // page_size]
    return arr[pages, g, j % page_size, :]


def q8_read_gates(live: np.ndarray, ref: np.ndarray, n: int):
    """Value-row and plane-B read bits of a read group (OR over its rows)."""
    vkey, vpage = read_gates(live, n)
    bkey, _ = read_gates(ref, n)
    return vkey, vpage, bkey


# ---------------------------------------------------------------- estimate -
def estimate_level_q8(qa, qb, eta, planes, *, num_kv_heads, page_size, seq_lens,
                      block_table=None, p: Dict[str, int] = EST_DEFAULT,
                      rows: Optional[Iterable[Tuple[int, int]]] = None) -> np.ndarray:
    """Z per row from the coarse scores (the kernel's own coarse logits)."""
    pa_, pb_, pe_ = planes
    b_, h, _ = qa.shape
    group = h // num_kv_heads
    z = np.zeros((b_, h))
    want = None if rows is None else set(rows)
    for r in range(b_):
        n = int(seq_lens[r])
        for g in range(num_kv_heads):
            heads = [g * group + hh for hh in range(group)]
            if want is not None and not any((r, hh) in want for hh in heads):
                continue
            if n == 0:
                continue
            a = _gather_raw(pa_, r, g, n, block_table, page_size)
            bb = _gather_raw(pb_, r, g, n, block_table, page_size)
            e = bf16_bits_to_f64(_gather_raw(pe_[..., None], r, g, n, block_table,
                                             page_size)[:, 0])
            coarse, _ = coarse_and_refine(qa[r, heads], qb[r, heads], eta[r, heads], a, bb, e)
            for i, hh in enumerate(heads):
                z[r, hh] = estimate_z(coarse[i], p)
    return z


__all__ = ["E4M3_MAX", "LOG2E_F64", "TILE", "bf16_ceil", "coarse_and_refine", "decode_level_q8",
           "dequant", "dequant_values", "e4m3_decode", "e4m3_encode", "e4m3_table", "split_values",
           "estimate_level_q8", "gate_bits", "hadamard", "q8_read_gates", "refine_tau",
           "rotate", "split_keys", "split_queries"]
