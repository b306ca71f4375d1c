"""FoldAttention decode step around the scan: a plain FP64 CPU oracle of the
token append, the certified decode (certificate rerun) and draft columns.

TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the
benchmark's CPU-baseline leg may import or call this module.  It imports
nothing from the product path and shares no code with it.

* S1  append (Section 4, "Weight-gated reads": the front appends the new
      token each step; paged cache with a per-request block table): token t
      of sequence r at position p lands in physical page
      ``block_table[r, p // P]``, slot ``p % P``, for every kv head.
* S2  certified decode (Section 3, certificate paragraph): a row whose
      ``L_i = 2^(l_i - Z_i)`` (``l_i`` its base-2 log-sum-exp) leaves
      ``[2^-1, 2^100]``, or whose output is not finite, is decoded again
      with ``Z_i = l_i``.  Where ``l_i`` is not finite (``L_i`` is 0 or
      infinite in the arithmetic that formed it) the reading moves ``Z_i``
      by ``STEP`` binades towards it; a row still flagged after
      ``max_reruns`` decodes keeps its flag.
* S3  drafts (Section 4, "Value product": speculative drafts and
      verification trees are extra query columns masked to their
      ancestors): request r holds ``n_r`` keys, the last ``m_r`` of them its
      draft tokens in column order; column c (draft c) sees the committed
      keys ``[0, n_r - m_r)`` and the keys of c and of its ancestors along
      ``parent`` (-1 ends the chain at the committed cache).

Parity: pinned by ``tests/test_oracle_step_pins.py`` (round trip through the
generator's logical cache, torch SDPA with an explicit boolean mask, chains
against truncated plain decodes, closed-form rerun counts).
"""

from __future__ import annotations

from typing import Callable, Sequence, Tuple

import numpy as np

from .fold_oracle import (CERT_HI, CERT_LO, bf16_bits_to_f64, fold, gather, live_mask,
                          scores)

STEP = 64.0  # binades per rerun when l_i is not finite (reading)


# ---------------------------------------------------------------- S1 -------
def append_tokens(cache_bits: np.ndarray, src_bits: np.ndarray, tok_seq: Sequence[int],
                  tok_pos: Sequence[int], block_table, page_size: int) -> np.ndarray:
    """A copy of ``cache_bits`` ``[pages, Hkv, P, D]`` (or contiguous
    ``[seqs, Hkv, max_len, D]`` when ``block_table`` is None) with token t's
    rows ``src_bits[t]`` ``[Hkv, D]`` stored at (``tok_seq[t]``,
    ``tok_pos[t]``).  A token whose sequence, position or page the view
    cannot address is skipped."""
    out = np.array(cache_bits, copy=True)
    for t, (r, p) in enumerate(zip(tok_seq, tok_pos)):
        r, p = int(r), int(p)
        if block_table is None:
            if 0 <= r < out.shape[0] and 0 <= p < out.shape[2]:
                out[r, :, p] = src_bits[t]
            continue
        bt = np.asarray(block_table)
        if not (0 <= r < bt.shape[0] and 0 <= p < bt.shape[1] * page_size):
            continue
        page = int(bt[r, p // page_size])
        if 0 <= page < out.shape[0]:
            out[page, :, p % page_size] = src_bits[t]
    return out


# ---------------------------------------------------------------- S2 -------
def certify(z: np.ndarray, l: np.ndarray, o: np.ndarray):
    """Per row: the base-2 log-sum-exp ``Z + log2 L``, the certificate bits
    (bit0 ``L < 2^-1``, bit1 ``L > 2^100``, bit2 a non-finite output) and
    the reference of the next decode (``l`` where finite, else ``Z`` moved
    ``STEP`` binades towards it; unflagged rows keep ``Z``)."""
    z = np.asarray(z, dtype=np.float64)
    with np.errstate(divide="ignore", invalid="ignore"):
        lse = z + np.log2(l)
    cert = ((l < CERT_LO).astype(np.uint8)
            | ((l > CERT_HI).astype(np.uint8) << 1)
            | ((~np.isfinite(o).all(axis=-1)).astype(np.uint8) << 2))
    nxt = np.where(np.isfinite(lse), lse,
                   np.where(l == 0, z - STEP, np.where(np.isinf(l), z + STEP, z)))
    return lse, cert, np.where(cert != 0, nxt, z)


def certified_decode(decode_fn: Callable[[np.ndarray], Tuple[np.ndarray, np.ndarray]],
                     z: np.ndarray, max_reruns: int = 8):
    """Decode, then decode again every flagged row with its new reference,
    at most ``max_reruns`` times.  ``decode_fn(z) -> (o [..., D], L [...])``.
    Returns ``(o, z_final, reruns, cert)``: the last output of every row, the
    reference it was decoded with, how many times the row was decoded again,
    and its final certificate bits."""
    z = np.asarray(z, dtype=np.float64).copy()
    o, l = decode_fn(z)
    _, cert, nxt = certify(z, l, o)
    reruns = np.zeros(z.shape, dtype=np.int64)
    for _ in range(max_reruns):
        flagged = cert != 0
        if not flagged.any():
            break
        z = nxt
        o2, l2 = decode_fn(z)
        o = np.where(flagged[..., None], o2, o)
        l = np.where(flagged, l2, l)
        reruns += flagged
        _, c2, n2 = certify(z, l, o)
        cert = np.where(flagged, c2, cert)
        nxt = np.where(flagged, n2, z)
    return o, z, reruns, cert


# ---------------------------------------------------------------- S3 -------
def draft_visible(n: int, m: int, parent: Sequence[int], c: int) -> np.ndarray:
    """Key positions column c of a request with n keys and m drafts sees:
    the committed keys, then its own and its ancestors' draft keys in
    position order."""
    anc = []
    t = c
    while t >= 0:
        anc.append(t)
        t = int(parent[t])
        if len(anc) > m:
            raise ValueError("parent links form a cycle")
    return np.concatenate([np.arange(n - m), (n - m) + np.array(sorted(anc))]).astype(np.int64)


def decode_drafts(q_bits, k_bits, v_bits, *, num_kv_heads: int, page_size: int,
                  sm_scale: float, seq_lens: Sequence[int], block_table,
                  col_indptr: Sequence[int], parent: Sequence[int], z: np.ndarray,
                  T: float):
    """Pairs ``(A [C, H, D], L [C, H])`` of draft columns: column c of
    request r folds the keys ``draft_visible`` names for it (Eq. fold with
    the depth rule), with its own references ``z[c]``; ``parent[c]`` is
    relative to the request's first column."""
    q = bf16_bits_to_f64(q_bits)
    cols, h, d = q.shape
    group = h // num_kv_heads
    part_a = np.zeros((cols, h, d))
    part_l = np.zeros((cols, h))
    for r, n in enumerate(seq_lens):
        c0, c1 = int(col_indptr[r]), int(col_indptr[r + 1])
        m = c1 - c0
        par = [int(p) for p in parent[c0:c1]]
        for g in range(num_kv_heads):
            keys = gather(k_bits, r, g, int(n), block_table, page_size)
            vals = gather(v_bits, r, g, int(n), block_table, page_size)
            for c in range(m):
                vis = draft_visible(int(n), m, par, c)
                heads = np.arange(g * group, (g + 1) * group)
                s = scores(q[c0 + c, heads], keys[vis], sm_scale)
                x = s - np.asarray(z, dtype=np.float64)[c0 + c, heads][:, None]
                a, l = fold(x, live_mask(x, T), vals[vis])
                part_a[c0 + c, heads] = a
                part_l[c0 + c, heads] = l
    return part_a, part_l
