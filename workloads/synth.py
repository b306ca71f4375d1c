"""Seeded BF16 decode workloads with the shapes of the paper's evaluation.

The paper measures on captured post-RoPE activations of real models
(Section 6.1), which are not available here. These synthetic workloads stand
in for them with the paper's shapes: head dims 64 and 128, GQA groups of 1,
4 and 8, 8-64 requests and 512 to 128K cached keys, a paged cache
(Section 4, paged cache with a per-request block table) and a shared-prefix
cascade (Section 4, value product paragraph; Appendix E).

Recipe (identical for every workload; the generator is a fresh
``torch.Generator`` on ``device`` seeded with ``seed``):

1. ragged lengths (if any) are drawn first;
2. queries ``q [B, H, D]``, then keys per request, then values per request,
   as FP32 ``randn`` rounded to BF16 (round to nearest even);
3. spike and sink indices per (request, kv head): sinks are keys
   ``0..n_sink-1``; spikes are distinct keys drawn uniformly from the
   non-sink indices;
4. a spike or sink adds ``alpha * sqrt(D) * u`` to the key in FP32 (from its
   BF16 value), then rounds to BF16 again, where ``u`` is the normalised sum
   of the group's query rows (for MHA, ``q_h / |q_h|``);
5. a random permutation maps (request, logical page) to a physical page.

Structured values (``values="structured"``, for the cut-key value models of
Section 4, "Depth as a dial"): the N(0,1) values of step 2 carry no
structure, so every value model sees zero-mean noise.  Real value caches
carry per-channel offsets and content that changes by stretches of the
text; this option imitates that.  After step 4 and before step 5, per
(request, kv head): a channel offset ``beta ~ 0.5 N(0,1)^D``; segment
lengths ``1 + floor(E)`` with ``E`` exponential of mean ``segment`` keys,
cut until the sequence is covered; one topic row ``tau ~ 0.5 N(0,1)^D`` per
segment; then ``v_j = beta + tau_seg(j) + 0.7 v_j`` in FP32 from the BF16
draw of step 2, rounded to BF16.

Nothing here computes attention scores, weights or references.
"""

from __future__ import annotations

import math
from dataclasses import dataclass, field
from typing import Dict, List, Optional, Tuple

import numpy as np
import torch

CONFIG_NAMES = {
    1: "tiny-mha-d64-512",
    2: "llama3-8b-gqa-16x8192-paged",
    3: "qwen3-8b-gqa-8x32768-paged-s16",
    4: "mha-stress-4x64k-128k-ragged-s32",
    5: "shared-prefix-cascade-64x(16384+1024)-g8",
}


@dataclass
class KVView:
    """One scan level's view of the shared cache.

    ``block_table`` is ``[num_seqs, max_pages]`` int32 (``None`` means the
    cache is contiguous ``[num_seqs, Hkv, max_seq_len, D]``).  ``row_indptr``
    and ``row_req`` list, per kv sequence, the requests whose query rows attend
    it (CSR); ``None`` means kv sequence ``r`` is attended by request ``r``.
    """

    block_table: Optional[torch.Tensor]
    seq_lens: torch.Tensor
    seq_lens_host: List[int]
    max_seq_len: int
    row_indptr: Optional[torch.Tensor] = None
    row_req: Optional[torch.Tensor] = None
    max_reqs_per_seq: int = 1

    @property
    def num_seqs(self) -> int:
        return int(self.seq_lens.shape[0])

    @property
    def max_pages(self) -> int:
        return 0 if self.block_table is None else int(self.block_table.shape[1])

    def to(self, device) -> "KVView":
        def mv(t):
            return None if t is None else t.to(device)

        return KVView(mv(self.block_table), mv(self.seq_lens), list(self.seq_lens_host),
                      self.max_seq_len, mv(self.row_indptr), mv(self.row_req),
                      self.max_reqs_per_seq)


@dataclass
class Workload:
    name: str
    q: torch.Tensor              # [B, H, D] bf16
    k: torch.Tensor              # paged [num_pages, Hkv, P, D] or contiguous [B, Hkv, n_max, D]
    v: torch.Tensor
    num_heads: int
    num_kv_heads: int
    head_dim: int
    page_size: int               # 0 for a contiguous cache
    sm_scale: float
    flat: KVView                 # per-request view (prefix ++ suffix for a cascade)
    levels: List[KVView]         # scan levels whose partials are added
    level_splits: List[int]      # default split count per level
    depths: List[float]
    meta: Dict = field(default_factory=dict)
    logical_k: Optional[torch.Tensor] = None  # [B, Hkv, n_max, D] (kept on request)
    logical_v: Optional[torch.Tensor] = None

    @property
    def batch(self) -> int:
        return int(self.q.shape[0])

    @property
    def group(self) -> int:
        return self.num_heads // self.num_kv_heads

    def to(self, device) -> "Workload":
        def mv(t):
            return None if t is None else t.to(device)

        return Workload(self.name, mv(self.q), mv(self.k), mv(self.v), self.num_heads,
                        self.num_kv_heads, self.head_dim, self.page_size, self.sm_scale,
                        self.flat.to(device), [lv.to(device) for lv in self.levels],
                        list(self.level_splits), list(self.depths), dict(self.meta),
                        mv(self.logical_k), mv(self.logical_v))

    def kv_bytes(self) -> int:
        """K+V bytes of every cached key of every level, once."""
        total = 0
        for lv in self.levels:
            total += sum(lv.seq_lens_host) * self.num_kv_heads * self.head_dim * 2 * 2
        return total


def host_bits(t: torch.Tensor) -> np.ndarray:
    """BF16 tensor -> numpy uint16 array of its bit patterns (host copy)."""
    assert t.dtype == torch.bfloat16
    return t.detach().contiguous().view(torch.int16).cpu().numpy().view(np.uint16)


def _bf16(x: torch.Tensor) -> torch.Tensor:
    return x.to(torch.bfloat16)


def _spike_keys(kh: torch.Tensor, idx: torch.Tensor, alpha: float, u: torch.Tensor, d: int):
    """kh [n, D] bf16; adds alpha*sqrt(D)*u to rows idx in FP32, rounds to BF16."""
    if idx.numel() == 0 or alpha == 0.0:
        return
    upd = kh[idx].float() + (alpha * math.sqrt(d)) * u[None, :]
    kh[idx] = _bf16(upd)


def _group_directions(q: torch.Tensor, hkv: int) -> torch.Tensor:
    """u[r, g] = normalised sum of the group's query rows, FP32 [B, Hkv, D]."""
    b, h, d = q.shape
    s = q.float().view(b, hkv, h // hkv, d).sum(dim=2)
    return s / s.norm(dim=-1, keepdim=True)


def _structure_values(v_log, lens, g, dev, segment):
    """Channel offset + per-segment topic rows + scaled noise (module recipe)."""
    batch, kv_heads, _, dim = v_log.shape
    for r in range(batch):
        n = lens[r]
        for kh in range(kv_heads):
            beta = 0.5 * torch.randn(dim, generator=g, device=dev)
            seg = torch.empty(n, dtype=torch.long, device=dev)
            pos, idx = 0, 0
            while pos < n:
                e = torch.empty(1, device=dev).exponential_(1.0 / segment, generator=g)
                ln = 1 + int(e.item())
                seg[pos:pos + ln] = idx
                pos += ln
                idx += 1
            tau = 0.5 * torch.randn(idx, dim, generator=g, device=dev)
            v = v_log[r, kh, :n].float()
            v_log[r, kh, :n] = _bf16(beta[None, :] + tau[seg] + 0.7 * v)


def _generate(*, name, batch, heads, kv_heads, dim, lens, paged, page_size, spike_count,
              alpha_spike, n_sink, alpha_sink, seed, device, level_splits, depths,
              keep_logical, draw_lens=None, values="normal", segment=256):
    dev = torch.device(device)
    g = torch.Generator(device=dev)
    g.manual_seed(seed)
    if draw_lens is not None:  # ragged lengths come first in the draw order
        lo, hi = draw_lens
        lens = torch.randint(lo, hi + 1, (batch,), generator=g, device=dev).cpu().tolist()
    lens = [int(x) for x in lens]
    n_max = max(lens)
    q = _bf16(torch.randn(batch, heads, dim, generator=g, device=dev))
    k_log = torch.empty(batch, kv_heads, n_max, dim, dtype=torch.bfloat16, device=dev)
    v_log = torch.empty_like(k_log)
    for r in range(batch):
        k_log[r] = _bf16(torch.randn(kv_heads, n_max, dim, generator=g, device=dev))
    for r in range(batch):
        v_log[r] = _bf16(torch.randn(kv_heads, n_max, dim, generator=g, device=dev))
    u = _group_directions(q, kv_heads)
    spikes = {}
    for r in range(batch):
        n = lens[r]
        ns = min(n_sink, n)
        cnt = spike_count(n)
        for kh in range(kv_heads):
            perm = torch.randperm(n - ns, generator=g, device=dev)[:cnt] + ns
            spikes[(r, kh)] = perm.cpu()
            _spike_keys(k_log[r, kh], perm, alpha_spike, u[r, kh], dim)
            if ns:
                _spike_keys(k_log[r, kh], torch.arange(ns, device=dev), alpha_sink, u[r, kh], dim)
    if values == "structured":
        _structure_values(v_log, lens, g, dev, segment)
    elif values != "normal":
        raise ValueError(f"values={values!r}: 'normal' or 'structured'")
    meta = {"spikes": spikes, "n_sink": n_sink, "alpha_spike": alpha_spike,
            "alpha_sink": alpha_sink, "seed": seed, "device": str(dev), "values": values}
    sl = torch.tensor(lens, dtype=torch.int32, device=dev)
    if not paged:
        view = KVView(None, sl, lens, n_max)
        wl = Workload(name, q, k_log, v_log, heads, kv_heads, dim, 0, 1.0 / math.sqrt(dim),
                      view, [view], level_splits, depths, meta)
        if keep_logical:
            wl.logical_k, wl.logical_v = k_log, v_log
        return wl
    npages = [(n + page_size - 1) // page_size for n in lens]
    total = sum(npages)
    perm = torch.randperm(total, generator=g, device=dev).to(torch.int32)
    maxp = max(npages)
    bt = torch.zeros(batch, maxp, dtype=torch.int32, device=dev)
    kp = torch.zeros(total, kv_heads, page_size, dim, dtype=torch.bfloat16, device=dev)
    vp = torch.zeros_like(kp)
    off = 0
    for r in range(batch):
        np_r, n = npages[r], lens[r]
        phys = perm[off:off + np_r]
        off += np_r
        bt[r, :np_r] = phys
        pad = np_r * page_size
        kr = torch.zeros(kv_heads, pad, dim, dtype=torch.bfloat16, device=dev)
        vr = torch.zeros_like(kr)
        kr[:, :n] = k_log[r, :, :n]
        vr[:, :n] = v_log[r, :, :n]
        kp[phys.long()] = kr.view(kv_heads, np_r, page_size, dim).transpose(0, 1)
        vp[phys.long()] = vr.view(kv_heads, np_r, page_size, dim).transpose(0, 1)
    view = KVView(bt, sl, lens, n_max)
    wl = Workload(name, q, kp, vp, heads, kv_heads, dim, page_size, 1.0 / math.sqrt(dim),
                  view, [view], level_splits, depths, meta)
    if keep_logical:
        wl.logical_k, wl.logical_v = k_log, v_log
    return wl


def _generate_cascade(*, name, requests, heads, kv_heads, dim, prefix_len, suffix_len,
                      page_size, seed, device, level_splits, depths, keep_logical):
    """Shared-prefix cascade: one prefix stored once plus one suffix per request."""
    dev = torch.device(device)
    g = torch.Generator(device=dev)
    g.manual_seed(seed)
    q = _bf16(torch.randn(requests, heads, dim, generator=g, device=dev))
    kpre = _bf16(torch.randn(kv_heads, prefix_len, dim, generator=g, device=dev))
    ksuf = _bf16(torch.randn(requests, kv_heads, suffix_len, dim, generator=g, device=dev))
    vpre = _bf16(torch.randn(kv_heads, prefix_len, dim, generator=g, device=dev))
    vsuf = _bf16(torch.randn(requests, kv_heads, suffix_len, dim, generator=g, device=dev))
    assert prefix_len % page_size == 0 and suffix_len % page_size == 0
    pp, ps = prefix_len // page_size, suffix_len // page_size
    total = pp + requests * ps
    perm = torch.randperm(total, generator=g, device=dev).to(torch.int32)
    kp = torch.zeros(total, kv_heads, page_size, dim, dtype=torch.bfloat16, device=dev)
    vp = torch.zeros_like(kp)
    pre_phys = perm[:pp]
    kp[pre_phys.long()] = kpre.view(kv_heads, pp, page_size, dim).transpose(0, 1)
    vp[pre_phys.long()] = vpre.view(kv_heads, pp, page_size, dim).transpose(0, 1)
    suf_bt = perm[pp:].view(requests, ps)
    for r in range(requests):
        ph = suf_bt[r].long()
        kp[ph] = ksuf[r].view(kv_heads, ps, page_size, dim).transpose(0, 1)
        vp[ph] = vsuf[r].view(kv_heads, ps, page_size, dim).transpose(0, 1)
    flat_bt = torch.cat([pre_phys[None, :].expand(requests, pp), suf_bt], dim=1).contiguous()
    n = prefix_len + suffix_len
    flat = KVView(flat_bt, torch.full((requests,), n, dtype=torch.int32, device=dev),
                  [n] * requests, n)
    prefix = KVView(pre_phys[None, :].contiguous(),
                    torch.tensor([prefix_len], dtype=torch.int32, device=dev), [prefix_len],
                    prefix_len,
                    torch.tensor([0, requests], dtype=torch.int32, device=dev),
                    torch.arange(requests, dtype=torch.int32, device=dev), requests)
    suffix = KVView(suf_bt.contiguous(),
                    torch.full((requests,), suffix_len, dtype=torch.int32, device=dev),
                    [suffix_len] * requests, suffix_len)
    meta = {"spikes": {}, "n_sink": 0, "seed": seed, "device": str(dev),
            "prefix_len": prefix_len, "suffix_len": suffix_len}
    wl = Workload(name, q, kp, vp, heads, kv_heads, dim, page_size, 1.0 / math.sqrt(dim),
                  flat, [prefix, suffix], level_splits, depths, meta)
    if keep_logical:
        wl.logical_k = torch.cat([kpre[None].expand(requests, -1, -1, -1), ksuf], dim=2)
        wl.logical_v = torch.cat([vpre[None].expand(requests, -1, -1, -1), vsuf], dim=2)
    return wl


INF = float("inf")


def make_config(i: int, seed: int = 0, device: str = "cpu", *, batch: Optional[int] = None,
                seq_len: Optional[int] = None, keep_logical: bool = False,
                values: str = "normal") -> Workload:
    """Workload ``i`` (1..5) at full size, or shrunk by ``batch`` / ``seq_len``.

    A shrunk workload keeps the structure (group size, spike density, sinks,
    paging) but is a different draw; it exists for CPU-sized tests.
    ``values="structured"`` (workloads 1-4) draws values with the structure
    described in the module recipe.
    """
    if values != "normal" and i == 5:
        raise ValueError("structured values are drawn for workloads 1-4")
    vx = {"values": values}
    if i == 1:
        n = seq_len or 512
        return _generate(name=CONFIG_NAMES[1], batch=batch or 1, heads=4, kv_heads=4, dim=64,
                         lens=[n] * (batch or 1), paged=False, page_size=0,
                         spike_count=lambda m: 8, alpha_spike=4.0, n_sink=0, alpha_sink=0.0,
                         seed=seed, device=device, level_splits=[1], depths=[INF, 16.0],
                         keep_logical=keep_logical, **vx)
    if i in (2, 3):
        n = seq_len or (8192 if i == 2 else 32768)
        b = batch or (16 if i == 2 else 8)
        return _generate(name=CONFIG_NAMES[i], batch=b, heads=32, kv_heads=8, dim=128,
                         lens=[n] * b, paged=True, page_size=16,
                         spike_count=lambda m: int(round(0.01 * m)), alpha_spike=3.0, n_sink=4,
                         alpha_sink=6.0, seed=seed, device=device,
                         level_splits=[4 if i == 2 else 16],
                         depths=[INF, 16.0] if i == 2 else [INF, 24.0, 16.0, 12.0],
                         keep_logical=keep_logical, **vx)
    if i == 4:
        b = batch or 4
        hi = seq_len or 131072
        lo = hi // 2
        return _generate(name=CONFIG_NAMES[4], batch=b, heads=32, kv_heads=32, dim=128,
                         lens=None, draw_lens=(lo, hi), paged=True, page_size=16,
                         spike_count=lambda m: int(round(0.005 * m)), alpha_spike=3.0, n_sink=0,
                         alpha_sink=0.0, seed=seed, device=device, level_splits=[32],
                         depths=[INF, 16.0], keep_logical=keep_logical, **vx)
    if i == 5:
        reqs = batch or 64
        pre = 16384 if seq_len is None else max(16, (seq_len // 16) * 16)
        return _generate_cascade(name=CONFIG_NAMES[5], requests=reqs, heads=8, kv_heads=1,
                                 dim=128, prefix_len=pre, suffix_len=1024 if seq_len is None
                                 else max(16, (seq_len // 256) * 16), page_size=16, seed=seed,
                                 device=device, level_splits=[32, 8], depths=[INF, 16.0],
                                 keep_logical=keep_logical)
    raise ValueError(f"no workload {i}")


def make_cascade(*, requests: int, heads: int, kv_heads: int, dim: int, prefix_len: int,
                 suffix_len: int, splits: Tuple[int, int] = (1, 1), seed: int = 0,
                 device: str = "cpu", keep_logical: bool = False) -> Workload:
    """A small shared-prefix cascade of any shape for tests (lengths multiples of 16)."""
    return _generate_cascade(name="custom-cascade", requests=requests, heads=heads,
                             kv_heads=kv_heads, dim=dim, prefix_len=prefix_len,
                             suffix_len=suffix_len, page_size=16, seed=seed, device=device,
                             level_splits=list(splits), depths=[INF, 16.0],
                             keep_logical=keep_logical)


def make_custom(*, batch: int, heads: int, kv_heads: int, dim: int, lens: List[int],
                paged: bool = True, page_size: int = 16, spike_count: int = 0,
                alpha_spike: float = 3.0, n_sink: int = 0, alpha_sink: float = 6.0,
                seed: int = 0, device: str = "cpu", keep_logical: bool = True,
                splits: int = 1, values: str = "normal", segment: int = 256) -> Workload:
    """A small workload of any shape (ragged lengths allowed) for tests."""
    return _generate(name="custom", batch=batch, heads=heads, kv_heads=kv_heads, dim=dim,
                     lens=list(lens), paged=paged, page_size=page_size,
                     spike_count=lambda m: min(spike_count, max(0, m - n_sink)),
                     alpha_spike=alpha_spike, n_sink=n_sink, alpha_sink=alpha_sink, seed=seed,
                     device=device, level_splits=[splits], depths=[INF, 16.0],
                     keep_logical=keep_logical, values=values, segment=segment)


@dataclass
class DraftWorkload:
    """Draft columns over a paged cache: request r holds ``committed[r]``
    committed keys followed by its ``m_r`` draft tokens' keys (in column
    order); ``q`` holds one query column per draft token; ``parent[c]`` is
    the parent column relative to the request's first column (-1: the
    committed cache); ``spare_pages [C][pages_per_col]`` are free pages of
    the pool reserved for each column."""
    wl: Workload                  # the cache (its q is unused), seq_lens = committed + m
    q: torch.Tensor               # [C, H, D] bf16
    col_indptr: torch.Tensor      # [B + 1] int32
    parent: torch.Tensor          # [C] int32
    spare_pages: torch.Tensor     # [C, pages_per_col] int32
    committed: List[int]

    @property
    def num_cols(self) -> int:
        return int(self.q.shape[0])


def chain_parents(m: int) -> List[int]:
    return [-1] + list(range(m - 1))


def make_drafts(*, committed: List[int], parents: List[List[int]], heads: int, kv_heads: int,
                dim: int, page_size: int = 16, spike_count: int = 0, n_sink: int = 0,
                seed: int = 0, device: str = "cpu") -> DraftWorkload:
    """A paged cache with draft tokens appended, one query column per draft
    (its request's query row plus N(0, 1/9) noise), and spare pages for each
    column (``ceil(max m / page_size)`` each)."""
    lens = [c + len(p) for c, p in zip(committed, parents)]
    wl = _generate(name="drafts", batch=len(lens), heads=heads, kv_heads=kv_heads, dim=dim,
                   lens=lens, paged=True, page_size=page_size,
                   spike_count=lambda m: min(spike_count, max(0, m - n_sink)),
                   alpha_spike=3.0, n_sink=n_sink, alpha_sink=6.0, seed=seed, device=device,
                   level_splits=[1], depths=[INF, 16.0], keep_logical=True)
    dev = torch.device(device)
    g = torch.Generator(device=dev)
    g.manual_seed(seed + 7919)
    cols = sum(len(p) for p in parents)
    # a column's query is its request's query plus noise of a third of its
    # scale: consecutive tokens' queries share the request's spike direction
    base = torch.cat([wl.q[r:r + 1].float().expand(len(p), -1, -1)
                      for r, p in enumerate(parents)]) if cols else wl.q[:0].float()
    noise = torch.randn(max(cols, 1), heads, dim, generator=g, device=dev)[:cols]
    q = _bf16(base + noise / 3.0)
    indptr = [0]
    for p in parents:
        indptr.append(indptr[-1] + len(p))
    ppc = max(1, (max((len(p) for p in parents), default=1) + page_size - 1) // page_size)
    n_pool = wl.k.shape[0]
    extra = cols * ppc
    pad = torch.zeros((extra,) + tuple(wl.k.shape[1:]), dtype=wl.k.dtype, device=dev)
    wl.k = torch.cat([wl.k, pad]).contiguous()
    wl.v = torch.cat([wl.v, pad]).contiguous()
    spare = (n_pool + torch.arange(extra, dtype=torch.int32, device=dev)).view(cols, ppc)
    flat_par = [x for p in parents for x in p]
    return DraftWorkload(wl, q, torch.tensor(indptr, dtype=torch.int32, device=dev),
                         torch.tensor(flat_par, dtype=torch.int32, device=dev), spare,
                         list(committed))
