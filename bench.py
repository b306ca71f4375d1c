"""Decode-attention benchmark on one MI355X.

A step is one pass of the whole decode hot path over one batch: the
reference estimate, the gated split-KV scan of every level, and the additive
combine.  The default workload is the Llama-3-8B-shaped GQA decode (batch 16,
32 query / 8 kv heads, head dim 128, 8192 cached keys per request, paged BF16
cache of 16-key pages).  Inputs are synthetic, seeded and resident in HBM
before timing.  Before every timed step a 1 GiB buffer is read, so that no
cache (4 MB L2 per XCD, 256 MB MALL) holds any of the step's data and no dirty
line is left to drain during the step; each step is bracketed by HIP events on
the stream the kernels are launched on.

Prints ONE JSON line (rank 0).  The line also carries the same workload over
a two-plane INT8 key cache (``q8_keys``; Section 4, cache format).  ``--all``
adds one JSON line per workload and depth on stderr (used for the design
notes' tables).
"""

from __future__ import annotations

import argparse
import json
import math
import os
import statistics
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBPS = 8000.0
METRIC = "decode-attn us/call + achieved HBM GB/s (% of peak) at T=16 and T=inf"


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--config", type=int, default=2)
    ap.add_argument("--all", action="store_true", help="also time workloads 1-5 (stderr)")
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle baseline")
    ap.add_argument("--no-q8", action="store_true",
                    help="skip the two-plane INT8 key legs (BF16 and 8-bit values)")
    ap.add_argument("--cpu-seconds", type=float, default=15.0)
    ap.add_argument("--splits", type=int, default=None, help="override the split count")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="end with one 1 GiB device copy (byte-counter calibration under rocprofv3)")
    return ap.parse_args()


class Path:
    """The decode path of one workload, bound to preallocated device buffers."""

    def __init__(self, wl, F, torch):
        self.wl, self.F, self.torch = wl, F, torch
        dev = wl.q.device
        self.levels = [F.kv_view(wl.k, wl.v, lv.seq_lens, num_kv_heads=wl.num_kv_heads,
                                 max_seq_len=lv.max_seq_len, block_table=lv.block_table,
                                 row_indptr=lv.row_indptr, row_req=lv.row_req,
                                 max_reqs_per_seq=lv.max_reqs_per_seq) for lv in wl.levels]
        self.flat = F.kv_view(wl.k, None, wl.flat.seq_lens, num_kv_heads=wl.num_kv_heads,
                              max_seq_len=wl.flat.max_seq_len, block_table=wl.flat.block_table)
        self.qv = F.q_view(wl.q)
        b, h, d = wl.q.shape
        self.splits = list(wl.level_splits)
        total = sum(self.splits)
        self.z = torch.empty(b, h, dtype=torch.float32, device=dev)
        self.part_A = torch.empty(total, b, h, d, dtype=torch.float32, device=dev)
        self.part_L = torch.empty(total, b, h, dtype=torch.float32, device=dev)
        self.out = torch.empty(b, h, d, dtype=torch.float32, device=dev)
        # one level over a per-request view with GQA groups of 2 to 8 rows: the
        # whole step also runs as one launch (fold_decode_fused, the same bits)
        lv = wl.levels[0]
        self.fusable = (len(wl.levels) == 1 and lv.row_indptr is None and 2 <= wl.group <= 8
                        and lv.num_seqs == b)
        self.arrivals = (torch.zeros(lv.num_seqs, wl.num_kv_heads, dtype=torch.int32, device=dev)
                         if self.fusable else None)

    def step(self, T, stream):
        """One whole call: the fused launch where it applies, else the three calls."""
        if self.fusable:
            self.fused(T, stream)
        else:
            self.three_calls(T, stream)

    def three_calls(self, T, stream):
        self.estimate(stream)
        self.decode(T, stream)
        self.combine(stream)

    def fused(self, T, stream):
        self.F.fold_decode_fused(self.levels[0], self.qv, self.wl.sm_scale, T, self.splits[0],
                                 self.part_A, self.part_L, self.arrivals, self.z, self.out,
                                 stream=stream)

    def estimate(self, stream):
        self.F.fold_ref_estimate(self.flat, self.qv, self.wl.sm_scale, self.z, stream=stream)

    def decode(self, T, stream):
        off = 0
        for kv, s in zip(self.levels, self.splits):
            self.F.fold_decode_split(kv, self.qv, self.wl.sm_scale, self.z, T, s, off,
                                     self.part_A, self.part_L, stream=stream)
            off += s

    def combine(self, stream):
        self.F.fold_combine(self.part_A, self.part_L, self.out, stream=stream)

    def read_fraction(self, T):
        """Fraction of (kv seq, kv head, key) value rows the scan reads at depth T
        (from the kernel's own read-gate export; untimed)."""
        torch, F = self.torch, self.F
        if math.isinf(T):
            return 1.0
        dev = self.wl.q.device
        read = total = 0
        off = 0
        b, h, d = self.wl.q.shape
        for lv, kv, s in zip(self.wl.levels, self.levels, self.splits):
            rg = F.fold_decode_row_groups(kv, self.qv)
            kg = torch.zeros(lv.num_seqs, self.wl.num_kv_heads, rg, lv.max_seq_len,
                             dtype=torch.uint8, device=dev)
            F.fold_decode_split(kv, self.qv, self.wl.sm_scale, self.z, T, s, off, self.part_A,
                                self.part_L, key_gate_out=kg)
            off += s
            read += int(kg.sum().item())
            total += sum(lv.seq_lens_host) * self.wl.num_kv_heads * rg
        return read / max(total, 1)


class Q8Path:
    """The same workload over a two-plane INT8 key cache, with BF16 values or
    (``values8``) two E4M3 value planes.

    The cache is written once by the cache writers (untimed set-up, as a
    prompt would be); a step is the query split, the reference estimate from
    coarse logits, every level's gated scan and the combine."""

    def __init__(self, wl, F, torch, kappa=-4.0, values8=False, kappa_v=-4.0):
        self.wl, self.F, self.torch, self.kappa = wl, F, torch, kappa
        self.kappa_v = kappa_v
        dev = wl.q.device
        n_pool, hkv, rows, d = wl.k.shape
        pool = F.kv_view(wl.k, None, torch.full((n_pool,), rows, dtype=torch.int32, device=dev),
                         num_kv_heads=hkv, max_seq_len=rows)
        self.keys = F.q8_empty_keys(wl.k)
        tok_seq = torch.arange(n_pool, dtype=torch.int32, device=dev).repeat_interleave(rows)
        tok_pos = torch.arange(rows, dtype=torch.int32, device=dev).repeat(n_pool)
        k_src = wl.k.permute(0, 2, 1, 3).reshape(n_pool * rows, hkv, d).contiguous()
        F.fold_q8_write_keys(pool, k_src, tok_seq, tok_pos, self.keys)
        del k_src
        self.vals = None
        if values8:
            vmax = float(wl.v.float().abs().max())
            e = int(math.ceil(math.log2(vmax / 448.0))) if vmax > 0 else 0
            self.vals = F.v8_empty_values(wl.v, e)
            v_src = wl.v.permute(0, 2, 1, 3).reshape(n_pool * rows, hkv, d).contiguous()
            F.fold_v8_write_values(pool, v_src, tok_seq, tok_pos, self.vals)
            del v_src
        del tok_seq, tok_pos
        # one appended token per request (the per-step append), for timing
        self.app_kv = F.kv_view(self.keys.plane_a, None, wl.flat.seq_lens,
                                num_kv_heads=hkv, max_seq_len=wl.flat.max_seq_len,
                                block_table=wl.flat.block_table, k_is_layout_only=True)
        b = wl.batch
        self.app_seq = torch.arange(b, dtype=torch.int32, device=dev)
        self.app_pos = (wl.flat.seq_lens - 1).to(torch.int32).contiguous()
        self.app_src = torch.randn(b, hkv, d, device=dev).to(torch.bfloat16)
        self.app_vsrc = torch.randn(b, hkv, d, device=dev).to(torch.bfloat16)
        self.levels = [F.kv_view(self.keys.plane_a, wl.v, lv.seq_lens,
                                 num_kv_heads=wl.num_kv_heads, max_seq_len=lv.max_seq_len,
                                 block_table=lv.block_table, row_indptr=lv.row_indptr,
                                 row_req=lv.row_req, max_reqs_per_seq=lv.max_reqs_per_seq,
                                 k_is_layout_only=True) for lv in wl.levels]
        self.flat = self.app_kv
        self.qq = F.q8_empty_query(wl.q)
        bq, h, d = wl.q.shape
        self.splits = list(wl.level_splits)
        total = sum(self.splits)
        self.z = torch.empty(bq, h, dtype=torch.float32, device=dev)
        self.part_A = torch.empty(total, bq, h, d, dtype=torch.float32, device=dev)
        self.part_L = torch.empty(total, bq, h, dtype=torch.float32, device=dev)
        self.out = torch.empty(bq, h, d, dtype=torch.float32, device=dev)
        torch.cuda.synchronize()

    def split(self, stream):
        self.F.fold_q8_split_query(self.wl.q, self.wl.sm_scale, self.qq,
                                   req_lens=self.wl.flat.seq_lens, kappa=self.kappa,
                                   kappa_v=self.kappa_v, stream=stream)

    def append(self, stream):
        self.F.fold_q8_write_keys(self.app_kv, self.app_src, self.app_seq, self.app_pos,
                                  self.keys, stream=stream)
        if self.vals is not None:
            self.F.fold_v8_write_values(self.app_kv, self.app_vsrc, self.app_seq, self.app_pos,
                                        self.vals, stream=stream)

    def estimate(self, stream):
        self.F.fold_q8_ref_estimate(self.flat, self.keys, self.qq, self.z, stream=stream)

    def fusable(self):
        lv = self.wl.levels[0]
        return (len(self.wl.levels) == 1 and lv.row_indptr is None and self.wl.group <= 8
                and lv.num_seqs == self.wl.batch)

    def fused(self, T, stream):
        """Front, scan and combine in one launch (fold_q8_decode_fused)."""
        if not hasattr(self, "arrivals"):
            self.arrivals = self.torch.zeros(self.wl.levels[0].num_seqs, self.wl.num_kv_heads,
                                             dtype=self.torch.int32, device=self.wl.q.device)
        self.F.fold_q8_decode_fused(self.levels[0], self.keys, self.wl.q, self.wl.sm_scale,
                                    self.qq, self.wl.flat.seq_lens, T, self.splits[0],
                                    self.part_A, self.part_L, self.arrivals, self.z, self.out,
                                    values=self.vals, kappa=self.kappa, kappa_v=self.kappa_v,
                                    stream=stream)

    def front(self, stream):
        """Query split and reference estimate in one launch (fold_q8_front)."""
        self.F.fold_q8_front(self.flat, self.keys, self.wl.q, self.wl.sm_scale, self.qq, self.z,
                             req_lens=self.wl.flat.seq_lens, kappa=self.kappa,
                             kappa_v=self.kappa_v, stream=stream)

    def decode(self, T, stream):
        off = 0
        for kv, s in zip(self.levels, self.splits):
            self.F.fold_q8_decode_split(kv, self.keys, self.qq, self.z, T, s, off, self.part_A,
                                        self.part_L, values=self.vals, stream=stream)
            off += s

    def combine(self, stream):
        self.F.fold_combine(self.part_A, self.part_L, self.out, stream=stream)

    def read_counts(self, T):
        """(value rows, plane-B rows, read-group key rows, second-value-plane
        rows) the scan reads at depth T, from its own read-bit exports
        (untimed)."""
        torch, F = self.torch, self.F
        dev = self.wl.q.device
        nv = nb = total = nr = 0
        off = 0
        for lv, kv, s in zip(self.wl.levels, self.levels, self.splits):
            rg = F.fold_q8_decode_row_groups(kv, self.qq)
            kg = torch.zeros(lv.num_seqs, self.wl.num_kv_heads, rg, lv.max_seq_len,
                             dtype=torch.uint8, device=dev)
            bg = torch.zeros_like(kg)
            ex = {}
            if self.vals is not None:
                ex["refine_v_gate_out"] = torch.zeros_like(kg)
            F.fold_q8_decode_split(kv, self.keys, self.qq, self.z, T, s, off, self.part_A,
                                   self.part_L, key_gate_out=kg, refine_gate_out=bg,
                                   values=self.vals, **ex)
            off += s
            nv += int(kg.sum().item())
            nb += int(bg.sum().item())
            if ex:
                nr += int(ex["refine_v_gate_out"].sum().item())
            total += sum(lv.seq_lens_host) * self.wl.num_kv_heads * rg
        return nv, nb, total, nr


def model_leg(path, wl, F, torch, flush, steps, warmup):
    """The cut-key value model on the benchmark workload at T=16: scan time with
    the cut masses written, and the output error against the dense output
    (exact softmax up to FP32 rounding) without and with the model."""
    dev = wl.q.device
    b, h, d = wl.q.shape
    fl = wl.flat
    kv = F.kv_view(wl.k, wl.v, fl.seq_lens, num_kv_heads=wl.num_kv_heads,
                   max_seq_len=fl.max_seq_len, block_table=fl.block_table)
    mean = torch.empty(fl.num_seqs, wl.num_kv_heads, d, dtype=torch.float32, device=dev)
    stream = torch.cuda.current_stream()
    path.estimate(stream)
    F.fold_value_mean(kv, mean)
    part_C = torch.empty_like(path.part_L)

    def decode_cut(stream):
        off = 0
        for kvl, s in zip(path.levels, path.splits):
            F.fold_decode_split(kvl, path.qv, wl.sm_scale, path.z, 16.0, s, off, path.part_A,
                                path.part_L, part_Lcut=part_C, stream=stream)
            off += s

    ts = []
    for it in range(warmup + steps):
        evict_caches(flush)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        decode_cut(stream)
        e1.record(stream)
        if it >= warmup:
            e1.synchronize()
            ts.append(e0.elapsed_time(e1))
    dense = torch.empty(b, h, d, dtype=torch.float32, device=dev)
    path.decode(math.inf, stream)
    F.fold_combine(path.part_A, path.part_L, dense, stream=stream)
    plain = torch.empty_like(dense)
    path.decode(16.0, stream)
    F.fold_combine(path.part_A, path.part_L, plain, stream=stream)
    model = torch.empty_like(dense)
    decode_cut(stream)
    F.fold_combine(path.part_A, path.part_L, model, part_Lcut=part_C, mean=mean, stream=stream)
    torch.cuda.synchronize()
    scale = dense.abs().amax(dim=-1).clamp_min(1e-30)

    def err(o):
        return float(((o - dense).abs().amax(dim=-1) / scale).max())

    def l2(o):
        return float((o - dense).norm() / dense.norm())

    return {"T": 16.0, "model": "request mean (cut keys carry their request's mean value row)",
            "decode_us_with_cut_masses": round(statistics.median(ts) * 1e3, 2),
            "max_row_err_vs_dense": {"no_model": err(plain), "request_mean": err(model)},
            "rel_l2_vs_dense": {"no_model": l2(plain), "request_mean": l2(model)}}


def q8_bytes(wl, nv, nb, nr=None):
    """Algorithmic bytes of one two-plane scan (all levels): plane A and the
    scale of every key, plane B of the nb refined rows, the nv value rows
    (BF16, or with ``nr`` the first E4M3 plane of nv rows and the second of
    nr), the query codes, eta, tau, references, block-table entries and
    partials."""
    d = wl.head_dim
    b, h, _ = wl.q.shape
    keys = sum(sum(lv.seq_lens_host) for lv in wl.levels) * wl.num_kv_heads
    total = keys * (d + 2) + nb * d + (nv * 2 * d if nr is None else (nv + nr) * d)
    total += 2 * b * h * d + 4 * b * h + 4 * b + 4 * b * h
    if wl.page_size:
        total += 4 * sum(sum((n + wl.page_size - 1) // wl.page_size for n in lv.seq_lens_host)
                         for lv in wl.levels)
    total += 4 * sum(wl.level_splits) * b * h * (d + 1)
    return total, keys


def time_q8(qp, T, steps, warmup, flush, torch):
    """Median per-kernel and per-step durations (ms) of the two-plane step
    (the step timed on its own, as in time_variant).  The step is the fused
    front (query split + estimate in one launch), the scan and the combine;
    ``split_then_est`` times the same step with the split and the estimate
    as two launches."""
    stream = torch.cuda.current_stream()
    res = {"front": [], "dec": [], "comb": [], "step": [], "append": [], "split_then_est": [],
           "fused": []}
    for it in range(warmup + steps):
        evict_caches(flush)
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(5)]
        ev[0].record(stream)
        qp.front(stream)
        ev[1].record(stream)
        qp.decode(T, stream)
        ev[2].record(stream)
        qp.combine(stream)
        ev[3].record(stream)
        qp.append(stream)
        ev[4].record(stream)
        if it >= warmup:
            ev[4].synchronize()
            res["front"].append(ev[0].elapsed_time(ev[1]))
            res["dec"].append(ev[1].elapsed_time(ev[2]))
            res["comb"].append(ev[2].elapsed_time(ev[3]))
            res["append"].append(ev[3].elapsed_time(ev[4]))
    one = qp.fusable()
    for it in range(warmup + steps):
        for key in ("step", "split_then_est") + (("fused",) if one else ()):
            evict_caches(flush)
            e0 = torch.cuda.Event(enable_timing=True)
            e1 = torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            if key == "fused":
                qp.fused(T, stream)
            else:
                if key == "step":
                    qp.front(stream)
                else:
                    qp.split(stream)
                    qp.estimate(stream)
                qp.decode(T, stream)
                qp.combine(stream)
            e1.record(stream)
            if it >= warmup:
                e1.synchronize()
                res[key].append(e0.elapsed_time(e1))
    if not one:
        del res["fused"]
    return {k: statistics.median(v) for k, v in res.items()}


def q8_leg(wl, F, torch, flush, steps, warmup, name=None, values8=False):
    """Timings of the two-plane key path (with ``values8``, also 8-bit values)
    on the benchmark workload."""
    qp = Q8Path(wl, F, torch, values8=values8)
    stream = torch.cuda.current_stream()
    qp.front(stream)
    out = {"kappa": qp.kappa,
           "cache": "two INT8 key planes + BF16 scale per key; " +
                    ("two E4M3 value planes, scale 2^%d" % qp.vals.scale_exp if values8
                     else "BF16 values"),
           "step": "front (query split + estimate from coarse logits, one launch) + split "
                   "scan + combine; the one-token append is timed apart; breakdown `fused`: "
                   "the same call as one launch (fold_q8_decode_fused), slower here"}
    if values8:
        out["kappa_v"] = qp.kappa_v
    for T in (math.inf, 16.0):
        nv, nb, total, nr = qp.read_counts(T)
        med = time_q8(qp, T, steps, warmup, flush, torch)
        nbytes, keys = q8_bytes(wl, nv, nb, nr if values8 else None)
        key = "T=inf" if math.isinf(T) else f"T={T:g}"
        out[key] = {"us_per_call": round(med["step"] * 1e3, 2),
                    "decode_us": round(med["dec"] * 1e3, 2),
                    "decode_bytes": int(nbytes),
                    "decode_gbps": round(nbytes / (med["dec"] * 1e-3) / 1e9, 1),
                    "bytes_per_key": round(nbytes / keys, 1),
                    "value_read_fraction": round(nv / max(total, 1), 5),
                    "refined_fraction": round(nb / max(total, 1), 5),
                    "breakdown_us": {k: round(v * 1e3, 2) for k, v in med.items()}}
        if values8:
            out[key]["refined_v_fraction"] = round(nr / max(total, 1), 5)
        if math.isinf(T):
            ach = nbytes / (med["dec"] * 1e-3) / 1e9
            tag = " [8-bit values]" if values8 else " [two-plane keys]"
            traffic = None if name is None else counter_traffic(name + tag)[0]
            out["roofline"] = {"bound": "hbm", "achieved": round(ach, 1), "peak": HBM_PEAK_GBPS,
                               "unit": "GB/s", "frac": round(ach / HBM_PEAK_GBPS, 4),
                               "traffic": None if traffic is None else int(traffic),
                               "kernel": "decode_q8_kernel (dense%s)"
                                         % (", 8-bit values" if values8 else "")}
    del qp
    torch.cuda.empty_cache()
    return out


def kv_bytes(wl, lam):
    """Algorithmic bytes of one decode scan (all levels): every key row, the
    value rows the read gates keep (fraction lam of read-group key rows), the
    query rows, references, block-table entries and partials written."""
    d = wl.head_dim
    b, h, _ = wl.q.shape
    keys = sum(sum(lv.seq_lens_host) for lv in wl.levels) * wl.num_kv_heads
    total = keys * 2 * d + lam * keys * 2 * d
    total += 2 * b * h * d + 4 * b * h
    if wl.page_size:
        total += 4 * sum(sum((n + wl.page_size - 1) // wl.page_size for n in lv.seq_lens_host)
                         for lv in wl.levels)
    total += 4 * sum(wl.level_splits) * b * h * (d + 1)
    return total, keys


class DraftPath:
    """Draft verification: ``requests`` requests of ``committed`` keys with a
    chain of ``m`` drafts each, one query column per draft (Llama-3-8B GQA
    heads).  A step is the per-column estimate, the committed level (every
    committed key read once for all of a request's columns), the ancestor
    level and the combine; the plan and the row gather run once (they
    belong to the append).  The baseline decodes every column as a request
    of its own (its committed keys plus its chain), reading the committed
    keys once per column."""

    def __init__(self, F, torch, requests=32, committed=4096, m=4, splits=4):
        from workloads import chain_parents, make_drafts
        self.F, self.torch = F, torch
        dw = make_drafts(committed=[committed] * requests, parents=[chain_parents(m)] * requests,
                         heads=32, kv_heads=8, dim=128, spike_count=committed // 100, n_sink=4,
                         seed=1, device="cuda")
        self.dw, wl = dw, dw.wl
        fl = wl.flat
        self.dv = F.fold_draft_views(wl.k, wl.v, fl.block_table, fl.seq_lens_host,
                                     dw.col_indptr.cpu().tolist(), dw.parent.cpu().tolist(),
                                     dw.spare_pages, num_kv_heads=8)
        c = dw.num_cols
        self.splits = [splits, 1]
        self.z = torch.empty(c, 32, dtype=torch.float32, device="cuda")
        self.pa = torch.empty(splits + 1, c, 32, 128, dtype=torch.float32, device="cuda")
        self.pl = torch.empty(splits + 1, c, 32, dtype=torch.float32, device="cuda")
        self.out = torch.empty(c, 32, 128, dtype=torch.float32, device="cuda")
        self.qv = F.q_view(dw.q)
        # baseline: column c of a chain is its request truncated at n0 + c + 1 keys
        col_req = self.dv.keep[1]
        lens = torch.tensor([committed + (i % m) + 1 for i in range(c)], dtype=torch.int32,
                            device="cuda")
        self.base_kv = F.kv_view(wl.k, wl.v, lens, num_kv_heads=8, max_seq_len=committed + m,
                                 block_table=fl.block_table.index_select(0, col_req.long()))
        self.base_pa = torch.empty(splits, c, 32, 128, dtype=torch.float32, device="cuda")
        self.base_pl = torch.empty(splits, c, 32, dtype=torch.float32, device="cuda")
        self.base_z = torch.empty(c, 32, dtype=torch.float32, device="cuda")
        self.keys = requests * committed * 8
        torch.cuda.synchronize()

    def step(self, T, stream):
        F = self.F
        F.fold_ref_estimate(self.dv.estimate, self.qv, self.dw.wl.sm_scale, self.z, stream=stream)
        F.fold_decode_split(self.dv.committed, self.qv, self.dw.wl.sm_scale, self.z, T,
                            self.splits[0], 0, self.pa, self.pl, stream=stream)
        F.fold_decode_split(self.dv.ancestors, self.qv, self.dw.wl.sm_scale, self.z, T, 1,
                            self.splits[0], self.pa, self.pl, stream=stream)
        F.fold_combine(self.pa, self.pl, self.out, stream=stream)

    def baseline(self, T, stream):
        F = self.F
        F.fold_ref_estimate(self.base_kv, self.qv, self.dw.wl.sm_scale, self.base_z,
                            stream=stream)
        F.fold_decode_split(self.base_kv, self.qv, self.dw.wl.sm_scale, self.base_z, T,
                            self.splits[0], 0, self.base_pa, self.base_pl, stream=stream)
        F.fold_combine(self.base_pa, self.base_pl, self.out, stream=stream)


def drafts_leg(F, torch, flush, steps, warmup):
    """Draft verification timings (chains of 2 and 4 drafts, 32 requests of
    4096 committed keys)."""
    out = {"workload": "32 requests x 4096 committed keys, GQA 32/8, D=128, chains of drafts",
           "step": "estimate + committed level + ancestor level + combine",
           "baseline": "every column decoded as its own request (estimate + scan + combine)"}
    stream = torch.cuda.current_stream()
    for m in (2, 4):
        dp = DraftPath(F, torch, m=m)
        rec = {}
        for T in (math.inf, 16.0):
            times = {"drafts": [], "per_column": []}
            for it in range(warmup + steps):
                for name, fn in (("drafts", dp.step), ("per_column", dp.baseline)):
                    evict_caches(flush)
                    e0 = torch.cuda.Event(enable_timing=True)
                    e1 = torch.cuda.Event(enable_timing=True)
                    e0.record(stream)
                    fn(T, stream)
                    e1.record(stream)
                    if it >= warmup:
                        e1.synchronize()
                        times[name].append(e0.elapsed_time(e1))
            med = {k: statistics.median(v) for k, v in times.items()}
            rec["T=inf" if math.isinf(T) else f"T={T:g}"] = {
                "drafts_us": round(med["drafts"] * 1e3, 2),
                "per_column_us": round(med["per_column"] * 1e3, 2),
                "speedup": round(med["per_column"] / med["drafts"], 3)}
        out[f"chain{m}"] = rec
        del dp
        torch.cuda.empty_cache()
    return out


def progress(msg):
    """One line on stderr as each leg ends (long runs under a profiler stay
    visibly alive)."""
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def fused_bytes(wl, lam):
    """Algorithmic bytes of one fused launch: the scan's (kv_bytes), the
    estimate's sampled key rows and their block-table entries (once per
    (request, kv head)), the combine's read of the slots and its output, and
    the arrival counts (read-modify-write and reset)."""
    d = wl.head_dim
    b, h, _ = wl.q.shape
    total, keys = kv_bytes(wl, lam)
    full = 1 + 63 + 128  # default sample: sink, recent keys, strata
    samples = sum(min(n, full) for n in wl.flat.seq_lens_host) * wl.num_kv_heads
    total += samples * 2 * d + (4 * samples if wl.page_size else 0)
    total += 4 * sum(wl.level_splits) * b * h * (d + 1) + 4 * b * h * d
    total += 2 * 4 * wl.flat.num_seqs * wl.num_kv_heads
    return total, keys


def scan_kernel_name(wl):
    """The scan kernel the library launches for a single-level workload."""
    if wl.group == 1:
        return "decode_split_kernel"
    return "decode_packed_kernel" if wl.group <= 8 else "decode_mfma_kernel"


def evict_caches(flush):
    """Read (not write) a 1 GiB buffer: every cache line of the step's data is
    evicted, and no dirty line is left to be written back during the step."""
    return flush.sum(dtype=flush.dtype)


def time_variant(path, T, steps, warmup, flush, torch):
    """Median per-kernel and per-step durations (ms) with a cache eviction
    before every step; events are recorded on the launch stream.

    The step is timed on its own, with events only before and after it: an
    event recorded between two kernels adds a queue marker that lengthens the
    step (by about 3.5 us each on MI355X).  The per-kernel breakdown comes
    from separate steps with events between the kernels; its parts add up to
    more than the step."""
    stream = torch.cuda.current_stream()
    res = {"est": [], "dec": [], "comb": [], "step": [], "step_three_calls": [],
           "step_with_markers": []}
    for it in range(warmup + steps):
        evict_caches(flush)
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(4)]
        ev[0].record(stream)
        path.estimate(stream)
        ev[1].record(stream)
        path.decode(T, stream)
        ev[2].record(stream)
        path.combine(stream)
        ev[3].record(stream)
        if it >= warmup:
            ev[3].synchronize()
            res["est"].append(ev[0].elapsed_time(ev[1]))
            res["dec"].append(ev[1].elapsed_time(ev[2]))
            res["comb"].append(ev[2].elapsed_time(ev[3]))
            res["step_with_markers"].append(ev[0].elapsed_time(ev[3]))
    for it in range(warmup + steps):
        for key, fn in (("step_three_calls", path.three_calls), ("step", path.step)):
            if key == "step" and not path.fusable:
                continue
            evict_caches(flush)
            e0 = torch.cuda.Event(enable_timing=True)
            e1 = torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            fn(T, stream)
            e1.record(stream)
            if it >= warmup:
                e1.synchronize()
                res[key].append(e0.elapsed_time(e1))
    if not path.fusable:
        res["step"] = res["step_three_calls"]
    torch.cuda.synchronize()
    return {k: statistics.median(v) for k, v in res.items()}, res


def time_graph(path, T, steps, warmup, flush, torch):
    """Median duration (ms) of one whole step replayed as a captured HIP graph
    (the fused launch, or the estimate, every level's scan and the combine),
    caches evicted before each replay."""
    stream = torch.cuda.current_stream()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        path.step(T, torch.cuda.current_stream())
    ts = []
    for it in range(warmup + steps):
        evict_caches(flush)
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        g.replay()
        e1.record(stream)
        if it >= warmup:
            e1.synchronize()
            ts.append(e0.elapsed_time(e1))
    torch.cuda.synchronize()
    return statistics.median(ts)


def kernel_sources_sha():
    """SHA-256 over the HIP sources of the library (identifies the kernels)."""
    import glob
    import hashlib

    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2609_33410_amd", "csrc")
    for f in sorted(glob.glob(os.path.join(csrc, "*"))):
        with open(f, "rb") as fh:
            h.update(os.path.basename(f).encode() + b"\0" + fh.read())
    return h.hexdigest()


def counter_traffic(workload_name):
    """HBM bytes per dense decode launch from the committed counter summary,
    or None when it is absent or was taken on other kernel sources."""
    path = os.path.join(ROOT, "profiles", "decode_traffic_counters.txt")
    if not os.path.exists(path):
        return None, None
    rec = {}
    with open(path) as f:
        for line in f:
            if line.startswith("record:"):
                r = json.loads(line[len("record:"):])
                rec[r["workload"]] = r
    r = rec.get(workload_name)
    if r is None or r.get("source_sha256") != kernel_sources_sha():
        return None, r
    kib = r["fetch_kib"] * r["fetch_scale"] + r["write_kib"] * r["write_scale"]
    return kib * 1024.0, r


def cpu_baseline(wl, budget_s):
    """The FP64 oracle timed on this host on a bounded sample of the workload's
    (kv sequence, kv head) chunks; scaled to one whole call."""
    import numpy as np

    import oracle
    from workloads import host_bits

    try:
        from threadpoolctl import threadpool_info
        threads = max([p.get("num_threads", 1) for p in threadpool_info()] or [1])
    except Exception:  # pragma: no cover
        threads = 1
    cores = len(os.sched_getaffinity(0))
    q_bits, k_bits, v_bits = host_bits(wl.q), host_bits(wl.k), host_bits(wl.v)
    lv = wl.levels[0]
    bt = None if lv.block_table is None else lv.block_table.cpu().numpy()
    z = np.zeros((wl.batch, wl.num_heads))
    chunks_all = [(s, g) for s in range(lv.num_seqs) for g in range(wl.num_kv_heads)]
    done = 0
    t0 = time.perf_counter()
    while True:  # whole calls (or a prefix of one) until the time budget is used
        for c in chunks_all:
            oracle.decode_level(q_bits, k_bits, v_bits, num_kv_heads=wl.num_kv_heads,
                                page_size=wl.page_size, sm_scale=wl.sm_scale,
                                seq_lens=lv.seq_lens_host, block_table=bt, z=z, T=math.inf,
                                num_splits=wl.level_splits[0], chunks=[c])
            done += 1
            if time.perf_counter() - t0 > budget_s:
                break
        if time.perf_counter() - t0 > budget_s:
            break
    dt = time.perf_counter() - t0
    per_call_s = dt * len(chunks_all) / done
    keys = sum(lv.seq_lens_host) * wl.num_kv_heads
    return {"value": round(per_call_s * 1e6, 1), "unit": "us/call", "cores": threads,
            "host_cores_visible": cores, "kind": "oracle",
            "keys_per_s": round(keys / per_call_s, 1),
            "sample": f"FP64 oracle decode (T=inf, gather + scores + fold + splits) of "
                      f"{done} (request, kv head) chunks = {done / len(chunks_all):.2f} whole "
                      f"calls in {dt:.1f} s, scaled to one call"}


def paired_depths(path, steps, warmup, flush, torch, T_cut=16.0):
    """Paired rounds: each round times one T=inf step and one T=T_cut step
    (order alternating by round, caches evicted before each); returns the
    medians of the per-round ratios (step and scan) and p10/p90 of the
    steps (ms)."""
    stream = torch.cuda.current_stream()
    ratios_step, ratios_dec = [], []
    steps_inf, steps_cut = [], []
    for it in range(warmup + steps):
        t = {}
        order = (math.inf, T_cut) if it % 2 == 0 else (T_cut, math.inf)
        for T in order:
            evict_caches(flush)
            ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
            ev[0].record(stream)
            path.step(T, stream)
            ev[1].record(stream)
            evict_caches(flush)
            ed = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
            ed[0].record(stream)
            path.decode(T, stream)
            ed[1].record(stream)
            ed[1].synchronize()
            t[T] = (ev[0].elapsed_time(ev[1]), ed[0].elapsed_time(ed[1]))
        if it >= warmup:
            ratios_step.append(t[math.inf][0] / t[T_cut][0])
            ratios_dec.append(t[math.inf][1] / t[T_cut][1])
            steps_inf.append(t[math.inf][0])
            steps_cut.append(t[T_cut][0])

    def pct(v, q):
        v = sorted(v)
        return v[min(len(v) - 1, max(0, int(round(q * (len(v) - 1)))))]

    return {"rounds": steps, "T": T_cut,
            "speedup_step_median": round(statistics.median(ratios_step), 3),
            "speedup_decode_median": round(statistics.median(ratios_dec), 3),
            "step_us_inf_p10_p50_p90": [round(pct(steps_inf, q) * 1e3, 2) for q in (0.1, 0.5, 0.9)],
            "step_us_T_p10_p50_p90": [round(pct(steps_cut, q) * 1e3, 2) for q in (0.1, 0.5, 0.9)]}


def run_workload(i, args, torch, F, make_config, flush, steps, warmup, splits=None):
    wl = make_config(i, device="cuda")
    if splits is not None and len(wl.level_splits) == 1:
        wl.level_splits = [splits]
    path = Path(wl, F, torch)
    stream = torch.cuda.current_stream()
    path.estimate(stream)
    out = {}
    for T in (math.inf, 16.0) + ((24.0, 12.0) if i == 3 else ()):
        lam = path.read_fraction(T)
        med, _ = time_variant(path, T, steps, warmup, flush, torch)
        graph_ms = time_graph(path, T, steps, warmup, flush, torch)
        nbytes, keys = kv_bytes(wl, lam)
        fbytes = fused_bytes(wl, lam)[0] if path.fusable else None
        out[T] = {"med": med, "graph": graph_ms, "lam": lam, "bytes": nbytes, "keys": keys,
                  "fused_bytes": fbytes, "fusable": path.fusable}
        progress(f"workload {i} T={T:g}: step {med['step'] * 1e3:.1f} us "
                 f"(three calls {med['step_three_calls'] * 1e3:.1f} us)")
    return wl, out


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only; --gpus {args.gpus} is not supported "
              "(the decode path has no multi-GPU leg in this build)", file=sys.stderr)
        sys.exit(2)
    import torch

    import paper_2609_33410_amd as F
    from workloads import CONFIG_NAMES, make_config

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    F.load_library()
    flush = torch.ones(1 << 28, dtype=torch.int32, device="cuda")  # 1 GiB

    wall0 = time.perf_counter()
    wl, res = run_workload(args.config, args, torch, F, make_config, flush, args.steps,
                           args.warmup, splits=args.splits)
    wall = time.perf_counter() - wall0
    dense, t16 = res[math.inf], res[16.0]
    fusable = dense["fusable"]
    dec_ms = dense["med"]["dec"]
    scan_achieved = dense["bytes"] / (dec_ms * 1e-3) / 1e9
    step_ms = dense["med"]["step"]
    # the dominant kernel: the fused launch (the whole step) where it applies,
    # else the scan of the three-call step
    if fusable:
        r_bytes, r_ms, r_kernel = dense["fused_bytes"], step_ms, "decode_fused_kernel"
        r_timing = "HIP events around the eager launch on its stream (the step is this one launch)"
    else:
        r_bytes, r_ms, r_kernel = dense["bytes"], dec_ms, scan_kernel_name(wl)
        r_timing = "HIP events around the eager launch on its stream"
    achieved = r_bytes / (r_ms * 1e-3) / 1e9
    traffic, trec = counter_traffic(CONFIG_NAMES[args.config] + (" [fused]" if fusable else ""))
    scan_traffic, _ = counter_traffic(CONFIG_NAMES[args.config])
    line = {
        "metric": METRIC,
        "value": round(step_ms * 1e3, 2),
        "unit": "us/call",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(step_ms, 5),
        "higher_is_better": False,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": CONFIG_NAMES[args.config], "batch": wl.batch,
                   "q_heads": wl.num_heads, "kv_heads": wl.num_kv_heads,
                   "head_dim": wl.head_dim, "keys_per_request": wl.flat.seq_lens_host[0],
                   "page_size": wl.page_size, "splits": wl.level_splits,
                   "step": ("estimate + split scan + combine at T=inf in one launch "
                            "(fold_decode_fused)" if fusable else
                            "estimate + split scan + combine at T=inf, launched on one stream"),
                   "timing": "median over steps of HIP events around the step on its stream "
                             "(no event inside the step); a 1 GiB read before each step evicts "
                             "all caches; the breakdown comes from separate steps with events "
                             "between the kernels"},
        "roofline": {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBPS,
                     "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBPS, 4),
                     "traffic": None if traffic is None else int(traffic),
                     "kernel": r_kernel,
                     "algorithmic_bytes_per_launch": int(r_bytes),
                     "avg_launch_us": round(r_ms * 1e3, 2),
                     "launch_timing": r_timing},
        "scan_roofline": {"kernel": scan_kernel_name(wl), "achieved": round(scan_achieved, 1),
                          "frac": round(scan_achieved / HBM_PEAK_GBPS, 4),
                          "traffic": None if scan_traffic is None else int(scan_traffic),
                          "algorithmic_bytes_per_launch": int(dense["bytes"]),
                          "avg_launch_us": round(dec_ms * 1e3, 2),
                          "launch_timing": "HIP events around the scan launch of the three-call "
                                           "step, events between its kernels"},
        "three_calls_us_per_call": {"T=inf": round(dense["med"]["step_three_calls"] * 1e3, 2),
                                    "T=16": round(t16["med"]["step_three_calls"] * 1e3, 2)},
        "t16_us_per_call": round(t16["med"]["step"] * 1e3, 2),
        "graph_replay_us_per_call": {"T=inf": round(dense["graph"] * 1e3, 2),
                                     "T=16": round(t16["graph"] * 1e3, 2)},
        "breakdown_us_eager": {"T=inf": {k: round(v * 1e3, 2) for k, v in dense["med"].items()},
                               "T=16": {k: round(v * 1e3, 2) for k, v in t16["med"].items()}},
        "t16_decode_gbps": round(t16["bytes"] / (t16["med"]["dec"] * 1e-3) / 1e9, 1),
        "t16_value_read_fraction": round(t16["lam"], 5),
        "t16_speedup_decode": round(dense["med"]["dec"] / t16["med"]["dec"], 3),
        "t16_speedup_step": round(dense["med"]["step"] / t16["med"]["step"], 3),
        "t16_paired": paired_depths(Path(wl, F, torch), max(args.steps, 21), 1, flush, torch),
        "keys_per_s": round(dense["keys"] / (step_ms * 1e-3), 1),
        "wall_s": round(wall, 2),
    }
    line["value_model"] = model_leg(Path(wl, F, torch), wl, F, torch, flush, args.steps,
                                    args.warmup)
    progress("value model leg done")
    if not args.no_q8:
        line["q8_keys"] = q8_leg(wl, F, torch, flush, args.steps, args.warmup,
                                 name=CONFIG_NAMES[args.config])
        progress("two-plane key leg done")
        line["v8_values"] = q8_leg(wl, F, torch, flush, args.steps, args.warmup,
                                   name=CONFIG_NAMES[args.config], values8=True)
        progress("8-bit value leg done")
    if args.all:
        line["drafts"] = drafts_leg(F, torch, flush, args.steps, args.warmup)
        progress("draft leg done")
    if not args.no_cpu:
        line["cpu_baseline"] = cpu_baseline(wl, args.cpu_seconds)
    print(json.dumps(line), flush=True)

    if args.calibrate_copy:  # a plain copy of known size for byte-counter calibration
        src = torch.ones(1 << 28, dtype=torch.int32, device="cuda")
        dst = torch.empty_like(src)
        evict_caches(flush)
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst

    if args.all:
        for i in (1, 2, 3, 4, 5):
            wl_i, r = run_workload(i, args, torch, F, make_config, flush, args.steps,
                                   args.warmup)
            for T, v in r.items():
                rec = {"workload": CONFIG_NAMES[i], "T": "inf" if math.isinf(T) else T,
                       "us_per_call": round(v["med"]["step"] * 1e3, 2),
                       "step": "fused" if v["fusable"] else "three calls",
                       "us_per_call_three_calls": round(v["med"]["step_three_calls"] * 1e3, 2),
                       "us_per_call_graph": round(v["graph"] * 1e3, 2),
                       "decode_us": round(v["med"]["dec"] * 1e3, 2),
                       "estimate_us": round(v["med"]["est"] * 1e3, 2),
                       "combine_us": round(v["med"]["comb"] * 1e3, 2),
                       "decode_bytes": int(v["bytes"]),
                       "decode_gbps": round(v["bytes"] / (v["med"]["dec"] * 1e-3) / 1e9, 1),
                       "value_read_fraction": round(v["lam"], 5),
                       "keys_per_s": round(v["keys"] / (v["med"]["step"] * 1e-3), 1)}
                print(json.dumps(rec), file=sys.stderr, flush=True)
            if not args.no_q8:
                rec = {"workload": CONFIG_NAMES[i],
                       "q8_keys": q8_leg(wl_i, F, torch, flush, args.steps, args.warmup,
                                         name=CONFIG_NAMES[i]),
                       "v8_values": q8_leg(wl_i, F, torch, flush, args.steps, args.warmup,
                                           name=CONFIG_NAMES[i], values8=True)}
                print(json.dumps(rec), file=sys.stderr, flush=True)
            del wl_i
            torch.cuda.empty_cache()


if __name__ == "__main__":
    main()
