"""Decode-attention benchmark on one MI355X.

A step is one pass of the whole decode hot path over one batch: the
reference estimate, the gated split-KV scan of every level, and the additive
combine.  The headline workload is the largest single-GPU one, the MHA
long-context stress decode (batch 4, 32 heads, head dim 128, 64K-128K cached
keys per request drawn uniformly, split-KV 32 ways, paged BF16 cache of
16-key pages), at T = inf, with its T = 16 step beside it.  The
Llama-3-8B-shaped GQA decode and the Qwen3-8B-shaped 32K-key decode (its
depth sweep T in {inf, 24, 16, 12}) ride along as extra keys.  Inputs are
synthetic, seeded and resident in HBM before timing.  Before every timed
step a 1 GiB buffer is read, so that no cache (4 MB L2 per XCD, 256 MB MALL)
holds any of the step's data and no dirty line is left to drain during the
step; each step is bracketed by HIP events on the stream the kernels are
launched on.

Prints ONE JSON line (rank 0).  The line also carries the headline workload
over a two-plane INT8 key cache (``q8_keys``; Section 4, cache format) and
with 8-bit values (``v8_values``), the cut-key value models' errors and costs
(``value_model``: no model, the request mean, the block model of BF16 values,
at T = 16 and 14; ``value_model_structured``: the same errors on the 32K-key
GQA shapes with structured values) and the FP64 oracle timed on the host
(``cpu_baseline``).
``--all`` adds one JSON line per workload and depth on stderr (used for the
design notes' tables).
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
    ap.add_argument("--config", type=int, default=4,
                    help="headline workload (default 4: MHA 4 x 64K-128K keys, the largest "
                         "single-GPU workload)")
    ap.add_argument("--only", action="store_true",
                    help="time only the headline workload (no workload-2/3 extra keys)")
    ap.add_argument("--all", action="store_true", help="also time workloads 1-5 (stderr)")
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle baseline")
    ap.add_argument("--no-q8", action="store_true",
                    help="skip the two-plane INT8 key legs (BF16 and 8-bit values)")
    ap.add_argument("--cpu-seconds", type=float, default=15.0)
    ap.add_argument("--no-graph", action="store_true", help="skip the graph-replay leg")
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
        # a cascade whose prefix level is stacked (64-row read groups) and whose
        # suffix level is per request: both levels in one scan launch
        # (fold_decode_cascade), whose splits[0] slots hold both levels' pairs
        self.one_scan = (len(wl.levels) == 2 and wl.levels[0].row_indptr is not None
                         and wl.levels[1].row_indptr is None and wl.levels[1].num_seqs == b
                         and F.fold_decode_rows_per_group(self.levels[0], self.qv) == 64)
        self.slots = self.splits[0] if self.one_scan else total

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
        if self.one_scan:
            self.F.fold_decode_cascade(self.levels[0], self.levels[1], self.qv, self.wl.sm_scale,
                                       self.z, T, self.slots, 0, self.part_A[:self.slots],
                                       self.part_L[:self.slots], stream=stream)
        else:
            self.decode_levels(T, stream)

    def decode_levels(self, T, stream):
        """Every level's scan as its own launch."""
        off = 0
        for kv, s in zip(self.levels, self.splits):
            self.F.fold_decode_split(kv, self.qv, self.wl.sm_scale, self.z, T, s, off,
                                     self.part_A, self.part_L, stream=stream)
            off += s

    def combine(self, stream):
        self.F.fold_combine(self.part_A[:self.slots], self.part_L[:self.slots], self.out,
                            stream=stream)

    def level_launches(self, T, stream):
        """The call with one scan launch per level (a cascade's alternative)."""
        self.estimate(stream)
        self.decode_levels(T, stream)
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
        # levels past 32 rows per kv sequence (a cascade prefix) run as a
        # stacked level over FP16 keys written once per prefix (BF16 values)
        self.stacked = [None] * len(wl.levels)
        if not values8:
            for i, lv in enumerate(wl.levels):
                reqs = lv.max_reqs_per_seq if lv.row_indptr is not None else 1
                if reqs * wl.group > 32:  # the stacked-row threshold
                    k16 = torch.empty(self.keys.plane_a.shape, dtype=torch.float16, device=dev)
                    F.fold_q8_stack_keys(self.levels[i], self.keys, k16)
                    self.stacked[i] = F.kv_view(
                        k16, wl.v, lv.seq_lens, num_kv_heads=wl.num_kv_heads,
                        max_seq_len=lv.max_seq_len, block_table=lv.block_table,
                        row_indptr=lv.row_indptr, row_req=lv.row_req,
                        max_reqs_per_seq=lv.max_reqs_per_seq)
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

    def front(self, stream):
        """Query split and reference estimate in one launch (fold_q8_front)."""
        self.F.fold_q8_front(self.flat, self.keys, self.wl.q, self.wl.sm_scale, self.qq, self.z,
                             req_lens=self.wl.flat.seq_lens, kappa=self.kappa,
                             kappa_v=self.kappa_v, stream=stream)

    def decode(self, T, stream):
        off = 0
        for kv, stk, s in zip(self.levels, self.stacked, self.splits):
            if stk is not None:
                self.F.fold_q8_decode_stacked(stk, self.qq, self.z, T, s, off, self.part_A,
                                              self.part_L, stream=stream)
            else:
                self.F.fold_q8_decode_split(kv, self.keys, self.qq, self.z, T, s, off,
                                            self.part_A, self.part_L, values=self.vals,
                                            stream=stream)
            off += s

    def stack_keys(self, stream):
        """Re-write the stacked levels' FP16 keys (a once-per-prefix cost)."""
        for kv, stk in zip(self.levels, self.stacked):
            if stk is not None:
                self.F.fold_q8_stack_keys(kv, self.keys, stk.tensors[0], stream=stream)

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
        for lv, kv, stk, s in zip(self.wl.levels, self.levels, self.stacked, self.splits):
            if stk is not None:  # the stacked level reads every key and value row
                n_keys = sum(lv.seq_lens_host) * self.wl.num_kv_heads
                nv += n_keys
                nb += n_keys
                total += n_keys
                off += s
                continue
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


def model_leg(path, wl, F, torch, flush, steps, warmup, depths=(16.0, 14.0), timed=True):
    """The cut-key value models on a workload: the output error against the
    dense output (exact softmax up to FP32 rounding) at finite depths with no
    model, the request mean (the model of 8-bit values) and the block model
    of BF16 values (64-key block means, one virtual row per tile); and, when
    ``timed``, the scan time with each model and the time of the block-mean
    fit over the whole cache (a prompt-time call)."""
    dev = wl.q.device
    b, h, d = wl.q.shape
    fl = wl.flat
    kv = F.kv_view(wl.k, wl.v, fl.seq_lens, num_kv_heads=wl.num_kv_heads,
                   max_seq_len=fl.max_seq_len, block_table=fl.block_table)
    mean = torch.empty(fl.num_seqs, wl.num_kv_heads, d, dtype=torch.float32, device=dev)
    stream = torch.cuda.current_stream()
    path.estimate(stream)
    F.fold_value_mean(kv, mean)
    bms = [torch.empty(lv.num_seqs, wl.num_kv_heads, F.block_count(lv.max_seq_len), d,
                       dtype=torch.float32, device=dev) for lv in wl.levels]

    def fit(stream):
        for kvl, bm in zip(path.levels, bms):
            F.fold_value_block_mean(kvl, bm, stream=stream)

    fit(stream)
    part_C = torch.empty_like(path.part_L)
    cut = torch.empty(b * h * max(F.chunk_count(lv.max_seq_len) for lv in wl.levels),
                      dtype=torch.float32, device=dev)

    def decode_cut(T, stream):
        off = 0
        for kvl, s in zip(path.levels, path.splits):
            F.fold_decode_split(kvl, path.qv, wl.sm_scale, path.z, T, s, off, path.part_A,
                                path.part_L, part_Lcut=part_C, stream=stream)
            off += s

    def decode_blocks(T, stream):
        off = 0
        for kvl, s, bm in zip(path.levels, path.splits, bms):
            F.fold_decode_split_blocks(kvl, path.qv, wl.sm_scale, path.z, T, s, off,
                                       path.part_A, path.part_L, bm, cut, stream=stream)
            off += s

    def timed_us(fn):
        ts = []
        for it in range(warmup + steps):
            evict_caches(flush)
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            fn(stream)
            e1.record(stream)
            if it >= warmup:
                e1.synchronize()
                ts.append(e0.elapsed_time(e1))
        return round(statistics.median(ts) * 1e3, 2)

    dense = torch.empty(b, h, d, dtype=torch.float32, device=dev)
    path.decode(math.inf, stream)
    F.fold_combine(path.part_A, path.part_L, dense, stream=stream)
    torch.cuda.synchronize()
    scale = dense.abs().amax(dim=-1).clamp_min(1e-30)

    def errs(o):
        e = (o - dense).abs().amax(dim=-1) / scale
        return {"max_row": float(e.max()), "median_row": float(e.median()),
                "rel_l2": float((o - dense).norm() / dense.norm())}

    rec = {"models": {"no_model": "cut keys add nothing to A",
                      "request_mean": "cut keys carry their request's mean value row",
                      "block_mean": "each 64-key tile's cut mass carries its block's mean value "
                                    "row (one virtual row per tile)"},
           "reference": "dense decode of the same kernel (T = inf)"}
    for T in depths:
        plain = torch.empty_like(dense)
        path.decode(T, stream)
        F.fold_combine(path.part_A, path.part_L, plain, stream=stream)
        model = torch.empty_like(dense)
        decode_cut(T, stream)
        F.fold_combine(path.part_A, path.part_L, model, part_Lcut=part_C, mean=mean,
                       stream=stream)
        blocks = torch.empty_like(dense)
        decode_blocks(T, stream)
        F.fold_combine(path.part_A, path.part_L, blocks, stream=stream)
        torch.cuda.synchronize()
        cut_share = float(part_C.double().sum() / path.part_L.double().sum())
        r = {"err_vs_dense": {"no_model": errs(plain), "request_mean": errs(model),
                              "block_mean": errs(blocks)},
             "cut_mass_share": cut_share}
        if timed:
            r["scan_us"] = {"no_model": timed_us(lambda st: path.decode(T, st)),
                            "request_mean_cut_masses": timed_us(lambda st: decode_cut(T, st)),
                            "block_mean_scan_and_virtual_rows":
                                timed_us(lambda st: decode_blocks(T, st))}
        rec[depth_key(T)] = r
    if timed:
        rec["block_mean_fit_us"] = timed_us(fit)
    return rec


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
    res = {"front": [], "dec": [], "comb": [], "step": [], "append": [], "split_then_est": []}
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
    for it in range(warmup + steps):
        for key in ("step", "split_then_est"):
            evict_caches(flush)
            e0 = torch.cuda.Event(enable_timing=True)
            e1 = torch.cuda.Event(enable_timing=True)
            e0.record(stream)
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
                   "scan + combine; the one-token append is timed apart"}
    if values8:
        out["kappa_v"] = qp.kappa_v
    if any(stk is not None for stk in qp.stacked):
        out["stacked_levels"] = ("levels past 32 rows per kv sequence run on FP16 keys "
                                 "fp16(e (a + b/256)) written once per prefix "
                                 "(fold_q8_stack_keys, timed apart)")
        ts = []
        for it in range(warmup + steps):
            evict_caches(flush)
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            qp.stack_keys(stream)
            e1.record(stream)
            if it >= warmup:
                e1.synchronize()
                ts.append(e0.elapsed_time(e1))
        out["stack_keys_us_once_per_prefix"] = round(statistics.median(ts) * 1e3, 2)
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
                               "kernel": q8_kernel_name(wl, values8)}
    del qp
    torch.cuda.empty_cache()
    return out


def kv_bytes(wl, lam, slots=None):
    """Algorithmic bytes of one decode scan (all levels): every key row, the
    value rows the read gates keep (fraction lam of read-group key rows), the
    query rows, references, block-table entries and partials written (`slots`
    of them; one per split of every level unless given)."""
    d = wl.head_dim
    b, h, _ = wl.q.shape
    keys = sum(sum(lv.seq_lens_host) for lv in wl.levels) * wl.num_kv_heads
    total = keys * 2 * d + lam * keys * 2 * d
    total += 2 * b * h * d + 4 * b * h
    if wl.page_size:
        total += 4 * sum(sum((n + wl.page_size - 1) // wl.page_size for n in lv.seq_lens_host)
                         for lv in wl.levels)
    total += 4 * (sum(wl.level_splits) if slots is None else slots) * b * h * (d + 1)
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
    """Algorithmic bytes of one fused launch: the scan's (every key row, the
    value rows the gates keep, queries, references, block-table entries,
    slots written) plus the combine's read of the slots and its FP32 output.
    The estimate's sampled key rows are rows the scan reads anyway; they are
    not counted a second time."""
    d = wl.head_dim
    b, h, _ = wl.q.shape
    total, keys = kv_bytes(wl, lam)
    total += 4 * sum(wl.level_splits) * b * h * (d + 1) + 4 * b * h * d
    return total, keys


def scan_kernel_name(wl, dense=True):
    """The scan kernel (with its template arguments as rocprofv3 prints them)
    the library launches for a single-level workload."""
    d, dn = wl.head_dim, "true" if dense else "false"
    if wl.group == 1:
        # waves per workgroup: 8 when each wave gets at least 4 chunks of the
        # longest sequence per split, else 4 (the library's rule)
        w = 8 if ((wl.flat.max_seq_len + 15) // 16) // wl.level_splits[0] >= 32 else 4
        return f"decode_split_kernel<{d}, 1, {dn}, false, {w}>"
    if wl.group <= 8:
        return f"decode_packed_kernel<{d}, {4 if wl.group <= 4 else 2}, {dn}, false>"
    return f"decode_mfma_kernel<{d}, ...>"


def q8_kernel_name(wl, values8):
    """The dense two-plane scan kernel of a single-level workload."""
    v8 = "true" if values8 else "false"
    if wl.group == 1:
        return f"decode_q8_split_kernel<{wl.head_dim}, true, false, {v8}, 4>"
    if wl.group <= 8:
        return f"decode_q8_packed_kernel<{wl.head_dim}, 2, true, false, {v8}>"
    return f"decode_q8_kernel<{wl.head_dim}, ..., true, false, {v8}>"


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


def time_call(fn, T, steps, warmup, flush, torch):
    """Median duration (ms) of one call fn(T, stream), caches evicted before
    each, events only around it."""
    stream = torch.cuda.current_stream()
    ts = []
    for it in range(warmup + steps):
        evict_caches(flush)
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        fn(T, stream)
        e1.record(stream)
        if it >= warmup:
            e1.synchronize()
            ts.append(e0.elapsed_time(e1))
    torch.cuda.synchronize()
    return statistics.median(ts)


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


def graph_leg(workloads, F, torch, flush, steps, warmup):
    """Timed last, after every eager leg: each workload's step replayed from a
    captured HIP graph, the same step eagerly again afterwards, and what a
    replay adds around one trivial kernel.  On this platform the first graph
    capture (like the first launch on a second stream) leaves every later
    kernel of the process about 8 % slower, with unchanged clocks; timing the
    graphs last keeps the eager figures free of that."""
    out = {}
    for name, wl in workloads:
        path = Path(wl, F, torch)
        path.estimate(torch.cuda.current_stream())
        rec = {}
        for T in (math.inf, 16.0):
            rec[depth_key(T)] = {"graph_replay_us": round(
                time_graph(path, T, steps, warmup, flush, torch) * 1e3, 2)}
        for T in (math.inf, 16.0):
            med, _ = time_variant(path, T, steps, warmup, flush, torch)
            rec[depth_key(T)]["eager_us_after_capture"] = round(med["step"] * 1e3, 2)
            rec[depth_key(T)]["eager_decode_us_after_capture"] = round(med["dec"] * 1e3, 2)
        out[name] = rec
        del path
        torch.cuda.empty_cache()
    out["one_fill_kernel"] = graph_overhead(max(steps, 11), flush, torch)
    out["note"] = ("graph replays and the eager steps after them run after the process's first "
                   "graph capture, which slows every kernel of the process by about 8 % on this "
                   "platform; the eager figures elsewhere in this line precede any capture")
    return out


def graph_overhead(steps, flush, torch):
    """What a graph replay adds around its kernels: one 4-byte fill kernel timed
    eagerly and as a one-node graph replay (events around each, caches evicted
    before each), medians in us."""
    stream = torch.cuda.current_stream()
    x = torch.zeros(1, dtype=torch.int32, device="cuda")
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        x.fill_(1)
    res = {"eager": [], "graph": []}
    for it in range(steps + 1):
        for key in ("eager", "graph"):
            evict_caches(flush)
            e0 = torch.cuda.Event(enable_timing=True)
            e1 = torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            if key == "graph":
                g.replay()
            else:
                x.fill_(1)
            e1.record(stream)
            e1.synchronize()
            if it:
                res[key].append(e0.elapsed_time(e1))
    med = {k: statistics.median(v) * 1e3 for k, v in res.items()}
    return {"one_fill_kernel_eager_us": round(med["eager"], 2),
            "one_fill_kernel_graph_us": round(med["graph"], 2),
            "graph_adds_us": round(med["graph"] - med["eager"], 2)}


def _local_includes(path):
    import re

    out = []
    with open(path) as f:
        for line in f:
            m = re.match(r'\s*#\s*include\s+"([^"]+)"', line)
            if m:
                out.append(m.group(1))
    return out


def kernel_sources_sha(source="*"):
    """SHA-256 over the source files of some kernels (a file name or a list of
    them) and every local header they include (transitively), or over every
    library source with ``source="*"``; it identifies the code a counter
    record was taken on."""
    import glob
    import hashlib

    csrc = os.path.join(ROOT, "paper_2609_33410_amd", "csrc")
    if source == "*":
        files = sorted(os.path.basename(f) for f in glob.glob(os.path.join(csrc, "*")))
    else:
        seen, todo = set(), [source] if isinstance(source, str) else list(source)
        while todo:
            f = todo.pop()
            if f in seen or not os.path.exists(os.path.join(csrc, f)):
                continue
            seen.add(f)
            todo.extend(_local_includes(os.path.join(csrc, f)))
        files = sorted(seen)
    h = hashlib.sha256()
    for f in files:
        with open(os.path.join(csrc, f), "rb") as fh:
            h.update(f.encode() + b"\0" + fh.read())
    return h.hexdigest()


def counter_traffic(workload_name):
    """HBM bytes per dense decode launch from the committed counter summary,
    or None when it is absent or the kernel's sources changed since."""
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
    if r is None or r.get("source_sha256") != kernel_sources_sha(r.get("sources", "*")):
        return None, r
    kib = r["fetch_kib"] * r["fetch_scale"] + r["write_kib"] * r["write_scale"]
    return kib * 1024.0, r


def cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:  # pragma: no cover
        pass
    return "unknown"


def cpu_baseline(wl, budget_s, T_cut=16.0):
    """The FP64 oracle, as it stands, timed on this host's cores on a bounded
    sample of the workload's (request, kv head) chunks and scaled to one whole
    call: the oracle's estimator (its own reference for the sampled rows), and
    the decode (gather, scores, depth rule, fold, splits) at T = inf and at
    T = T_cut with that reference.  Chunks are taken in a seeded random order,
    so long and short requests of a ragged batch are both sampled."""
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
    fl = wl.flat
    bt = None if fl.block_table is None else fl.block_table.cpu().numpy()
    group = wl.group
    chunks_all = [(s, g) for s in range(fl.num_seqs) for g in range(wl.num_kv_heads)]
    order = np.random.default_rng(0).permutation(len(chunks_all))
    chunks_all = [chunks_all[i] for i in order]
    z = np.zeros((wl.batch, wl.num_heads))
    keys_of = {c: int(fl.seq_lens_host[c[0]]) for c in chunks_all}
    all_keys = sum(keys_of.values())

    def run(leg, budget):
        done, keys = [], 0
        t0 = time.perf_counter()
        for c in chunks_all:
            if leg == "estimate":
                rows = [(c[0], c[1] * group + hh) for hh in range(group)]
                zc = oracle.estimate_level(q_bits, k_bits, num_kv_heads=wl.num_kv_heads,
                                           page_size=wl.page_size, sm_scale=wl.sm_scale,
                                           seq_lens=fl.seq_lens_host, block_table=bt, rows=rows)
                for r, h in rows:
                    z[r, h] = zc[r, h]
            else:
                oracle.decode_level(q_bits, k_bits, v_bits, num_kv_heads=wl.num_kv_heads,
                                    page_size=wl.page_size, sm_scale=wl.sm_scale,
                                    seq_lens=fl.seq_lens_host, block_table=bt, z=z, T=leg,
                                    num_splits=wl.level_splits[0], chunks=[c])
            done.append(c)
            keys += keys_of[c]
            if time.perf_counter() - t0 > budget:
                break
        dt = time.perf_counter() - t0
        return dt * all_keys / keys, len(done), dt  # scaled by keys to one whole call

    est_s, n_est, dt_est = run("estimate", budget_s / 4)
    chunks_all = chunks_all[:n_est]  # the decode needs the sampled rows' references
    inf_s, n_inf, dt_inf = run(math.inf, budget_s * 3 / 8)
    cut_s, n_cut, dt_cut = run(T_cut, budget_s * 3 / 8)
    keys = sum(fl.seq_lens_host) * wl.num_kv_heads
    del q_bits, k_bits, v_bits
    return {"value": round((est_s + inf_s) * 1e6, 1), "unit": "us/call", "cores": threads,
            "host_cores_visible": cores, "cpu_model": cpu_model(), "kind": "oracle",
            "decode_us_per_call": {"T=inf": round(inf_s * 1e6, 1),
                                   f"T={T_cut:g}": round(cut_s * 1e6, 1)},
            "estimate_us_per_call": round(est_s * 1e6, 1),
            "keys_per_s": {"T=inf": round(keys / inf_s, 1), f"T={T_cut:g}": round(keys / cut_s, 1)},
            "sample": f"FP64 oracle on {cores} visible host cores ({threads} BLAS threads): "
                      f"estimator on {n_est} of {fl.num_seqs * wl.num_kv_heads} (request, kv head) "
                      f"chunks in {dt_est:.1f} s; decode of {n_inf} of them at T=inf in "
                      f"{dt_inf:.1f} s and of {n_cut} at T={T_cut:g} in {dt_cut:.1f} s; each "
                      f"leg scaled by keys to one whole call; value = estimator + T=inf decode"}


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


def run_workload(i, args, torch, F, make_config, flush, steps, warmup, splits=None,
                 depths=None, wl=None):
    if wl is None:
        wl = make_config(i, device="cuda")
    if splits is not None and len(wl.level_splits) == 1:
        wl.level_splits = [splits]
    path = Path(wl, F, torch)
    stream = torch.cuda.current_stream()
    path.estimate(stream)
    out = {}
    if depths is None:
        depths = (math.inf, 16.0) + ((24.0, 12.0) if i == 3 else ())
    for T in depths:
        lam = path.read_fraction(T)
        med, _ = time_variant(path, T, steps, warmup, flush, torch)
        nbytes, keys = kv_bytes(wl, lam, path.slots)
        fbytes = fused_bytes(wl, lam)[0] if path.fusable else None
        out[T] = {"med": med, "lam": lam, "bytes": nbytes, "keys": keys,
                  "fused_bytes": fbytes, "fusable": path.fusable, "one_scan": path.one_scan}
        if path.one_scan:
            out[T]["level_launches"] = time_call(path.level_launches, T, steps, warmup, flush,
                                                 torch)
        progress(f"workload {i} T={T:g}: step {med['step'] * 1e3:.1f} us "
                 f"(three calls {med['step_three_calls'] * 1e3:.1f} us)")
    return wl, out


def depth_key(T):
    return "T=inf" if math.isinf(T) else f"T={T:g}"


def gbps(nbytes, ms):
    return round(nbytes / (ms * 1e-3) / 1e9, 1)


def depth_record(wl, v, T):
    """One depth of a workload: the step, its kernels, bytes and rates."""
    med = v["med"]
    rec = {"us_per_call": round(med["step"] * 1e3, 2),
           "step": "fused" if v["fusable"] else "three calls",
           "us_per_call_three_calls": round(med["step_three_calls"] * 1e3, 2),
           "decode_us": round(med["dec"] * 1e3, 2),
           "estimate_us_with_marker": round(med["est"] * 1e3, 2),
           "combine_us_with_marker": round(med["comb"] * 1e3, 2),
           "decode_bytes": int(v["bytes"]),
           "decode_gbps": gbps(v["bytes"], med["dec"]),
           "decode_frac_of_peak": round(v["bytes"] / (med["dec"] * 1e-3) / 1e9 / HBM_PEAK_GBPS, 4),
           "value_read_fraction": round(v["lam"], 5),
           "keys_per_s": round(v["keys"] / (med["step"] * 1e-3), 1)}
    if v["fusable"]:
        rec["fused_bytes"] = int(v["fused_bytes"])
        rec["fused_gbps"] = gbps(v["fused_bytes"], med["step"])
    if v.get("one_scan"):
        rec["scan"] = ("fold_decode_cascade: the prefix and suffix levels in one launch, "
                       "their pairs in the prefix's slots")
        rec["us_per_call_level_launches"] = round(v["level_launches"] * 1e3, 2)
    return rec


def workload_summary(i, wl, res, paired):
    """Extra-key record of a workload: every depth, and the paired speedups."""
    names = __import__("workloads").CONFIG_NAMES
    out = {"workload": names[i], "batch": wl.batch, "q_heads": wl.num_heads,
           "kv_heads": wl.num_kv_heads, "head_dim": wl.head_dim,
           "keys_per_request": list(wl.flat.seq_lens_host) if len(set(wl.flat.seq_lens_host)) > 1
           else wl.flat.seq_lens_host[0], "splits": wl.level_splits,
           "scan_kernel": scan_kernel_name(wl)}
    for T, v in res.items():
        out[depth_key(T)] = depth_record(wl, v, T)
    for T, pr in paired.items():
        out[depth_key(T)]["paired_vs_T=inf"] = pr
    return out


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only; --gpus {args.gpus} is not supported "
              "(the path runs on one GPU; how it would shard is a design, not code)",
              file=sys.stderr)
        sys.exit(2)
    import torch

    import paper_2609_33410_amd as F
    from workloads import CONFIG_NAMES, make_config

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    F.load_library()
    flush = torch.ones(1 << 28, dtype=torch.int32, device="cuda")  # 1 GiB

    cfg = args.config
    wall0 = time.perf_counter()
    wl, res = run_workload(cfg, args, torch, F, make_config, flush, args.steps, args.warmup,
                           splits=args.splits)
    wall = time.perf_counter() - wall0
    dense, t16 = res[math.inf], res[16.0]
    fusable = dense["fusable"]
    dec_ms = dense["med"]["dec"]
    step_ms = dense["med"]["step"]
    # the dominant kernel: the fused launch (the whole step) where it applies,
    # else the scan of the three-call step
    if fusable:
        r_bytes, r_ms, r_kernel = dense["fused_bytes"], step_ms, "decode_fused_kernel"
        r_timing = "HIP events around the eager launch on its stream (the step is this one launch)"
        tkey = CONFIG_NAMES[cfg] + " [fused]"
    else:
        r_bytes, r_ms, r_kernel = dense["bytes"], dec_ms, scan_kernel_name(wl)
        r_timing = ("HIP events on the launch stream around the scan launch of the "
                    "three-call step (events between its kernels)")
        tkey = CONFIG_NAMES[cfg]
    achieved = r_bytes / (r_ms * 1e-3) / 1e9
    traffic, _ = counter_traffic(tkey)
    keys = dense["keys"]
    pairs = sum(wl.flat.seq_lens_host) * wl.num_heads
    paired16 = paired_depths(Path(wl, F, torch), max(args.steps, 21), 1, flush, torch)
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
        "config": {"workload": CONFIG_NAMES[cfg], "batch": wl.batch,
                   "q_heads": wl.num_heads, "kv_heads": wl.num_kv_heads,
                   "head_dim": wl.head_dim,
                   "keys_per_request": list(wl.flat.seq_lens_host),
                   "page_size": wl.page_size, "splits": wl.level_splits, "depth": "T=inf",
                   "step": ("estimate + split scan + combine at T=inf in one launch "
                            "(fold_decode_fused)" if fusable else
                            "fold_ref_estimate + fold_decode_split + fold_combine at T=inf, "
                            "launched on one stream"),
                   "timing": "median over steps of HIP events around the step on its stream "
                             "(no event inside the step); a 1 GiB read before each step evicts "
                             "all caches; the kernel breakdown comes from separate steps with "
                             "events between the kernels"},
        "roofline": {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBPS,
                     "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBPS, 4),
                     "traffic": None if traffic is None else int(traffic),
                     "kernel": r_kernel,
                     "algorithmic_bytes_per_launch": int(r_bytes),
                     "avg_launch_us": round(r_ms * 1e3, 2),
                     "launch_timing": r_timing},
        "T=16": dict(depth_record(wl, t16, 16.0), paired_vs_T_inf=paired16),
        "T=inf": depth_record(wl, dense, math.inf),
        "t16_us_per_call": round(t16["med"]["step"] * 1e3, 2),
        "t16_speedup_step": paired16["speedup_step_median"],
        "t16_speedup_decode": paired16["speedup_decode_median"],
        "keys_per_s": round(keys / (step_ms * 1e-3), 1),
        "query_key_pairs_per_s": round(pairs / (step_ms * 1e-3), 1),
        "wall_s": round(wall, 2),
    }
    keep = [(CONFIG_NAMES[cfg], wl)]
    del res
    torch.cuda.empty_cache()
    # the other long-context and GQA workloads, as extra keys
    for extra in (2, 3):
        if extra == cfg or args.only:
            continue
        wl_x, r = run_workload(extra, args, torch, F, make_config, flush, args.steps,
                               args.warmup)
        paired = {}
        for T in r:
            if not math.isinf(T):
                paired[T] = paired_depths(Path(wl_x, F, torch), max(args.steps, 21), 1, flush,
                                          torch, T_cut=T)
        rec = workload_summary(extra, wl_x, r, paired)
        if r[math.inf]["fusable"]:
            fb = r[math.inf]["fused_bytes"]
            fms = r[math.inf]["med"]["step"]
            ft, _ = counter_traffic(CONFIG_NAMES[extra] + " [fused]")
            rec["roofline"] = {"bound": "hbm", "kernel": "decode_fused_kernel",
                               "achieved": gbps(fb, fms), "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                               "frac": round(fb / (fms * 1e-3) / 1e9 / HBM_PEAK_GBPS, 4),
                               "traffic": None if ft is None else int(ft),
                               "algorithmic_bytes_per_launch": int(fb),
                               "avg_launch_us": round(fms * 1e3, 2)}
        line[f"workload{extra}"] = rec
        progress(f"workload {extra} leg done")
        keep.append((CONFIG_NAMES[extra], wl_x))
        del r
        torch.cuda.empty_cache()
    line["value_model"] = model_leg(Path(wl, F, torch), wl, F, torch, flush, args.steps,
                                    args.warmup)
    progress("value model leg done")
    if not args.only:
        # structured values (channel offset + per-segment topics + noise) on
        # the 32K-key GQA shapes, where the models have something to capture
        wl_s = make_config(3, device="cuda", values="structured")
        rec = model_leg(Path(wl_s, F, torch), wl_s, F, torch, flush, args.steps, args.warmup,
                        depths=(16.0, 14.0, 12.0), timed=False)
        rec["workload"] = CONFIG_NAMES[3] + " with structured values"
        line["value_model_structured"] = rec
        del wl_s
        torch.cuda.empty_cache()
        progress("structured-value model leg done")
    if not args.no_q8:
        line["q8_keys"] = q8_leg(wl, F, torch, flush, args.steps, args.warmup,
                                 name=CONFIG_NAMES[cfg])
        progress("two-plane key leg done")
        line["v8_values"] = q8_leg(wl, F, torch, flush, args.steps, args.warmup,
                                   name=CONFIG_NAMES[cfg], values8=True)
        progress("8-bit value leg done")
    if args.all:
        line["drafts"] = drafts_leg(F, torch, flush, args.steps, args.warmup)
        progress("draft leg done")
    if not args.no_cpu:
        line["cpu_baseline"] = cpu_baseline(wl, args.cpu_seconds)
        progress("CPU baseline done")
    if not args.no_graph:
        line["graph_replay"] = graph_leg(keep, F, torch, flush, args.steps, args.warmup)
        progress("graph leg done")
    del keep
    print(json.dumps(line), flush=True)

    if args.calibrate_copy:  # a plain copy of known size for byte-counter calibration
        src = torch.ones(1 << 28, dtype=torch.int32, device="cuda")
        dst = torch.empty_like(src)
        evict_caches(flush)
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst

    if args.all:
        del wl
        torch.cuda.empty_cache()
        for i in (1, 2, 3, 4, 5):
            wl_i, r = run_workload(i, args, torch, F, make_config, flush, args.steps,
                                   args.warmup)
            for T, v in r.items():
                rec = dict({"workload": CONFIG_NAMES[i], "T": "inf" if math.isinf(T) else T},
                           **depth_record(wl_i, v, T))
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
