"""Run the HIP path through the C ABI on a synthetic workload (GPU tests)."""

import math

import numpy as np
import torch

import paper_2609_33410_amd as F


def kv_views(wl, with_v=True):
    levels = [F.kv_view(wl.k, wl.v if with_v else None, lv.seq_lens,
                        num_kv_heads=wl.num_kv_heads, max_seq_len=lv.max_seq_len,
                        block_table=lv.block_table, row_indptr=lv.row_indptr,
                        row_req=lv.row_req, max_reqs_per_seq=lv.max_reqs_per_seq)
              for lv in wl.levels]
    flat = F.kv_view(wl.k, None, wl.flat.seq_lens, num_kv_heads=wl.num_kv_heads,
                     max_seq_len=wl.flat.max_seq_len, block_table=wl.flat.block_table)
    return levels, flat


def estimate(wl):
    _, flat = kv_views(wl, with_v=False)
    z = torch.empty(wl.batch, wl.num_heads, dtype=torch.float32, device=wl.q.device)
    F.fold_ref_estimate(flat, F.q_view(wl.q), wl.sm_scale, z)
    return z


def run(wl, T, splits=None, z=None, debug=False, out_dtype=torch.float32):
    """Estimate (unless z is given), scan every level, combine.  Returns a dict
    of host tensors; debug adds each level's x / key gates / page gates."""
    dev = wl.q.device
    splits = list(splits or wl.level_splits)
    levels, flat = kv_views(wl)
    qv = F.q_view(wl.q)
    if z is None:
        z = torch.empty(wl.batch, wl.num_heads, dtype=torch.float32, device=dev)
        F.fold_ref_estimate(flat, qv, wl.sm_scale, z)
    b, h, d = wl.q.shape
    total = sum(splits)
    part_a = torch.full((total, b, h, d), float("nan"), dtype=torch.float32, device=dev)
    part_l = torch.full((total, b, h), float("nan"), dtype=torch.float32, device=dev)
    dbg = []
    off = 0
    for lv, kv, s in zip(wl.levels, levels, splits):
        x = kg = pg = None
        if debug:
            rg = F.fold_decode_row_groups(kv, qv)
            x = torch.full((b, h, lv.max_seq_len), float("nan"), dtype=torch.float32, device=dev)
            kg = torch.full((lv.num_seqs, wl.num_kv_heads, rg, lv.max_seq_len), 255,
                            dtype=torch.uint8, device=dev)
            pg = torch.full((lv.num_seqs, wl.num_kv_heads, rg, (lv.max_seq_len + 15) // 16), 255,
                            dtype=torch.uint8, device=dev)
        F.fold_decode_split(kv, qv, wl.sm_scale, z, T, s, off, part_a, part_l, x_out=x,
                            key_gate_out=kg, page_gate_out=pg)
        if debug:
            dbg.append({"x": x, "kg": kg, "pg": pg, "R": F.fold_decode_rows_per_group(kv, qv)})
        off += s
    out = torch.empty(b, h, d, dtype=out_dtype, device=dev)
    lse = torch.empty(b, h, dtype=torch.float32, device=dev)
    cert = torch.empty(b, h, dtype=torch.uint8, device=dev)
    F.fold_combine(part_a, part_l, out, z=z, lse_out=lse, cert_out=cert)
    torch.cuda.synchronize()
    res = {"z": z.cpu(), "out": out.cpu(), "part_A": part_a.cpu(), "part_L": part_l.cpu(),
           "lse": lse.cpu(), "cert": cert.cpu(), "splits": splits}
    res["dbg"] = [{k: (v.cpu() if torch.is_tensor(v) else v) for k, v in e.items()} for e in dbg]
    return res


def row_errors(o_gpu, o_ref):
    """Per-row max-abs error divided by the row's inf-norm."""
    o_gpu = np.asarray(o_gpu, dtype=np.float64)
    scale = np.abs(o_ref).max(axis=-1)
    return np.abs(o_gpu - o_ref).max(axis=-1) / np.where(scale > 0, scale, 1.0)


def rel_l2(o_gpu, o_ref):
    o_gpu = np.asarray(o_gpu, dtype=np.float64)
    return float(np.linalg.norm(o_gpu - o_ref) / np.linalg.norm(o_ref))


def is_inf(T):
    return T is None or math.isinf(T)
