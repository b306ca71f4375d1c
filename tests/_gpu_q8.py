"""Run the two-plane INT8 key path through the C ABI on a synthetic workload."""

import torch

import paper_2609_33410_amd as F


def pool_view(wl):
    """A contiguous view whose kv sequences are the cache's physical pages (or,
    for a contiguous cache, its sequences): position j of sequence p is slot j
    of page p, so writing every (p, j) encodes the whole cache once."""
    n_pool, hkv, rows, d = wl.k.shape
    lens = torch.full((n_pool,), rows, dtype=torch.int32, device=wl.k.device)
    return F.kv_view(wl.k, None, lens, num_kv_heads=hkv, max_seq_len=rows), lens


def encode_cache(wl):
    """Planes and scales of every stored key, written by the cache writer."""
    n_pool, hkv, rows, d = wl.k.shape
    kv, lens = pool_view(wl)
    keys = F.q8_empty_keys(wl.k)
    keys.plane_a.fill_(0x55)
    keys.plane_b.fill_(0x55)
    keys.scale.fill_(0x5555)
    tok_seq = torch.arange(n_pool, dtype=torch.int32, device=wl.k.device).repeat_interleave(rows)
    tok_pos = torch.arange(rows, dtype=torch.int32, device=wl.k.device).repeat(n_pool)
    k_src = wl.k.permute(0, 2, 1, 3).reshape(n_pool * rows, hkv, d).contiguous()
    F.fold_q8_write_keys(kv, k_src, tok_seq, tok_pos, keys)
    return keys


def value_scale_exp(wl):
    """Smallest e with max|v| 2^-e <= 448 (the cache's value scale)."""
    import math
    vmax = float(wl.v.float().abs().max())
    return int(math.ceil(math.log2(vmax / 448.0))) if vmax > 0 else 0


def encode_values(wl, scale_exp=None):
    """Both E4M3 value planes of every stored value row, by the value writer."""
    n_pool, hkv, rows, d = wl.v.shape
    kv, lens = pool_view(wl)
    vals = F.v8_empty_values(wl.v, value_scale_exp(wl) if scale_exp is None else scale_exp)
    vals.plane_p.fill_(0x55)
    vals.plane_r.fill_(0x55)
    tok_seq = torch.arange(n_pool, dtype=torch.int32, device=wl.v.device).repeat_interleave(rows)
    tok_pos = torch.arange(rows, dtype=torch.int32, device=wl.v.device).repeat(n_pool)
    v_src = wl.v.permute(0, 2, 1, 3).reshape(n_pool * rows, hkv, d).contiguous()
    F.fold_v8_write_values(kv, v_src, tok_seq, tok_pos, vals)
    return vals


def level_views(wl, keys):
    """Level and flat views of the cache; plane A supplies the layout."""
    levels = [F.kv_view(keys.plane_a, wl.v, lv.seq_lens, num_kv_heads=wl.num_kv_heads,
                        max_seq_len=lv.max_seq_len, block_table=lv.block_table,
                        row_indptr=lv.row_indptr, row_req=lv.row_req,
                        max_reqs_per_seq=lv.max_reqs_per_seq, k_is_layout_only=True)
              for lv in wl.levels]
    flat = F.kv_view(keys.plane_a, None, wl.flat.seq_lens, num_kv_heads=wl.num_kv_heads,
                     max_seq_len=wl.flat.max_seq_len, block_table=wl.flat.block_table,
                     k_is_layout_only=True)
    return levels, flat


def split_query(wl, kappa, kappa_v=0.0):
    qq = F.q8_empty_query(wl.q)
    F.fold_q8_split_query(wl.q, wl.sm_scale, qq, req_lens=wl.flat.seq_lens, kappa=kappa,
                          kappa_v=kappa_v)
    return qq


def estimate(wl, keys, qq):
    _, flat = level_views(wl, keys)
    z = torch.empty(wl.batch, wl.num_heads, dtype=torch.float32, device=wl.q.device)
    F.fold_q8_ref_estimate(flat, keys, qq, z)
    return z


def run(wl, T, kappa=0.0, splits=None, z=None, keys=None, debug=False, values=None,
        kappa_v=0.0):
    """Encode (unless keys are given), split the query, estimate (unless z is
    given), scan every level, combine.  Returns host tensors; debug adds each
    level's x, xc, value/page/plane-B (and second value plane) read bits.
    ``values`` (a V8Values) selects 8-bit values."""
    dev = wl.q.device
    splits = list(splits or wl.level_splits)
    if keys is None:
        keys = encode_cache(wl)
    qq = split_query(wl, kappa, kappa_v)
    levels, flat = level_views(wl, keys)
    if z is None:
        z = torch.empty(wl.batch, wl.num_heads, dtype=torch.float32, device=dev)
        F.fold_q8_ref_estimate(flat, keys, qq, z)
    b, h, d = wl.q.shape
    total = sum(splits)
    part_a = torch.full((total, b, h, d), float("nan"), dtype=torch.float32, device=dev)
    part_l = torch.full((total, b, h), float("nan"), dtype=torch.float32, device=dev)
    dbg = []
    off = 0
    for lv, kv, s in zip(wl.levels, levels, splits):
        ex = {}
        if debug:
            rg = F.fold_q8_decode_row_groups(kv, qq)
            npg = (lv.max_seq_len + 15) // 16
            ex = {"x_out": torch.full((b, h, lv.max_seq_len), float("nan"), device=dev),
                  "xc_out": torch.full((b, h, lv.max_seq_len), float("nan"), device=dev),
                  "key_gate_out": torch.full((lv.num_seqs, wl.num_kv_heads, rg, lv.max_seq_len),
                                             255, dtype=torch.uint8, device=dev),
                  "page_gate_out": torch.full((lv.num_seqs, wl.num_kv_heads, rg, npg), 255,
                                              dtype=torch.uint8, device=dev),
                  "refine_gate_out": torch.full((lv.num_seqs, wl.num_kv_heads, rg,
                                                 lv.max_seq_len), 255, dtype=torch.uint8,
                                                device=dev)}
            if values is not None:
                ex["refine_v_gate_out"] = torch.full_like(ex["refine_gate_out"], 255)
        F.fold_q8_decode_split(kv, keys, qq, z, T, s, off, part_a, part_l, values=values, **ex)
        if debug:
            e = {k: v for k, v in ex.items()}
            e["R"] = F.fold_q8_decode_rows_per_group(kv, qq)
            dbg.append(e)
        off += s
    out = torch.empty(b, h, d, dtype=torch.float32, device=dev)
    F.fold_combine(part_a, part_l, out)
    torch.cuda.synchronize()
    res = {"z": z.cpu(), "out": out.cpu(), "part_A": part_a.cpu(), "part_L": part_l.cpu(),
           "splits": splits, "planes": qq.planes.cpu(), "eta": qq.eta.cpu(), "tau": qq.tau.cpu(),
           "tau_v": qq.tau_v.cpu()}
    res["dbg"] = [{k: (v.cpu() if torch.is_tensor(v) else v) for k, v in e.items()} for e in dbg]
    return res, keys
