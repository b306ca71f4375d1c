"""Turn a synthetic workload into the plain numpy arguments the oracle takes."""

import numpy as np

from workloads import host_bits


def level_args(view):
    def np_or_none(t):
        return None if t is None else t.detach().cpu().numpy()

    return {
        "seq_lens": list(view.seq_lens_host),
        "block_table": np_or_none(view.block_table),
        "row_indptr": np_or_none(view.row_indptr),
        "row_req": np_or_none(view.row_req),
    }


def oracle_inputs(wl):
    return {
        "q_bits": host_bits(wl.q),
        "k_bits": host_bits(wl.k),
        "v_bits": host_bits(wl.v),
        "num_kv_heads": wl.num_kv_heads,
        "page_size": wl.page_size,
        "sm_scale": wl.sm_scale,
        "levels": [level_args(lv) for lv in wl.levels],
        "flat": level_args(wl.flat),
    }


def estimate(oi, rows=None):
    from oracle import estimate_level

    flat = oi["flat"]
    return estimate_level(oi["q_bits"], oi["k_bits"], num_kv_heads=oi["num_kv_heads"],
                          page_size=oi["page_size"], sm_scale=oi["sm_scale"],
                          seq_lens=flat["seq_lens"], block_table=flat["block_table"], rows=rows)


def decode(oi, z, T, splits, imposed=None):
    from oracle import decode as odecode

    return odecode(oi["q_bits"], oi["k_bits"], oi["v_bits"], num_kv_heads=oi["num_kv_heads"],
                   page_size=oi["page_size"], sm_scale=oi["sm_scale"], levels=oi["levels"],
                   z=z, T=T, splits=splits, imposed_x_per_level=imposed)


def bits_to_np(bits):
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)
