"""The C ABI library loads, exports every declared entry point, and rejects
invalid arguments on the host before launching anything (CPU only)."""

import ctypes
import math
import os
import re

import pytest

import paper_2609_33410_amd as F
from paper_2609_33410_amd import build_lib
from paper_2609_33410_amd.fold import fold_debug, fold_kv_view, fold_q_view

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(F.LIB_PATH):
        build_lib.build()
    return F.load_library()


def _declared():
    names = set()
    for h in sorted(os.listdir(os.path.join(ROOT, "include"))):
        if h.endswith(".h"):
            src = open(os.path.join(ROOT, "include", h)).read()
            src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
            names |= set(re.findall(r"\b(fold_[a-z0-9_]+)\s*\(", src))
    return sorted(names)


def test_every_declared_symbol_is_exported(lib):
    names = _declared()
    assert len(names) >= 14 and "fold_q8_decode_split" in names
    for n in names:
        assert hasattr(lib, n), n
    assert set(names) == set(F.EXPORTED)


def test_version_and_status_strings(lib):
    assert lib.fold_abi_version() == 2
    for code, word in ((0, b"FOLD_OK"), (1, b"FOLD_E_INVAL"), (2, b"FOLD_E_UNSUPPORTED"),
                       (3, b"FOLD_E_HIP")):
        assert lib.fold_status_string(code).startswith(word)


FAKE = 1 << 20  # a 16-byte aligned, never dereferenced address: validation fails first


def _kv(**over):
    kv = fold_kv_view()
    kv.k = kv.v = kv.seq_lens = FAKE
    kv.block_table = FAKE
    kv.num_seqs, kv.num_kv_heads, kv.head_dim = 2, 2, 128
    kv.page_size, kv.max_pages_per_seq, kv.num_pages = 16, 4, 8
    kv.max_seq_len, kv.max_reqs_per_seq = 64, 1
    for k, v in over.items():
        setattr(kv, k, v)
    return kv


def _q(**over):
    q = fold_q_view()
    q.q, q.batch, q.num_heads = FAKE, 2, 8
    for k, v in over.items():
        setattr(q, k, v)
    return q


def _decode(lib, kv, q, T=math.inf, splits=1, slot_offset=0, num_slots=1, z=FAKE):
    return lib.fold_decode_split(ctypes.byref(kv), ctypes.byref(q), 0.125, z, T, splits,
                                 slot_offset, num_slots, FAKE, FAKE, None, None, None)


@pytest.mark.parametrize("case", [
    ("head_dim", {"head_dim": 96}, {}),
    ("heads % kv_heads", {"num_kv_heads": 3}, {}),
    ("page_size", {"page_size": 8}, {}),
    ("misaligned k", {"k": FAKE + 2}, {}),
    ("misaligned q", {}, {"q": FAKE + 8}),
    ("null v", {"v": None}, {}),
    ("num_seqs > batch", {"num_seqs": 3}, {}),
    ("csr half set", {"row_indptr": FAKE}, {}),
])
def test_decode_rejects_bad_views(lib, case):
    _, kvo, qo = case
    assert _decode(lib, _kv(**kvo), _q(**qo)) == F.FOLD_E_INVAL
    assert len(lib.fold_last_error()) > 0


@pytest.mark.parametrize("kw", [
    {"T": float("nan")}, {"T": -1.0}, {"splits": 0}, {"slot_offset": 1, "num_slots": 1},
    {"z": None},
])
def test_decode_rejects_bad_call_args(lib, kw):
    assert _decode(lib, _kv(), _q(), **kw) == F.FOLD_E_INVAL


def test_estimate_rejects_csr_view_and_bad_params(lib):
    from paper_2609_33410_amd.fold import fold_est_params
    kv = _kv(row_indptr=FAKE, row_req=FAKE, max_reqs_per_seq=4)
    assert lib.fold_ref_estimate(ctypes.byref(kv), ctypes.byref(_q()), 0.1, None, FAKE,
                                 None) == F.FOLD_E_INVAL
    p = fold_est_params(1, 63, 128, 64, 64)
    assert lib.fold_ref_estimate(ctypes.byref(_kv()), ctypes.byref(_q()), 0.1, ctypes.byref(p),
                                 FAKE, None) == F.FOLD_E_INVAL
    p = fold_est_params(1, 63, 500, 8, 8)
    assert lib.fold_ref_estimate(ctypes.byref(_kv()), ctypes.byref(_q()), 0.1, ctypes.byref(p),
                                 FAKE, None) == F.FOLD_E_INVAL


def test_combine_rejects_bad_args(lib):
    c = lib.fold_combine
    assert c(FAKE, FAKE, 0, 4, 128, None, FAKE, 0, None, None, None, None) == F.FOLD_E_INVAL
    assert c(FAKE, FAKE, 2, 4, 80, None, FAKE, 0, None, None, None, None) == F.FOLD_E_INVAL
    assert c(FAKE, FAKE, 2, 4, 128, None, FAKE, 7, None, None, None, None) == F.FOLD_E_INVAL
    assert c(FAKE, FAKE, 2, 4, 128, None, FAKE, 0, FAKE, None, None, None) == F.FOLD_E_INVAL
    from paper_2609_33410_amd.fold import fold_value_model
    bad = (fold_value_model(None, FAKE, 8, 2), fold_value_model(FAKE, FAKE, 8, 3),
           fold_value_model(FAKE, FAKE, 6, 2))  # no masses; 8 % 3; 4 rows % 6
    for m in bad:
        assert c(FAKE, FAKE, 2, 4, 128, None, FAKE, 0, None, None, ctypes.byref(m),
                 None) == F.FOLD_E_INVAL


def test_value_mean_rejects_bad_args(lib):
    kv = _kv(row_indptr=FAKE, row_req=FAKE, max_reqs_per_seq=2)
    assert lib.fold_value_mean(ctypes.byref(kv), FAKE, None) == F.FOLD_E_INVAL
    assert lib.fold_value_mean(ctypes.byref(_kv(v=None)), FAKE, None) == F.FOLD_E_INVAL
    assert lib.fold_value_mean(ctypes.byref(_kv()), None, None) == F.FOLD_E_INVAL
    ap = lib.fold_value_mean_append
    assert ap(ctypes.byref(_kv()), FAKE, FAKE, FAKE, -1, FAKE, None) == F.FOLD_E_INVAL
    assert ap(ctypes.byref(_kv()), None, FAKE, FAKE, 3, FAKE, None) == F.FOLD_E_INVAL
    assert ap(ctypes.byref(_kv()), None, None, None, 0, None, None) == F.FOLD_OK


def _blocks(lib, kv=None, q=None, T=4.0, model="ok", dbg=None):
    from paper_2609_33410_amd.fold import fold_block_model
    m = fold_block_model(FAKE, 1, FAKE) if model == "ok" else model
    return lib.fold_decode_split_blocks(ctypes.byref(kv or _kv()), ctypes.byref(q or _q()), 0.125,
                                        FAKE, T, 1, 0, 1, FAKE, FAKE,
                                        None if m is None else ctypes.byref(m), dbg, None)


def test_block_model_decode_rejects_bad_args(lib):
    from paper_2609_33410_amd.fold import fold_block_model
    assert _blocks(lib, kv=_kv(head_dim=96)) == F.FOLD_E_INVAL          # the scan's checks
    assert _blocks(lib, T=float("nan")) == F.FOLD_E_INVAL
    assert _blocks(lib, model=None) == F.FOLD_E_INVAL                    # no model
    assert _blocks(lib, model=fold_block_model(None, 1, FAKE)) == F.FOLD_E_INVAL
    assert _blocks(lib, model=fold_block_model(FAKE, 0, FAKE)) == F.FOLD_E_INVAL  # 64 keys: 1 block
    assert _blocks(lib, kv=_kv(max_seq_len=65), model=fold_block_model(FAKE, 1, FAKE)) \
        == F.FOLD_E_INVAL                                                # 65 keys: 2 blocks
    assert _blocks(lib, model=fold_block_model(FAKE + 4, 1, FAKE)) == F.FOLD_E_INVAL  # misaligned
    assert _blocks(lib, model=fold_block_model(FAKE, 1, None)) == F.FOLD_E_INVAL  # finite T: workspace
    assert "chunk_cut" in lib.fold_last_error().decode()


def test_block_mean_rejects_bad_args(lib):
    bm = lib.fold_value_block_mean
    assert bm(ctypes.byref(_kv()), 0, FAKE, None) == F.FOLD_E_INVAL          # needs 1 block
    assert bm(ctypes.byref(_kv(max_seq_len=200)), 3, FAKE, None) == F.FOLD_E_INVAL  # needs 4
    assert bm(ctypes.byref(_kv()), 1, None, None) == F.FOLD_E_INVAL
    assert bm(ctypes.byref(_kv(v=None)), 1, FAKE, None) == F.FOLD_E_INVAL
    assert bm(ctypes.byref(_kv()), 1, FAKE + 8, None) == F.FOLD_E_INVAL      # misaligned
    assert bm(ctypes.byref(_kv(head_dim=80)), 1, FAKE, None) == F.FOLD_E_INVAL
    ap = lib.fold_value_block_mean_append
    assert ap(ctypes.byref(_kv()), 1, FAKE, FAKE, FAKE, -1, FAKE, None) == F.FOLD_E_INVAL
    assert ap(ctypes.byref(_kv()), 0, FAKE, FAKE, FAKE, 1, FAKE, None) == F.FOLD_E_INVAL
    assert ap(ctypes.byref(_kv()), 1, None, FAKE, FAKE, 3, FAKE, None) == F.FOLD_E_INVAL
    assert ap(ctypes.byref(_kv()), 1, None, None, None, 0, None, None) == F.FOLD_OK


def test_block_model_binding_checks_shapes_and_devices():
    import torch
    t = _fused_tensors()
    kv = F.kv_view(t["k"], t["v"], t["seq_lens"], num_kv_heads=t["k"].shape[1], max_seq_len=32,
                   block_table=t["block_table"])
    qv = F.q_view(t["q"])
    b, h = t["q"].shape[:2]
    z = torch.zeros(b, h)
    pa, pl = torch.zeros(1, b, h, 128), torch.zeros(1, b, h)
    mb = F.block_count(kv.view.max_seq_len)
    good = torch.zeros(kv.view.num_seqs, kv.view.num_kv_heads, mb, 128)
    cut = torch.zeros(b * h * F.chunk_count(kv.view.max_seq_len))
    with pytest.raises(ValueError, match="block_mean must be"):
        F.fold_decode_split_blocks(kv, qv, 0.1, z, 4.0, 1, 0, pa, pl, good[:, :, :, :64], cut)
    with pytest.raises(ValueError, match="blocks; the view needs"):
        F.fold_decode_split_blocks(kv, qv, 0.1, z, 4.0, 1, 0, pa, pl, good[:, :, :mb - 1], cut)
    with pytest.raises(ValueError, match="chunk_cut needs"):
        F.fold_decode_split_blocks(kv, qv, 0.1, z, 4.0, 1, 0, pa, pl, good, cut[:-1])
    with pytest.raises(ValueError, match="device tensor"):
        F.fold_decode_split_blocks(kv, qv, 0.1, z, 4.0, 1, 0, pa, pl, good, cut)
    with pytest.raises(ValueError, match="device tensor"):
        F.fold_value_block_mean(kv, good)


def test_q8_stacked_rejects_bad_args(lib):
    from paper_2609_33410_amd.fold import fold_q8_keys, fold_q8_query
    keys = fold_q8_keys(FAKE, FAKE, FAKE)
    sk = lib.fold_q8_stack_keys
    assert sk(ctypes.byref(_kv()), None, FAKE, None) == F.FOLD_E_INVAL
    assert sk(ctypes.byref(_kv()), ctypes.byref(keys), None, None) == F.FOLD_E_INVAL
    assert sk(ctypes.byref(_kv()), ctypes.byref(keys), FAKE + 2, None) == F.FOLD_E_INVAL
    assert sk(ctypes.byref(_kv(head_dim=96)), ctypes.byref(keys), FAKE, None) == F.FOLD_E_INVAL
    assert sk(ctypes.byref(_kv(num_seqs=0)), ctypes.byref(keys), None, None) == F.FOLD_OK
    q = fold_q8_query(FAKE, FAKE, None, 2, 8, None)
    ds = lib.fold_q8_decode_stacked

    def call(kv, qq=q, T=math.inf, z=FAKE, splits=1):
        return ds(ctypes.byref(kv), ctypes.byref(qq), z, T, splits, 0, 1, FAKE, FAKE, None, None,
                  None)
    # 8 heads over 2 kv heads, one request per sequence: 4 rows, not a stacked level
    assert call(_kv()) == F.FOLD_E_UNSUPPORTED
    wide = dict(row_indptr=FAKE, row_req=FAKE, max_reqs_per_seq=16)  # 64 rows per sequence
    assert call(_kv(v=None, **wide)) == F.FOLD_E_INVAL
    assert call(_kv(**wide), qq=fold_q8_query(None, FAKE, None, 2, 8, None)) == F.FOLD_E_INVAL
    assert call(_kv(**wide), z=None) == F.FOLD_E_INVAL
    assert call(_kv(**wide), T=-1.0) == F.FOLD_E_INVAL
    assert call(_kv(**wide), splits=0) == F.FOLD_E_INVAL
    assert call(_kv(k=FAKE + 2, **wide)) == F.FOLD_E_INVAL


def test_cascade_rejects_bad_args(lib):
    cd = lib.fold_decode_cascade
    wide = dict(row_indptr=FAKE, row_req=FAKE, max_reqs_per_seq=16)  # 64 rows per sequence

    def call(pre, suf, T=math.inf, z=FAKE, splits=1):
        return cd(ctypes.byref(pre), None if suf is None else ctypes.byref(suf),
                  ctypes.byref(_q()), 0.125, z, T, splits, 0, splits, FAKE, FAKE, None, None)
    assert call(_kv(**wide), None) == F.FOLD_E_INVAL
    assert call(_kv(**wide), _kv(), z=None) == F.FOLD_E_INVAL
    assert call(_kv(**wide), _kv(), T=-1.0) == F.FOLD_E_INVAL
    assert call(_kv(**wide), _kv(seq_lens=None)) == F.FOLD_E_INVAL
    # the prefix must be a stacked CSR level, the suffix a per-request view
    assert call(_kv(), _kv()) == F.FOLD_E_UNSUPPORTED
    assert call(_kv(**wide), _kv(**wide)) == F.FOLD_E_UNSUPPORTED
    assert call(_kv(**wide), _kv(num_seqs=1)) == F.FOLD_E_UNSUPPORTED
    # one cache and one paged layout
    assert call(_kv(**wide), _kv(k=FAKE + 16)) == F.FOLD_E_UNSUPPORTED
    assert call(_kv(**wide), _kv(v=FAKE + 16)) == F.FOLD_E_UNSUPPORTED
    assert call(_kv(**wide), _kv(page_size=32, max_pages_per_seq=2)) == F.FOLD_E_UNSUPPORTED
    assert call(_kv(**wide), _kv(num_pages=9)) == F.FOLD_E_UNSUPPORTED
    # at most 64 tiles per workgroup: 125 prefix tiles in one split
    long = dict(wide, max_seq_len=8000, max_pages_per_seq=500)
    assert call(_kv(**long), _kv()) == F.FOLD_E_UNSUPPORTED
    assert "raise num_splits" in lib.fold_last_error().decode()


def test_cascade_binding_checks_devices_and_slots():
    import torch
    t = _fused_tensors()
    kv = F.kv_view(t["k"], t["v"], t["seq_lens"], num_kv_heads=t["k"].shape[1], max_seq_len=32,
                   block_table=t["block_table"])
    qv = F.q_view(t["q"])
    b, h = t["q"].shape[:2]
    z = torch.zeros(b, h)
    pa, pl = torch.zeros(2, b, h, 128), torch.zeros(2, b, h)
    with pytest.raises(ValueError):
        F.fold_decode_cascade(kv, kv, qv, 0.1, z, 16.0, 2, 0, pa, pl[:1])
    with pytest.raises(ValueError, match="device tensor"):
        F.fold_decode_cascade(kv, kv, qv, 0.1, z, 16.0, 2, 0, pa, pl)


def test_row_group_queries(lib):
    kv = _kv()
    # GQA group of 4: one matrix-core read group of 16 rows
    assert lib.fold_decode_rows_per_group(ctypes.byref(kv), ctypes.byref(_q())) == 16
    assert lib.fold_decode_row_groups(ctypes.byref(kv), ctypes.byref(_q())) == 1
    # MHA: one row per read group (VALU scan)
    mha = _kv(num_kv_heads=8)
    assert lib.fold_decode_rows_per_group(ctypes.byref(mha), ctypes.byref(_q())) == 1
    # 64 requests x 8 heads stacked on one kv sequence: 512 rows in groups of 64
    csr = _kv(row_indptr=FAKE, row_req=FAKE, max_reqs_per_seq=64, num_kv_heads=1)
    assert lib.fold_decode_rows_per_group(ctypes.byref(csr), ctypes.byref(_q())) == 64
    assert lib.fold_decode_row_groups(ctypes.byref(csr), ctypes.byref(_q())) == 8
    # 4 requests x 8 heads: 32 rows, one matrix-core group; 5 requests: 40 rows, stacked
    csr4 = _kv(row_indptr=FAKE, row_req=FAKE, max_reqs_per_seq=4, num_kv_heads=1)
    assert lib.fold_decode_rows_per_group(ctypes.byref(csr4), ctypes.byref(_q())) == 32
    csr5 = _kv(row_indptr=FAKE, row_req=FAKE, max_reqs_per_seq=5, num_kv_heads=1)
    assert lib.fold_decode_rows_per_group(ctypes.byref(csr5), ctypes.byref(_q())) == 64
    assert lib.fold_decode_row_groups(ctypes.byref(csr5), ctypes.byref(_q())) == 1
    assert lib.fold_decode_row_groups(ctypes.byref(_kv(head_dim=5)), ctypes.byref(_q())) == -1


def test_binding_raises_when_library_missing(tmp_path):
    import importlib
    from paper_2609_33410_amd import fold as fmod
    saved = fmod._lib
    try:
        fmod._lib = None
        with pytest.raises(F.FoldLibraryMissing):
            fmod.load_library(str(tmp_path / "libfold.so"))
    finally:
        fmod._lib = saved


# ------------------------------------------------- two-plane INT8 key cache --
def _q8(kv_heads=2, heads=8, **over):
    from paper_2609_33410_amd.fold import fold_q8_keys, fold_q8_query
    keys = fold_q8_keys(FAKE, FAKE, FAKE)
    q = fold_q8_query(FAKE, FAKE, FAKE, 2, heads, FAKE)
    for k, v in over.items():
        setattr(keys if k in ("plane_a", "plane_b", "scale") else q, k, v)
    return keys, q


def _q8_decode(lib, kv, keys, q, T=math.inf, splits=1, z=FAKE):
    return lib.fold_q8_decode_split(ctypes.byref(kv), ctypes.byref(keys), ctypes.byref(q), None,
                                    z, T, splits, 0, splits, FAKE, FAKE, None, None, None)


@pytest.mark.parametrize("over,kvo,want", [
    ({"plane_b": None}, {}, F.FOLD_E_INVAL),
    ({"scale": FAKE + 2}, {}, F.FOLD_E_INVAL),
    ({"planes": FAKE + 4}, {}, F.FOLD_E_INVAL),
    ({"tau": None}, {}, F.FOLD_E_INVAL),
    ({"eta": None}, {}, F.FOLD_E_INVAL),
    ({}, {"v": None}, F.FOLD_E_INVAL),
    ({"num_heads": 6}, {}, F.FOLD_E_UNSUPPORTED),     # GQA group 3
    ({"num_heads": 128}, {}, F.FOLD_E_UNSUPPORTED),   # GQA group 64
])
def test_q8_decode_rejects_bad_args(lib, over, kvo, want):
    keys, q = _q8(**over)
    kv = _kv(**kvo)
    kv.k = None                     # the two-plane calls never read the BF16 key pointer
    assert _q8_decode(lib, kv, keys, q) == want
    assert len(lib.fold_last_error()) > 0


def test_q8_decode_rejects_bad_depth_and_split(lib):
    keys, q = _q8()
    assert _q8_decode(lib, _kv(), keys, q, T=float("nan")) == F.FOLD_E_INVAL
    assert _q8_decode(lib, _kv(), keys, q, splits=0) == F.FOLD_E_INVAL
    assert _q8_decode(lib, _kv(), keys, q, z=None) == F.FOLD_E_INVAL


def test_q8_front_rejects_bad_args(lib):
    kv = _kv()
    # writer: a token list without planes; negative count
    assert lib.fold_q8_write_keys(ctypes.byref(kv), FAKE, FAKE, FAKE, 4, None, FAKE, FAKE,
                                  None) == F.FOLD_E_INVAL
    assert lib.fold_q8_write_keys(ctypes.byref(kv), FAKE, FAKE, FAKE, -1, FAKE, FAKE, FAKE,
                                  None) == F.FOLD_E_INVAL
    assert lib.fold_q8_write_keys(ctypes.byref(_kv(page_size=8)), FAKE, FAKE, FAKE, 4, FAKE,
                                  FAKE, FAKE, None) == F.FOLD_E_INVAL
    # an empty token list is a valid no-op
    assert lib.fold_q8_write_keys(ctypes.byref(kv), None, None, None, 0, None, None, None,
                                  None) == F.FOLD_OK
    q = _q()
    split = lib.fold_q8_split_query
    assert split(ctypes.byref(q), 96, 0.1, None, 0.0, 0.0, FAKE, FAKE, None, None,
                 None) == F.FOLD_E_INVAL
    assert split(ctypes.byref(q), 128, 0.1, FAKE, 0.0, 0.0, FAKE, FAKE, None, None,
                 None) == F.FOLD_E_INVAL
    assert split(ctypes.byref(q), 128, 0.1, FAKE, float("nan"), 0.0, FAKE, FAKE, FAKE, None,
                 None) == F.FOLD_E_INVAL
    assert split(ctypes.byref(q), 128, 0.1, FAKE, 0.0, float("nan"), FAKE, FAKE, FAKE, None,
                 None) == F.FOLD_E_INVAL
    assert split(ctypes.byref(q), 128, 0.1, None, 0.0, 0.0, FAKE, FAKE, None, FAKE,
                 None) == F.FOLD_E_INVAL   # tau_v without lengths
    assert split(ctypes.byref(q), 128, float("inf"), None, 0.0, 0.0, FAKE, FAKE, None, None,
                 None) == F.FOLD_E_INVAL
    from paper_2609_33410_amd.fold import fold_v8_values
    keys8, q88 = _q8(tau_v=None)
    v8 = fold_v8_values(FAKE, FAKE, 0)
    kvv = _kv()
    assert lib.fold_q8_decode_split(ctypes.byref(kvv), ctypes.byref(keys8), ctypes.byref(q88),
                                    ctypes.byref(v8), FAKE, math.inf, 1, 0, 1, FAKE, FAKE, None,
                                    None, None) == F.FOLD_E_INVAL   # no tau_v
    keys8, q88 = _q8()
    v8 = fold_v8_values(FAKE + 1, FAKE, 0)
    assert lib.fold_q8_decode_split(ctypes.byref(kvv), ctypes.byref(keys8), ctypes.byref(q88),
                                    ctypes.byref(v8), FAKE, math.inf, 1, 0, 1, FAKE, FAKE, None,
                                    None, None) == F.FOLD_E_INVAL   # misaligned plane
    assert lib.fold_v8_write_values(ctypes.byref(kvv), FAKE, FAKE, FAKE, 2, 500, FAKE, FAKE,
                                    None) == F.FOLD_E_INVAL   # scale exponent
    assert lib.fold_v8_write_values(ctypes.byref(kvv), FAKE, FAKE, FAKE, 2, 0, None, FAKE,
                                    None) == F.FOLD_E_INVAL
    keys, q8 = _q8()
    csr = _kv(row_indptr=FAKE, row_req=FAKE, max_reqs_per_seq=4)
    assert lib.fold_q8_ref_estimate(ctypes.byref(csr), ctypes.byref(keys), ctypes.byref(q8), None,
                                    FAKE, None) == F.FOLD_E_INVAL


def test_q8_row_group_queries(lib):
    keys, q = _q8()
    kv = _kv()
    assert lib.fold_q8_decode_rows_per_group(ctypes.byref(kv), ctypes.byref(q)) == 16
    assert lib.fold_q8_decode_row_groups(ctypes.byref(kv), ctypes.byref(q)) == 1
    # 64 requests x 8 heads stacked on one kv sequence: groups of 32 rows (whole GQA groups)
    csr = _kv(row_indptr=FAKE, row_req=FAKE, max_reqs_per_seq=64, num_kv_heads=1)
    assert lib.fold_q8_decode_rows_per_group(ctypes.byref(csr), ctypes.byref(q)) == 32
    assert lib.fold_q8_decode_row_groups(ctypes.byref(csr), ctypes.byref(q)) == 16
    assert lib.fold_q8_decode_row_groups(ctypes.byref(_kv(head_dim=5)), ctypes.byref(q)) == -1
    # one row per kv sequence and head (MHA): read groups of one row
    mha = _kv(num_kv_heads=8)
    assert lib.fold_q8_decode_rows_per_group(ctypes.byref(mha), ctypes.byref(q)) == 1
    assert lib.fold_q8_decode_row_groups(ctypes.byref(mha), ctypes.byref(q)) == 1


# ------------------------------------------------------------- the step ----
def _i32(xs):
    import torch
    return torch.tensor(xs, dtype=torch.int32)


def test_append_and_cert_reject_bad_args(lib):
    kv = _kv()
    V = ctypes.c_void_p
    # a written cache needs its sources; tokens need their lists
    assert lib.fold_append_kv(ctypes.byref(kv), None, None, V(FAKE), V(FAKE), 3, V(FAKE), None,
                              None) == F.FOLD_E_INVAL
    assert lib.fold_append_kv(ctypes.byref(kv), V(FAKE), V(FAKE), None, V(FAKE), 3, V(FAKE),
                              V(FAKE), None) == F.FOLD_E_INVAL
    assert lib.fold_append_kv(ctypes.byref(kv), V(FAKE + 4), V(FAKE), V(FAKE), V(FAKE), 3,
                              V(FAKE), V(FAKE), None) == F.FOLD_E_INVAL      # misaligned
    assert lib.fold_append_kv(ctypes.byref(_kv(head_dim=96)), V(FAKE), V(FAKE), V(FAKE), V(FAKE),
                              3, V(FAKE), V(FAKE), None) == F.FOLD_E_INVAL
    assert lib.fold_append_kv(ctypes.byref(kv), V(FAKE), V(FAKE), V(FAKE), V(FAKE), -1,
                              V(FAKE), V(FAKE), None) == F.FOLD_E_INVAL
    assert lib.fold_cert_update(V(FAKE), V(FAKE), V(FAKE), 4, None, None, None) == F.FOLD_E_INVAL
    assert lib.fold_cert_update(None, V(FAKE), V(FAKE), 4, None, V(FAKE), None) == F.FOLD_E_INVAL
    assert lib.fold_cert_update(V(FAKE), V(FAKE), V(FAKE), -1, None, V(FAKE),
                                None) == F.FOLD_E_INVAL


def _plan(lib, seq_lens, indptr, parent, page=16, ppc=1):
    import torch
    b = len(seq_lens)
    cols = indptr[-1]
    out = [torch.full((b,), -7, dtype=torch.int32)] + \
          [torch.full((cols,), -7, dtype=torch.int32) for _ in range(3)] + \
          [torch.full((cols, page * ppc), -7, dtype=torch.int32)]
    sl, ind, par = _i32(seq_lens), _i32(indptr), _i32(parent if parent else [0])
    st = lib.fold_draft_plan(b, sl.data_ptr(), ind.data_ptr(), par.data_ptr(), page, ppc,
                             *[t.data_ptr() for t in out])
    return st, out


def test_draft_plan_matches_the_oracle_visible_sets(lib):
    """The host plan's ancestor positions are the draft part of the oracle's
    visible set for every column of a chain and two trees."""
    from oracle import step_oracle as st_oracle
    parents = [[-1, 0, 1, 2], [-1, 0, 0, 1, 2, 2, 3, -1], [-1]]
    seq_lens = [40, 100, 3]
    indptr = [0, 4, 12, 13]
    st, (committed, col_req, col_lens, anc_lens, anc_pos) = _plan(
        lib, seq_lens, indptr, [p for ps in parents for p in ps])
    assert st == F.FOLD_OK
    assert committed.tolist() == [36, 92, 2]
    for r, ps in enumerate(parents):
        n, m = seq_lens[r], len(ps)
        for c in range(m):
            col = indptr[r] + c
            vis = st_oracle.draft_visible(n, m, ps, c)
            anc = vis[vis >= n - m].tolist()
            assert col_req[col] == r and col_lens[col] == n - m
            assert anc_lens[col] == len(anc)
            assert anc_pos[col, :len(anc)].tolist() == anc
            assert (anc_pos[col, len(anc):] == -1).all()


@pytest.mark.parametrize("seq_lens, indptr, parent", [
    ([10, 10], [1, 2, 3], [-1, -1, -1]),        # col_indptr[0] != 0
    ([10, 10], [0, 2, 1], [-1, 0]),             # decreasing
    ([1, 10], [0, 2, 3], [-1, 0, -1]),          # more drafts than keys
    ([10], [0, 3], [-1, 2, 0]),                 # parent not before its child
    ([10], [0, 2], [-1, -2]),                   # parent below -1
    ([40], [0, 17], [-1] + list(range(16))),    # 17 ancestors, 16 spare slots
])
def test_draft_plan_rejects_bad_trees(lib, seq_lens, indptr, parent):
    st, outs = _plan(lib, seq_lens, indptr, parent)
    assert st == F.FOLD_E_INVAL
    assert all((t == -7).all() for t in outs)  # nothing written


def test_draft_gather_rejects_bad_args(lib):
    V = ctypes.c_void_p
    kv = _kv()
    args = [V(FAKE)] * 4
    assert lib.fold_draft_gather(ctypes.byref(_kv(block_table=None)), *args, 2, 1, 256, V(FAKE),
                                 V(FAKE), None, None) == F.FOLD_E_INVAL      # contiguous view
    assert lib.fold_draft_gather(ctypes.byref(kv), *args, 2, 0, 256, V(FAKE), V(FAKE), None,
                                 None) == F.FOLD_E_INVAL                    # pages_per_col
    assert lib.fold_draft_gather(ctypes.byref(kv), *args, 2, 1, 0, V(FAKE), V(FAKE), None,
                                 None) == F.FOLD_E_INVAL                    # row_bytes
    assert lib.fold_draft_gather(ctypes.byref(kv), *args, 2, 1, 256, V(FAKE), None, None,
                                 None) == F.FOLD_E_INVAL                    # src without dst
    assert lib.fold_draft_gather(ctypes.byref(kv), *args, 2, 1, 256, V(FAKE + 2), V(FAKE), None,
                                 None) == F.FOLD_E_INVAL                    # misaligned rows
    assert lib.fold_draft_gather(ctypes.byref(kv), None, V(FAKE), V(FAKE), V(FAKE), 2, 1, 256,
                                 V(FAKE), V(FAKE), None, None) == F.FOLD_E_INVAL


# ------------------------------------------------------ one-launch decodes --
def _fused(lib, kv=None, q=None, T=math.inf, splits=2, part_a=FAKE, arrivals=FAKE, out=FAKE,
           out_dtype=0):
    return lib.fold_decode_fused(ctypes.byref(kv or _kv()), ctypes.byref(q or _q()), 0.125, None,
                                 T, splits, part_a, FAKE, arrivals, FAKE, out, out_dtype, None,
                                 None, None)


@pytest.mark.parametrize("kw,want", [
    ({"arrivals": None}, F.FOLD_E_INVAL),
    ({"T": float("nan")}, F.FOLD_E_INVAL),
    ({"splits": 0}, F.FOLD_E_INVAL),
    ({"out_dtype": 7}, F.FOLD_E_INVAL),
    ({"out": FAKE + 4}, F.FOLD_E_INVAL),                  # misaligned output
    ({"part_a": FAKE + 8}, F.FOLD_E_INVAL),               # misaligned slots
    ({"q": _q(num_heads=2)}, F.FOLD_E_UNSUPPORTED),       # MHA
    ({"q": _q(num_heads=32)}, F.FOLD_E_UNSUPPORTED),      # groups of 16 rows
    ({"kv": _kv(num_seqs=1)}, F.FOLD_E_INVAL),            # num_seqs != batch
    ({"kv": _kv(row_indptr=FAKE, row_req=FAKE, max_reqs_per_seq=2)}, F.FOLD_E_INVAL),
    ({"splits": 1 << 20}, F.FOLD_E_UNSUPPORTED),          # slots of 8 GiB
])
def test_fused_decode_rejects_bad_args(lib, kw, want):
    """Every refusal happens in validation, before anything is launched."""
    assert _fused(lib, **kw) == want
    assert len(lib.fold_last_error()) > 0




# ------------------------------------- binding checks of the one-launch calls --
def _fused_tensors(b=2, h=8, hkv=2, d=128, slots=2, npages=4):
    import torch

    bf = torch.bfloat16
    t = {
        "q": torch.zeros(b, h, d, dtype=bf),
        "k": torch.zeros(npages, hkv, 16, d, dtype=bf),
        "v": torch.zeros(npages, hkv, 16, d, dtype=bf),
        "seq_lens": torch.full((b,), 32, dtype=torch.int32),
        "block_table": torch.zeros(b, 2, dtype=torch.int32),
        "part_A": torch.zeros(slots, b, h, d),
        "part_L": torch.zeros(slots, b, h),
        "arrivals": torch.zeros(b, hkv, dtype=torch.int32),
        "z_out": torch.zeros(b, h),
        "out": torch.zeros(b, h, d),
        "lse_out": torch.zeros(b, h),
        "cert_out": torch.zeros(b, h, dtype=torch.uint8),
    }
    return t


def _call_fused(t, splits=2):
    kv = F.kv_view(t["k"], t["v"], t["seq_lens"], num_kv_heads=t["k"].shape[1],
                   max_seq_len=32, block_table=t["block_table"])
    return F.fold_decode_fused(kv, F.q_view(t["q"]), 0.125, math.inf, splits, t["part_A"],
                               t["part_L"], t["arrivals"], t["z_out"], t["out"],
                               lse_out=t["lse_out"], cert_out=t["cert_out"])


@pytest.mark.parametrize("name,shape,match", [
    ("arrivals", (3,), "arrivals needs"),
    ("part_A", (2, 2, 8, 64), "part_A must be"),
    ("part_A", (2, 1, 8, 128), "part_A must be"),
    ("part_L", (2, 2, 4), "part_L must be"),
    ("part_L", (1, 2, 8), "num_splits slots"),
    ("z_out", (2, 7), "z_out needs"),
    ("out", (2, 8, 127), "out needs"),
    ("lse_out", (15,), "lse_out needs"),
    ("cert_out", (1, 8), "cert_out needs"),
])
def test_fused_binding_rejects_short_workspace(name, shape, match):
    """The binding refuses a workspace or output too small for the view and
    the query before the library is called (a short tensor would be written
    past its end)."""
    import torch

    t = _fused_tensors()
    t[name] = torch.zeros(shape, dtype=t[name].dtype)
    with pytest.raises(ValueError, match=match):
        _call_fused(t)


def test_fused_binding_rejects_host_tensors():
    """Correctly sized host tensors are refused as not in device memory."""
    with pytest.raises(ValueError, match="device tensor"):
        _call_fused(_fused_tensors())


# --------------------------------------------- one-launch decode, no allocation --
def _noalloc(lib, kv=None, q=None, T=math.inf, splits=2, z=FAKE, out=FAKE, out_dtype=0):
    return lib.fold_decode_fused_noalloc(None if kv is False else ctypes.byref(kv or _kv()),
                                         ctypes.byref(q or _q()), 0.125, None, T, splits, z, out,
                                         out_dtype, None, None, None)


@pytest.mark.parametrize("kw,want,text", [
    ({"splits": 4096}, F.FOLD_E_INVAL, "scratch"),            # 33.8 MB of slots > 8 MiB
    ({"splits": 1 << 21}, F.FOLD_E_INVAL, "scratch"),
    ({"q": _q(batch=1 << 20, num_heads=8), "kv": _kv(num_seqs=1 << 20)}, F.FOLD_E_INVAL, "scratch"),
    ({"splits": 0}, F.FOLD_E_INVAL, "num_splits"),
    ({"T": float("nan")}, F.FOLD_E_INVAL, ""),
    ({"z": None}, F.FOLD_E_INVAL, ""),
    ({"out": FAKE + 4}, F.FOLD_E_INVAL, "aligned"),
    ({"out_dtype": 7}, F.FOLD_E_INVAL, ""),
    ({"kv": False}, F.FOLD_E_INVAL, ""),
    ({"q": _q(num_heads=2)}, F.FOLD_E_UNSUPPORTED, ""),       # MHA
    ({"kv": _kv(num_seqs=1)}, F.FOLD_E_INVAL, ""),            # num_seqs != batch
])
def test_noalloc_decode_rejects_before_touching_the_device(lib, kw, want, text):
    """Every refusal (scratch too small included) happens on the host before
    the scratch address is looked up or anything is launched: these calls run
    here without a GPU."""
    assert _noalloc(lib, **kw) == want
    msg = lib.fold_last_error().decode()
    assert len(msg) > 0 and text in msg
