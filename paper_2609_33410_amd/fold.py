"""ctypes binding of ``libfold.so`` (the C ABI in ``include/fold.h``,
``include/fold_q8.h`` and ``include/fold_draft.h``).

Argument marshalling only: torch tensors supply device memory and
``torch.cuda.current_stream()`` supplies the HIP stream; every step of the
decode path runs in the library's HIP kernels.  The library must be built
(``python -m paper_2609_33410_amd.build_lib``); without it every entry point
raises ``FoldLibraryMissing``.  There is no fallback.
"""

from __future__ import annotations

import ctypes
import math
import os
from dataclasses import dataclass
from typing import Optional

import torch

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libfold.so")

FOLD_OK, FOLD_E_INVAL, FOLD_E_UNSUPPORTED, FOLD_E_HIP = 0, 1, 2, 3
FOLD_DTYPE_F32, FOLD_DTYPE_BF16 = 0, 1

EXPORTED = (
    "fold_abi_version",
    "fold_status_string",
    "fold_last_error",
    "fold_decode_rows_per_group",
    "fold_decode_row_groups",
    "fold_ref_estimate",
    "fold_decode_split",
    "fold_combine",
    "fold_decode_fused",
    "fold_decode_fused_noalloc",
    "fold_value_mean",
    "fold_value_mean_append",
    "fold_value_block_mean",
    "fold_value_block_mean_append",
    "fold_decode_split_blocks",
    "fold_decode_cascade",
    "fold_q8_write_keys",
    "fold_v8_write_values",
    "fold_q8_split_query",
    "fold_q8_ref_estimate",
    "fold_q8_front",
    "fold_q8_decode_rows_per_group",
    "fold_q8_decode_row_groups",
    "fold_q8_decode_split",
    "fold_q8_stack_keys",
    "fold_q8_decode_stacked",
    "fold_append_kv",
    "fold_cert_update",
    "fold_draft_plan",
    "fold_draft_gather",
)


class FoldLibraryMissing(RuntimeError):
    pass


class FoldError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(message)
        self.status = status


class fold_kv_view(ctypes.Structure):
    _fields_ = [
        ("k", ctypes.c_void_p),
        ("v", ctypes.c_void_p),
        ("block_table", ctypes.c_void_p),
        ("seq_lens", ctypes.c_void_p),
        ("row_indptr", ctypes.c_void_p),
        ("row_req", ctypes.c_void_p),
        ("num_seqs", ctypes.c_int32),
        ("num_kv_heads", ctypes.c_int32),
        ("head_dim", ctypes.c_int32),
        ("page_size", ctypes.c_int32),
        ("max_pages_per_seq", ctypes.c_int32),
        ("num_pages", ctypes.c_int32),
        ("max_seq_len", ctypes.c_int32),
        ("max_reqs_per_seq", ctypes.c_int32),
    ]


class fold_q_view(ctypes.Structure):
    _fields_ = [("q", ctypes.c_void_p), ("batch", ctypes.c_int32), ("num_heads", ctypes.c_int32)]


class fold_est_params(ctypes.Structure):
    _fields_ = [("sink", ctypes.c_int32), ("recent", ctypes.c_int32), ("strata", ctypes.c_int32),
                ("trim_lo", ctypes.c_int32), ("trim_hi", ctypes.c_int32)]


class fold_debug(ctypes.Structure):
    _fields_ = [("x_out", ctypes.c_void_p), ("key_gate_out", ctypes.c_void_p),
                ("page_gate_out", ctypes.c_void_p)]


class fold_value_model(ctypes.Structure):
    _fields_ = [("part_Lcut", ctypes.c_void_p), ("mean", ctypes.c_void_p),
                ("num_heads", ctypes.c_int32), ("num_kv_heads", ctypes.c_int32)]


class fold_block_model(ctypes.Structure):
    _fields_ = [("block_mean", ctypes.c_void_p), ("max_blocks", ctypes.c_int32),
                ("chunk_cut", ctypes.c_void_p)]


class fold_q8_keys(ctypes.Structure):
    _fields_ = [("plane_a", ctypes.c_void_p), ("plane_b", ctypes.c_void_p),
                ("scale", ctypes.c_void_p)]


class fold_q8_query(ctypes.Structure):
    _fields_ = [("planes", ctypes.c_void_p), ("eta", ctypes.c_void_p), ("tau", ctypes.c_void_p),
                ("batch", ctypes.c_int32), ("num_heads", ctypes.c_int32),
                ("tau_v", ctypes.c_void_p)]


class fold_v8_values(ctypes.Structure):
    _fields_ = [("plane_p", ctypes.c_void_p), ("plane_r", ctypes.c_void_p),
                ("scale_exp", ctypes.c_int32)]


class fold_q8_debug(ctypes.Structure):
    _fields_ = [("x_out", ctypes.c_void_p), ("xc_out", ctypes.c_void_p),
                ("key_gate_out", ctypes.c_void_p), ("page_gate_out", ctypes.c_void_p),
                ("refine_gate_out", ctypes.c_void_p), ("refine_v_gate_out", ctypes.c_void_p)]


_lib = None


def load_library(path: str = LIB_PATH) -> ctypes.CDLL:
    """Load the library once.  torch is imported first so that the library
    binds to the HIP runtime torch already loaded (same soname)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise FoldLibraryMissing(
            f"{path} is not built; run `python -m paper_2609_33410_amd.build_lib`")
    lib = ctypes.CDLL(path)
    P = ctypes.POINTER
    lib.fold_abi_version.restype = ctypes.c_int
    lib.fold_abi_version.argtypes = []
    lib.fold_status_string.restype = ctypes.c_char_p
    lib.fold_status_string.argtypes = [ctypes.c_int]
    lib.fold_last_error.restype = ctypes.c_char_p
    lib.fold_last_error.argtypes = []
    for name in ("fold_decode_rows_per_group", "fold_decode_row_groups"):
        fn = getattr(lib, name)
        fn.restype = ctypes.c_int32
        fn.argtypes = [P(fold_kv_view), P(fold_q_view)]
    lib.fold_ref_estimate.restype = ctypes.c_int
    lib.fold_ref_estimate.argtypes = [P(fold_kv_view), P(fold_q_view), ctypes.c_float,
                                      P(fold_est_params), ctypes.c_void_p, ctypes.c_void_p]
    lib.fold_decode_split.restype = ctypes.c_int
    lib.fold_decode_split.argtypes = [P(fold_kv_view), P(fold_q_view), ctypes.c_float,
                                      ctypes.c_void_p, ctypes.c_float, ctypes.c_int32,
                                      ctypes.c_int32, ctypes.c_int32, ctypes.c_void_p,
                                      ctypes.c_void_p, ctypes.c_void_p, P(fold_debug),
                                      ctypes.c_void_p]
    lib.fold_decode_split_blocks.restype = ctypes.c_int
    lib.fold_decode_cascade.argtypes = [P(fold_kv_view), P(fold_kv_view), P(fold_q_view),
                                        ctypes.c_float, ctypes.c_void_p, ctypes.c_float,
                                        ctypes.c_int32, ctypes.c_int32, ctypes.c_int32,
                                        ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                                        ctypes.c_void_p]
    lib.fold_decode_cascade.restype = ctypes.c_int
    lib.fold_decode_split_blocks.argtypes = [P(fold_kv_view), P(fold_q_view), ctypes.c_float,
                                             ctypes.c_void_p, ctypes.c_float, ctypes.c_int32,
                                             ctypes.c_int32, ctypes.c_int32, ctypes.c_void_p,
                                             ctypes.c_void_p, P(fold_block_model),
                                             P(fold_debug), ctypes.c_void_p]
    lib.fold_value_block_mean.restype = ctypes.c_int
    lib.fold_value_block_mean.argtypes = [P(fold_kv_view), ctypes.c_int32, ctypes.c_void_p,
                                          ctypes.c_void_p]
    lib.fold_value_block_mean_append.restype = ctypes.c_int
    lib.fold_value_block_mean_append.argtypes = [P(fold_kv_view), ctypes.c_int32,
                                                 ctypes.c_void_p, ctypes.c_void_p,
                                                 ctypes.c_void_p, ctypes.c_int32,
                                                 ctypes.c_void_p, ctypes.c_void_p]
    lib.fold_combine.restype = ctypes.c_int
    lib.fold_combine.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int32, ctypes.c_int32,
                                 ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int,
                                 ctypes.c_void_p, ctypes.c_void_p, P(fold_value_model),
                                 ctypes.c_void_p]
    lib.fold_decode_fused.restype = ctypes.c_int
    lib.fold_decode_fused.argtypes = [P(fold_kv_view), P(fold_q_view), ctypes.c_float,
                                      P(fold_est_params), ctypes.c_float, ctypes.c_int32,
                                      ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                                      ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int,
                                      ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p]
    lib.fold_decode_fused_noalloc.restype = ctypes.c_int
    lib.fold_decode_fused_noalloc.argtypes = [P(fold_kv_view), P(fold_q_view), ctypes.c_float,
                                              P(fold_est_params), ctypes.c_float, ctypes.c_int32,
                                              ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int,
                                              ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p]
    lib.fold_value_mean.restype = ctypes.c_int
    lib.fold_value_mean.argtypes = [P(fold_kv_view), ctypes.c_void_p, ctypes.c_void_p]
    lib.fold_value_mean_append.restype = ctypes.c_int
    lib.fold_value_mean_append.argtypes = [P(fold_kv_view), ctypes.c_void_p, ctypes.c_void_p,
                                           ctypes.c_void_p, ctypes.c_int32, ctypes.c_void_p,
                                           ctypes.c_void_p]
    lib.fold_q8_write_keys.restype = ctypes.c_int
    lib.fold_q8_write_keys.argtypes = [P(fold_kv_view), ctypes.c_void_p, ctypes.c_void_p,
                                       ctypes.c_void_p, ctypes.c_int32, ctypes.c_void_p,
                                       ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p]
    lib.fold_q8_split_query.restype = ctypes.c_int
    lib.fold_q8_split_query.argtypes = [P(fold_q_view), ctypes.c_int32, ctypes.c_float,
                                        ctypes.c_void_p, ctypes.c_float, ctypes.c_float,
                                        ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                                        ctypes.c_void_p, ctypes.c_void_p]
    lib.fold_v8_write_values.restype = ctypes.c_int
    lib.fold_v8_write_values.argtypes = [P(fold_kv_view), ctypes.c_void_p, ctypes.c_void_p,
                                         ctypes.c_void_p, ctypes.c_int32, ctypes.c_int32,
                                         ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p]
    lib.fold_q8_ref_estimate.restype = ctypes.c_int
    lib.fold_q8_ref_estimate.argtypes = [P(fold_kv_view), P(fold_q8_keys), P(fold_q8_query),
                                         P(fold_est_params), ctypes.c_void_p, ctypes.c_void_p]
    lib.fold_q8_front.restype = ctypes.c_int
    lib.fold_q8_front.argtypes = [P(fold_kv_view), P(fold_q8_keys), P(fold_q_view), ctypes.c_float,
                                  ctypes.c_void_p, ctypes.c_float, ctypes.c_float,
                                  ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                                  ctypes.c_void_p, P(fold_est_params), ctypes.c_void_p,
                                  ctypes.c_void_p]
    for name in ("fold_q8_decode_rows_per_group", "fold_q8_decode_row_groups"):
        fn = getattr(lib, name)
        fn.restype = ctypes.c_int32
        fn.argtypes = [P(fold_kv_view), P(fold_q8_query)]
    lib.fold_q8_decode_split.restype = ctypes.c_int
    lib.fold_q8_decode_split.argtypes = [P(fold_kv_view), P(fold_q8_keys), P(fold_q8_query),
                                         P(fold_v8_values),
                                         ctypes.c_void_p, ctypes.c_float, ctypes.c_int32,
                                         ctypes.c_int32, ctypes.c_int32, ctypes.c_void_p,
                                         ctypes.c_void_p, ctypes.c_void_p, P(fold_q8_debug),
                                         ctypes.c_void_p]
    lib.fold_q8_stack_keys.restype = ctypes.c_int
    lib.fold_q8_stack_keys.argtypes = [P(fold_kv_view), P(fold_q8_keys), ctypes.c_void_p,
                                       ctypes.c_void_p]
    lib.fold_q8_decode_stacked.restype = ctypes.c_int
    lib.fold_q8_decode_stacked.argtypes = [P(fold_kv_view), P(fold_q8_query), ctypes.c_void_p,
                                           ctypes.c_float, ctypes.c_int32, ctypes.c_int32,
                                           ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p,
                                           ctypes.c_void_p, P(fold_debug), ctypes.c_void_p]
    V = ctypes.c_void_p
    I32 = ctypes.c_int32
    lib.fold_append_kv.restype = ctypes.c_int
    lib.fold_append_kv.argtypes = [P(fold_kv_view), V, V, V, V, I32, V, V, V]
    lib.fold_cert_update.restype = ctypes.c_int
    lib.fold_cert_update.argtypes = [V, V, V, I32, V, V, V]
    lib.fold_draft_plan.restype = ctypes.c_int
    lib.fold_draft_plan.argtypes = [I32, V, V, V, I32, I32, V, V, V, V, V]
    lib.fold_draft_gather.restype = ctypes.c_int
    lib.fold_draft_gather.argtypes = [P(fold_kv_view), V, V, V, V, I32, I32, I32, V, V, V, V]
    _lib = lib
    return lib


def _check(status: int) -> None:
    if status != FOLD_OK:
        lib = load_library()
        msg = lib.fold_last_error().decode(errors="replace")
        raise FoldError(status, f"{lib.fold_status_string(status).decode()}: {msg}")


def _ptr(t: Optional[torch.Tensor]) -> Optional[int]:
    return None if t is None else t.data_ptr()


def _stream(stream) -> Optional[int]:
    if stream is None:
        stream = torch.cuda.current_stream()
    return stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream)


def _need(t: torch.Tensor, name: str, dtype: torch.dtype) -> None:
    if t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")


def _need_device(named) -> None:
    """Every tensor handed to a launch must live in device memory."""
    for nm, t in named:
        if t is not None and not t.is_cuda:
            raise ValueError(f"{nm} must be a device tensor")


def _slot_checks(q: torch.Tensor, part_A: torch.Tensor, part_L: torch.Tensor,
                 part_Lcut: Optional[torch.Tensor], z: Optional[torch.Tensor]) -> None:
    """Slots are [slots, B, H, D] / [slots, B, H] for the query [B, H, D]."""
    b, h, d = (int(x) for x in q.shape)
    if part_A.dim() != 4 or tuple(part_A.shape[1:]) != (b, h, d):
        raise ValueError(f"part_A must be [slots, {b}, {h}, {d}], got {tuple(part_A.shape)}")
    for t, nm in ((part_L, "part_L"), (part_Lcut, "part_Lcut")):
        if t is not None and (t.dim() != 3 or tuple(t.shape) != (int(part_A.shape[0]), b, h)):
            raise ValueError(f"{nm} must be [{int(part_A.shape[0])}, {b}, {h}], "
                             f"got {tuple(t.shape)}")
    if z is not None and z.numel() < b * h:
        raise ValueError(f"z needs {b * h} elements, got {z.numel()}")


def _fused_checks(kv: KV, q: torch.Tensor, num_splits: int, part_A: torch.Tensor,
                  part_L: torch.Tensor, arrivals: torch.Tensor, z_out: torch.Tensor,
                  out: torch.Tensor, lse_out: Optional[torch.Tensor],
                  cert_out: Optional[torch.Tensor], extra=()) -> None:
    """Sizes of the one-launch decodes' workspace and outputs: the kernels
    write every slot, arrival count and output row the view and the query
    imply, so a short tensor would be written past its end."""
    b, h, d = (int(x) for x in q.shape)
    if part_A.dim() != 4 or tuple(part_A.shape[1:]) != (b, h, d):
        raise ValueError(f"part_A must be [slots, {b}, {h}, {d}], got {tuple(part_A.shape)}")
    if part_L.dim() != 3 or tuple(part_L.shape[1:]) != (b, h):
        raise ValueError(f"part_L must be [slots, {b}, {h}], got {tuple(part_L.shape)}")
    if int(part_A.shape[0]) < num_splits or int(part_L.shape[0]) < num_splits:
        raise ValueError("part_A and part_L need num_splits slots")
    need = int(kv.view.num_seqs) * int(kv.view.num_kv_heads)
    if arrivals.numel() < need:
        raise ValueError(f"arrivals needs num_seqs * num_kv_heads = {need} counters, "
                         f"got {arrivals.numel()}")
    for t, nm, n in ((z_out, "z_out", b * h), (out, "out", b * h * d),
                     (lse_out, "lse_out", b * h), (cert_out, "cert_out", b * h)):
        if t is not None and t.numel() < n:
            raise ValueError(f"{nm} needs {n} elements, got {t.numel()}")
    _need_device([("q", q), ("part_A", part_A), ("part_L", part_L), ("arrivals", arrivals),
                  ("z_out", z_out), ("out", out), ("lse_out", lse_out), ("cert_out", cert_out)]
                 + [(f"view tensor {i}", t) for i, t in enumerate(kv.tensors)] + list(extra))


@dataclass
class KV:
    """A cache view plus the tensors it points into (kept alive here)."""
    view: fold_kv_view
    tensors: tuple


@dataclass
class Q:
    view: fold_q_view
    tensor: torch.Tensor


def kv_view(k: torch.Tensor, v: Optional[torch.Tensor], seq_lens: torch.Tensor, *,
            num_kv_heads: int, max_seq_len: int, block_table: Optional[torch.Tensor] = None,
            row_indptr: Optional[torch.Tensor] = None, row_req: Optional[torch.Tensor] = None,
            max_reqs_per_seq: int = 1, k_is_layout_only: bool = False) -> KV:
    """Describe one scan level.  Paged: ``k, v [num_pages, Hkv, P, D]`` with
    ``block_table [num_seqs, max_pages]``; contiguous: ``k, v [num_seqs, Hkv,
    max_seq_len, D]``.  With ``k_is_layout_only`` (two-plane key caches), ``k``
    is a key plane that gives the shape only and the view's key pointer is
    NULL.  A float16 ``k`` is the FP16 keys of a stacked two-plane level
    (``fold_q8_stack_keys``), read by ``fold_q8_decode_stacked`` only."""
    if k_is_layout_only:
        _need(k, "plane", torch.int8)
    elif k.dtype != torch.float16:
        _need(k, "k", torch.bfloat16)
    if v is not None:
        _need(v, "v", torch.bfloat16)
    _need(seq_lens, "seq_lens", torch.int32)
    d = int(k.shape[-1])
    s = fold_kv_view()
    s.k, s.v = (None if k_is_layout_only else _ptr(k)), _ptr(v)
    s.seq_lens = _ptr(seq_lens)
    s.num_seqs = int(seq_lens.shape[0])
    s.num_kv_heads = num_kv_heads
    s.head_dim = d
    s.max_seq_len = max_seq_len
    if block_table is not None:
        _need(block_table, "block_table", torch.int32)
        s.block_table = _ptr(block_table)
        s.page_size = int(k.shape[2])
        s.max_pages_per_seq = int(block_table.shape[1])
        s.num_pages = int(k.shape[0])
    if row_indptr is not None:
        _need(row_indptr, "row_indptr", torch.int32)
        _need(row_req, "row_req", torch.int32)
        s.row_indptr, s.row_req = _ptr(row_indptr), _ptr(row_req)
        s.max_reqs_per_seq = max_reqs_per_seq
    return KV(s, (k, v, seq_lens, block_table, row_indptr, row_req))


def q_view(q: torch.Tensor) -> Q:
    _need(q, "q", torch.bfloat16)
    s = fold_q_view()
    s.q = _ptr(q)
    s.batch, s.num_heads = int(q.shape[0]), int(q.shape[1])
    return Q(s, q)


def fold_decode_rows_per_group(kv: KV, q: Q) -> int:
    return load_library().fold_decode_rows_per_group(ctypes.byref(kv.view), ctypes.byref(q.view))


def fold_decode_row_groups(kv: KV, q: Q) -> int:
    return load_library().fold_decode_row_groups(ctypes.byref(kv.view), ctypes.byref(q.view))


def fold_ref_estimate(kv: KV, q: Q, sm_scale: float, z_out: torch.Tensor, params=None,
                      stream=None) -> torch.Tensor:
    _need(z_out, "z_out", torch.float32)
    p = None
    if params is not None:
        p = fold_est_params(params["sink"], params["recent"], params["strata"],
                            params["trim_lo"], params["trim_hi"])
    _check(load_library().fold_ref_estimate(ctypes.byref(kv.view), ctypes.byref(q.view),
                                            sm_scale, None if p is None else ctypes.byref(p),
                                            _ptr(z_out), _stream(stream)))
    return z_out


def fold_decode_split(kv: KV, q: Q, sm_scale: float, z: torch.Tensor, depth_T: float,
                      num_splits: int, slot_offset: int, part_A: torch.Tensor,
                      part_L: torch.Tensor, x_out: Optional[torch.Tensor] = None,
                      key_gate_out: Optional[torch.Tensor] = None,
                      page_gate_out: Optional[torch.Tensor] = None,
                      part_Lcut: Optional[torch.Tensor] = None, stream=None) -> None:
    _need(z, "z", torch.float32)
    _need(part_A, "part_A", torch.float32)
    _need(part_L, "part_L", torch.float32)
    if part_Lcut is not None:
        _need(part_Lcut, "part_Lcut", torch.float32)
    _slot_checks(q.tensor, part_A, part_L, part_Lcut, z)
    _need_device([("q", q.tensor), ("z", z), ("part_A", part_A), ("part_L", part_L),
                  ("part_Lcut", part_Lcut), ("x_out", x_out), ("key_gate_out", key_gate_out),
                  ("page_gate_out", page_gate_out)]
                 + [(f"view tensor {i}", t) for i, t in enumerate(kv.tensors)])
    dbg = None
    if x_out is not None or key_gate_out is not None or page_gate_out is not None:
        for t, nm, dt in ((x_out, "x_out", torch.float32), (key_gate_out, "key_gate_out", torch.uint8),
                          (page_gate_out, "page_gate_out", torch.uint8)):
            if t is not None:
                _need(t, nm, dt)
        dbg = fold_debug(_ptr(x_out), _ptr(key_gate_out), _ptr(page_gate_out))
    _check(load_library().fold_decode_split(
        ctypes.byref(kv.view), ctypes.byref(q.view), sm_scale, _ptr(z), depth_T, num_splits,
        slot_offset, int(part_A.shape[0]), _ptr(part_A), _ptr(part_L), _ptr(part_Lcut),
        None if dbg is None else ctypes.byref(dbg), _stream(stream)))


def fold_decode_cascade(prefix: KV, suffix: KV, q: Q, sm_scale: float, z: torch.Tensor,
                        depth_T: float, num_splits: int, slot_offset: int, part_A: torch.Tensor,
                        part_L: torch.Tensor, part_Lcut: Optional[torch.Tensor] = None,
                        stream=None) -> None:
    """Prefix level (stacked rows) and per-request suffix level of a cascade in
    one scan launch; slot ``slot_offset + s`` gets split ``s`` of both."""
    _need(z, "z", torch.float32)
    _need(part_A, "part_A", torch.float32)
    _need(part_L, "part_L", torch.float32)
    if part_Lcut is not None:
        _need(part_Lcut, "part_Lcut", torch.float32)
    _slot_checks(q.tensor, part_A, part_L, part_Lcut, z)
    _need_device([("q", q.tensor), ("z", z), ("part_A", part_A), ("part_L", part_L),
                  ("part_Lcut", part_Lcut)]
                 + [(f"prefix view tensor {i}", t) for i, t in enumerate(prefix.tensors)]
                 + [(f"suffix view tensor {i}", t) for i, t in enumerate(suffix.tensors)])
    _check(load_library().fold_decode_cascade(
        ctypes.byref(prefix.view), ctypes.byref(suffix.view), ctypes.byref(q.view), sm_scale,
        _ptr(z), depth_T, num_splits, slot_offset, int(part_A.shape[0]), _ptr(part_A),
        _ptr(part_L), _ptr(part_Lcut), _stream(stream)))


def block_count(max_seq_len: int) -> int:
    """Blocks of the block model a view of ``max_seq_len`` keys needs."""
    return (int(max_seq_len) + 63) // 64


def chunk_count(max_seq_len: int) -> int:
    """16-key chunks per row of the block model's cut-mass workspace."""
    return (int(max_seq_len) + 15) // 16


def _block_mean_checks(kv: KV, block_mean: torch.Tensor) -> int:
    v = kv.view
    want = (v.num_seqs, v.num_kv_heads)
    if block_mean.dim() != 4 or tuple(block_mean.shape[:2]) != want or \
            int(block_mean.shape[3]) != v.head_dim:
        raise ValueError(f"block_mean must be [{want[0]}, {want[1]}, max_blocks, {v.head_dim}], "
                         f"got {tuple(block_mean.shape)}")
    if not block_mean.is_contiguous():
        raise ValueError("block_mean must be contiguous")
    mb = int(block_mean.shape[2])
    if mb < block_count(v.max_seq_len):
        raise ValueError(f"block_mean holds {mb} blocks; the view needs {block_count(v.max_seq_len)}")
    return mb


def fold_value_block_mean(kv: KV, mean_out: torch.Tensor, stream=None) -> torch.Tensor:
    """Mean value row of every 64-key block, ``[num_seqs, Hkv, max_blocks, D]``."""
    _need(mean_out, "mean_out", torch.float32)
    mb = _block_mean_checks(kv, mean_out)
    _need_device([("mean_out", mean_out)] + [(f"view tensor {i}", t) for i, t in enumerate(kv.tensors)])
    _check(load_library().fold_value_block_mean(ctypes.byref(kv.view), mb, _ptr(mean_out),
                                                _stream(stream)))
    return mean_out


def fold_value_block_mean_append(kv: KV, v_src: torch.Tensor, tok_seq: torch.Tensor,
                                 tok_pos: torch.Tensor, mean: torch.Tensor, stream=None) -> None:
    """Running update of the appended tokens' blocks (one token per sequence)."""
    _need(v_src, "v_src", torch.bfloat16)
    _need(tok_seq, "tok_seq", torch.int32)
    _need(tok_pos, "tok_pos", torch.int32)
    _need(mean, "mean", torch.float32)
    mb = _block_mean_checks(kv, mean)
    _need_device([("v_src", v_src), ("tok_seq", tok_seq), ("tok_pos", tok_pos), ("mean", mean)])
    _check(load_library().fold_value_block_mean_append(
        ctypes.byref(kv.view), mb, _ptr(v_src), _ptr(tok_seq), _ptr(tok_pos),
        int(tok_seq.shape[0]), _ptr(mean), _stream(stream)))


def fold_decode_split_blocks(kv: KV, q: Q, sm_scale: float, z: torch.Tensor, depth_T: float,
                             num_splits: int, slot_offset: int, part_A: torch.Tensor,
                             part_L: torch.Tensor, block_mean: torch.Tensor,
                             chunk_cut: Optional[torch.Tensor],
                             x_out: Optional[torch.Tensor] = None,
                             key_gate_out: Optional[torch.Tensor] = None,
                             page_gate_out: Optional[torch.Tensor] = None, stream=None) -> None:
    """``fold_decode_split`` with the block model of BF16 values: each tile's
    cut mass times its block's mean is added to the owning split's A.
    ``chunk_cut`` (``[B * H * chunk_count(max_seq_len)]`` float32 workspace)
    receives the cut masses per row and 16-key chunk."""
    _need(z, "z", torch.float32)
    _need(part_A, "part_A", torch.float32)
    _need(part_L, "part_L", torch.float32)
    _need(block_mean, "block_mean", torch.float32)
    mb = _block_mean_checks(kv, block_mean)
    _slot_checks(q.tensor, part_A, part_L, None, z)
    b, h, _ = (int(x) for x in q.tensor.shape)
    if chunk_cut is not None:
        _need(chunk_cut, "chunk_cut", torch.float32)
        need = b * h * chunk_count(kv.view.max_seq_len)
        if chunk_cut.numel() < need:
            raise ValueError(f"chunk_cut needs {need} elements, got {chunk_cut.numel()}")
    _need_device([("q", q.tensor), ("z", z), ("part_A", part_A), ("part_L", part_L),
                  ("block_mean", block_mean), ("chunk_cut", chunk_cut), ("x_out", x_out),
                  ("key_gate_out", key_gate_out), ("page_gate_out", page_gate_out)]
                 + [(f"view tensor {i}", t) for i, t in enumerate(kv.tensors)])
    dbg = None
    if x_out is not None or key_gate_out is not None or page_gate_out is not None:
        for t, nm, dt in ((x_out, "x_out", torch.float32), (key_gate_out, "key_gate_out", torch.uint8),
                          (page_gate_out, "page_gate_out", torch.uint8)):
            if t is not None:
                _need(t, nm, dt)
        dbg = fold_debug(_ptr(x_out), _ptr(key_gate_out), _ptr(page_gate_out))
    model = fold_block_model(_ptr(block_mean), mb, _ptr(chunk_cut))
    _check(load_library().fold_decode_split_blocks(
        ctypes.byref(kv.view), ctypes.byref(q.view), sm_scale, _ptr(z), depth_T, num_splits,
        slot_offset, int(part_A.shape[0]), _ptr(part_A), _ptr(part_L), ctypes.byref(model),
        None if dbg is None else ctypes.byref(dbg), _stream(stream)))


def fold_combine(part_A: torch.Tensor, part_L: torch.Tensor, out: torch.Tensor,
                 z: Optional[torch.Tensor] = None, lse_out: Optional[torch.Tensor] = None,
                 cert_out: Optional[torch.Tensor] = None,
                 part_Lcut: Optional[torch.Tensor] = None, mean: Optional[torch.Tensor] = None,
                 num_kv_heads: Optional[int] = None, stream=None) -> torch.Tensor:
    """Slot-order combine; with ``part_Lcut`` and ``mean`` ([B, Hkv, D]) the
    cut-key value model adds the cut masses times the request means."""
    _need(part_A, "part_A", torch.float32)
    _need(part_L, "part_L", torch.float32)
    model = None
    if part_Lcut is not None or mean is not None:
        _need(part_Lcut, "part_Lcut", torch.float32)
        _need(mean, "mean", torch.float32)
        heads = int(part_A.shape[-2])
        model = fold_value_model(_ptr(part_Lcut), _ptr(mean), heads,
                                 int(num_kv_heads if num_kv_heads is not None else mean.shape[1]))
    if out.dtype == torch.float32:
        odt = FOLD_DTYPE_F32
    elif out.dtype == torch.bfloat16:
        odt = FOLD_DTYPE_BF16
    else:
        raise TypeError("out must be float32 or bfloat16")
    if not out.is_contiguous():
        raise ValueError("out must be contiguous")
    num_slots = int(part_A.shape[0])
    d = int(part_A.shape[-1])
    rows = part_A[0].numel() // d if num_slots else 0
    _check(load_library().fold_combine(_ptr(part_A), _ptr(part_L), num_slots, rows, d, _ptr(z),
                                       _ptr(out), odt, _ptr(lse_out), _ptr(cert_out),
                                       None if model is None else ctypes.byref(model),
                                       _stream(stream)))
    return out


def fold_decode_fused(kv: KV, q: Q, sm_scale: float, depth_T: float, num_splits: int,
                      part_A: torch.Tensor, part_L: torch.Tensor, arrivals: torch.Tensor,
                      z_out: torch.Tensor, out: torch.Tensor,
                      lse_out: Optional[torch.Tensor] = None,
                      cert_out: Optional[torch.Tensor] = None, params=None,
                      stream=None) -> torch.Tensor:
    """Estimate, scan and combine of one per-request level in one launch.
    ``arrivals`` ([num_seqs, Hkv] int32) must be zero before the first call and
    is zero after every call; ``part_A``/``part_L`` hold ``num_splits`` slots."""
    _need(part_A, "part_A", torch.float32)
    _need(part_L, "part_L", torch.float32)
    _need(arrivals, "arrivals", torch.int32)
    _need(z_out, "z_out", torch.float32)
    if lse_out is not None:
        _need(lse_out, "lse_out", torch.float32)
    if cert_out is not None:
        _need(cert_out, "cert_out", torch.uint8)
    if out.dtype == torch.float32:
        odt = FOLD_DTYPE_F32
    elif out.dtype == torch.bfloat16:
        odt = FOLD_DTYPE_BF16
    else:
        raise TypeError("out must be float32 or bfloat16")
    if not out.is_contiguous():
        raise ValueError("out must be contiguous")
    _fused_checks(kv, q.tensor, num_splits, part_A, part_L, arrivals, z_out, out, lse_out,
                  cert_out)
    p = None
    if params is not None:
        p = fold_est_params(params["sink"], params["recent"], params["strata"],
                            params["trim_lo"], params["trim_hi"])
    _check(load_library().fold_decode_fused(
        ctypes.byref(kv.view), ctypes.byref(q.view), sm_scale,
        None if p is None else ctypes.byref(p), depth_T, num_splits, _ptr(part_A), _ptr(part_L),
        _ptr(arrivals), _ptr(z_out), _ptr(out), odt, _ptr(lse_out), _ptr(cert_out),
        _stream(stream)))
    return out


def fold_decode_fused_noalloc(kv: KV, q: Q, sm_scale: float, depth_T: float, num_splits: int,
                              z_out: torch.Tensor, out: torch.Tensor,
                              lse_out: Optional[torch.Tensor] = None,
                              cert_out: Optional[torch.Tensor] = None, params=None,
                              stream=None) -> torch.Tensor:
    """fold_decode_fused with its slots and arrival counts in the library's
    fixed device scratch (8 MiB per GPU): no workspace, no allocation.  Calls
    that overlap on one GPU race on that scratch."""
    _need(z_out, "z_out", torch.float32)
    if lse_out is not None:
        _need(lse_out, "lse_out", torch.float32)
    if cert_out is not None:
        _need(cert_out, "cert_out", torch.uint8)
    if out.dtype == torch.float32:
        odt = FOLD_DTYPE_F32
    elif out.dtype == torch.bfloat16:
        odt = FOLD_DTYPE_BF16
    else:
        raise TypeError("out must be float32 or bfloat16")
    if not out.is_contiguous():
        raise ValueError("out must be contiguous")
    b, h, d = (int(x) for x in q.tensor.shape)
    for t, nm, n in ((z_out, "z_out", b * h), (out, "out", b * h * d),
                     (lse_out, "lse_out", b * h), (cert_out, "cert_out", b * h)):
        if t is not None and t.numel() < n:
            raise ValueError(f"{nm} needs {n} elements, got {t.numel()}")
    _need_device([("q", q.tensor), ("z_out", z_out), ("out", out), ("lse_out", lse_out),
                  ("cert_out", cert_out)]
                 + [(f"view tensor {i}", t) for i, t in enumerate(kv.tensors)])
    p = None
    if params is not None:
        p = fold_est_params(params["sink"], params["recent"], params["strata"],
                            params["trim_lo"], params["trim_hi"])
    _check(load_library().fold_decode_fused_noalloc(
        ctypes.byref(kv.view), ctypes.byref(q.view), sm_scale,
        None if p is None else ctypes.byref(p), depth_T, num_splits, _ptr(z_out), _ptr(out), odt,
        _ptr(lse_out), _ptr(cert_out), _stream(stream)))
    return out


def fold_value_mean(kv: KV, mean_out: torch.Tensor, stream=None) -> torch.Tensor:
    """Request mean value rows ``[num_seqs, Hkv, D]`` of a per-request view."""
    _need(mean_out, "mean_out", torch.float32)
    _check(load_library().fold_value_mean(ctypes.byref(kv.view), _ptr(mean_out), _stream(stream)))
    return mean_out


def fold_value_mean_append(kv: KV, v_src: torch.Tensor, tok_seq: torch.Tensor,
                           tok_pos: torch.Tensor, mean: torch.Tensor, stream=None) -> None:
    """Running update of the request means for appended tokens (one per sequence)."""
    _need(v_src, "v_src", torch.bfloat16)
    _need(tok_seq, "tok_seq", torch.int32)
    _need(tok_pos, "tok_pos", torch.int32)
    _need(mean, "mean", torch.float32)
    _check(load_library().fold_value_mean_append(
        ctypes.byref(kv.view), _ptr(v_src), _ptr(tok_seq), _ptr(tok_pos), int(tok_seq.shape[0]),
        _ptr(mean), _stream(stream)))


def fold_decode(levels, q: torch.Tensor, z: torch.Tensor, depth_T: float, splits,
                sm_scale: float, out_dtype=torch.float32, lse: bool = False, cert: bool = False,
                value_mean: Optional[torch.Tensor] = None, block_means=None, stream=None):
    """Every level's split scan into one slot array, then the combine.

    ``levels`` is a list of ``KV`` views; ``splits`` their split counts;
    ``value_mean`` ([B, Hkv, D], from ``fold_value_mean``) turns on the
    request-mean value model, ``block_means`` (one ``fold_value_block_mean``
    array per level) the block model of BF16 values; at most one of them.
    Returns ``(out, part_A, part_L, lse_out, cert_out)``.
    """
    if value_mean is not None and block_means is not None:
        raise ValueError("value_mean and block_means are two value models: pass one")
    b, h, d = q.shape
    qv = q_view(q)
    total = sum(splits)
    part_A = torch.empty(total, b, h, d, dtype=torch.float32, device=q.device)
    part_L = torch.empty(total, b, h, dtype=torch.float32, device=q.device)
    part_C = (torch.empty(total, b, h, dtype=torch.float32, device=q.device)
              if value_mean is not None else None)
    cut = None
    if block_means is not None:
        if len(block_means) != len(levels):
            raise ValueError("block_means needs one array per level")
        cut = torch.empty(b * h * max(chunk_count(kv.view.max_seq_len) for kv in levels),
                          dtype=torch.float32, device=q.device)
    off = 0
    for i, (kv, s) in enumerate(zip(levels, splits)):
        if block_means is not None:
            fold_decode_split_blocks(kv, qv, sm_scale, z, depth_T, s, off, part_A, part_L,
                                     block_means[i], cut, stream=stream)
        else:
            fold_decode_split(kv, qv, sm_scale, z, depth_T, s, off, part_A, part_L,
                              part_Lcut=part_C, stream=stream)
        off += s
    out = torch.empty(b, h, d, dtype=out_dtype, device=q.device)
    lse_out = torch.empty(b, h, dtype=torch.float32, device=q.device) if lse else None
    cert_out = torch.empty(b, h, dtype=torch.uint8, device=q.device) if cert else None
    fold_combine(part_A, part_L, out, z=z if lse else None, lse_out=lse_out, cert_out=cert_out,
                 part_Lcut=part_C, mean=value_mean, stream=stream)
    return out, part_A, part_L, lse_out, cert_out


def fold_append_kv(kv: KV, k_src: Optional[torch.Tensor], v_src: Optional[torch.Tensor],
                   tok_seq: torch.Tensor, tok_pos: torch.Tensor, k_cache: Optional[torch.Tensor],
                   v_cache: Optional[torch.Tensor], stream=None) -> None:
    """Store token rows ``[n_tok, Hkv, D]`` bf16 at (``tok_seq``, ``tok_pos``)
    of the caches laid out as ``kv`` (either cache may be None)."""
    for t, nm in ((k_src, "k_src"), (v_src, "v_src"), (k_cache, "k_cache"), (v_cache, "v_cache")):
        if t is not None:
            _need(t, nm, torch.bfloat16)
    _need(tok_seq, "tok_seq", torch.int32)
    _need(tok_pos, "tok_pos", torch.int32)
    _check(load_library().fold_append_kv(
        ctypes.byref(kv.view), _ptr(k_src), _ptr(v_src), _ptr(tok_seq), _ptr(tok_pos),
        int(tok_seq.shape[0]), _ptr(k_cache), _ptr(v_cache), _stream(stream)))


def fold_cert_update(cert: torch.Tensor, lse: torch.Tensor, z: torch.Tensor,
                     count: torch.Tensor, reruns: Optional[torch.Tensor] = None,
                     stream=None) -> None:
    """New references of the certificate's flagged rows, in place in ``z``;
    ``count`` (int32, one element) receives how many rows were flagged."""
    _need(cert, "cert", torch.uint8)
    _need(lse, "lse", torch.float32)
    _need(z, "z", torch.float32)
    _need(count, "count", torch.int32)
    if reruns is not None:
        _need(reruns, "reruns", torch.int32)
    _check(load_library().fold_cert_update(_ptr(cert), _ptr(lse), _ptr(z), int(z.numel()),
                                           _ptr(reruns), _ptr(count), _stream(stream)))


def fold_certified_decode(levels, q: torch.Tensor, z: torch.Tensor, depth_T: float, splits,
                          sm_scale: float, max_reruns: int = 8, out_dtype=torch.float32,
                          value_mean: Optional[torch.Tensor] = None, stream=None):
    """``fold_decode`` under the range certificate: rows outside the window are
    decoded again with their new references, at most ``max_reruns`` times
    (each rerun reads a flag count back to the host).  Returns
    ``(out, z_final, reruns [B, H] int32, cert [B, H] u8)``; ``z`` is not
    modified."""
    z = z.clone()
    reruns = torch.zeros(z.shape, dtype=torch.int32, device=z.device)
    count = torch.zeros(1, dtype=torch.int32, device=z.device)
    out, _, _, lse, cert = fold_decode(levels, q, z, depth_T, splits, sm_scale, out_dtype,
                                       lse=True, cert=True, value_mean=value_mean, stream=stream)
    for _ in range(max_reruns):
        fold_cert_update(cert, lse, z, count, reruns, stream=stream)
        if int(count.item()) == 0:
            break
        out, _, _, lse, cert = fold_decode(levels, q, z, depth_T, splits, sm_scale, out_dtype,
                                           lse=True, cert=True, value_mean=value_mean,
                                           stream=stream)
    return out, z, reruns, cert


# ---------------------------------------------------------------- drafts ----
@dataclass
class DraftViews:
    """The two levels and the estimate view of draft columns (include/fold_draft.h)."""
    committed: KV          # requests' pages, committed lengths, columns stacked as CSR rows
    ancestors: KV          # one kv sequence per column: its ancestors' keys
    estimate: KV           # per-column view of the committed keys
    num_cols: int
    keep: tuple


def _host_i32(x) -> torch.Tensor:
    return torch.as_tensor(x, dtype=torch.int32).contiguous().cpu()


def fold_draft_views(k: torch.Tensor, v: Optional[torch.Tensor], block_table: torch.Tensor,
                     seq_lens, col_indptr, parent, spare_pages: torch.Tensor, *,
                     num_kv_heads: int, extra=(), layout: Optional[torch.Tensor] = None,
                     stream=None) -> DraftViews:
    """Plan draft columns on the host (``seq_lens``, ``col_indptr`` and
    ``parent`` are host sequences), copy each column's ancestor rows of
    ``k``, ``v`` and every ``(array, row_bytes)`` of ``extra`` into its spare
    pages, and return the views.  ``layout`` (a key plane) replaces ``k`` as
    the views' shape for a two-plane cache; then ``k`` may be None."""
    lib = load_library()
    shape_src = layout if layout is not None else k
    dev = shape_src.device
    n_pool, hkv, page, d = shape_src.shape
    sl = _host_i32(seq_lens)
    ind = _host_i32(col_indptr)
    par = _host_i32(parent)
    b = int(sl.shape[0])
    cols = int(ind[-1]) if b else 0
    ppc = int(spare_pages.shape[1])
    cap = ppc * page
    committed = torch.empty(b, dtype=torch.int32)
    col_req = torch.empty(cols, dtype=torch.int32)
    col_lens = torch.empty(cols, dtype=torch.int32)
    anc_lens = torch.empty(cols, dtype=torch.int32)
    anc_pos = torch.empty(cols, cap, dtype=torch.int32)
    _check(lib.fold_draft_plan(b, _ptr(sl), _ptr(ind), _ptr(par), page, ppc, _ptr(committed),
                               _ptr(col_req), _ptr(col_lens), _ptr(anc_lens), _ptr(anc_pos)))
    committed_d, col_req_d, col_lens_d = committed.to(dev), col_req.to(dev), col_lens.to(dev)
    anc_lens_d, anc_pos_d, ind_d = anc_lens.to(dev), anc_pos.to(dev), ind.to(dev)
    _need(spare_pages, "spare_pages", torch.int32)
    _need(block_table, "block_table", torch.int32)
    max_len = int(sl.max()) if b else 0
    req_view = kv_view(shape_src, None, sl.to(dev), num_kv_heads=num_kv_heads,
                       max_seq_len=max_len, block_table=block_table,
                       k_is_layout_only=layout is not None)
    col_bt = torch.empty(cols, block_table.shape[1], dtype=torch.int32, device=dev)
    arrays = [(a, 2 * d) for a in (k, v) if a is not None] + list(extra)
    first = True
    for arr, row_bytes in arrays:
        _check(lib.fold_draft_gather(ctypes.byref(req_view.view), _ptr(col_req_d), _ptr(anc_lens_d),
                                     _ptr(anc_pos_d), _ptr(spare_pages), cols, ppc, int(row_bytes),
                                     _ptr(arr), _ptr(arr), _ptr(col_bt) if first else None,
                                     _stream(stream)))
        first = False
    if first:
        _check(lib.fold_draft_gather(ctypes.byref(req_view.view), _ptr(col_req_d), _ptr(anc_lens_d),
                                     _ptr(anc_pos_d), _ptr(spare_pages), cols, ppc, 2 * d, None,
                                     None, _ptr(col_bt), _stream(stream)))
    lay = layout is not None
    kk = layout if lay else k
    row_req = torch.arange(cols, dtype=torch.int32, device=dev)
    max_m = int((ind[1:] - ind[:-1]).max()) if b else 1
    max_committed = int(committed.max()) if b else 0
    committed_kv = kv_view(kk, v, committed_d, num_kv_heads=num_kv_heads,
                           max_seq_len=max_committed, block_table=block_table, row_indptr=ind_d,
                           row_req=row_req, max_reqs_per_seq=max(1, max_m), k_is_layout_only=lay)
    anc_kv = kv_view(kk, v, anc_lens_d, num_kv_heads=num_kv_heads, max_seq_len=cap,
                     block_table=spare_pages, k_is_layout_only=lay)
    est_kv = kv_view(kk, None, col_lens_d, num_kv_heads=num_kv_heads, max_seq_len=max_committed,
                     block_table=col_bt, k_is_layout_only=lay)
    return DraftViews(committed_kv, anc_kv, est_kv, cols,
                      (committed_d, col_req_d, col_lens_d, anc_lens_d, anc_pos_d, ind_d, col_bt,
                       row_req, req_view))


def depth_value(T) -> float:
    """``None`` / ``inf`` -> +INFINITY (dense decode); otherwise float(T)."""
    return math.inf if T is None else float(T)


# ------------------------------------------------- two-plane INT8 key cache --
@dataclass
class Q8Keys:
    """The planes and scales of a two-plane key cache (kept alive here).

    ``plane_a, plane_b`` int8 and ``scale`` int16 (BF16 bits) in the element
    layout of the BF16 key cache they replace."""
    plane_a: torch.Tensor
    plane_b: torch.Tensor
    scale: torch.Tensor

    def view(self) -> fold_q8_keys:
        return fold_q8_keys(_ptr(self.plane_a), _ptr(self.plane_b), _ptr(self.scale))


@dataclass
class Q8Query:
    """Query codes ``planes [B, H, 2, D]`` int8, ``eta [B, H]``, ``tau [B]`` and
    (8-bit values) ``tau_v [B]`` fp32."""
    planes: torch.Tensor
    eta: torch.Tensor
    tau: Optional[torch.Tensor]
    tau_v: Optional[torch.Tensor] = None

    def view(self) -> fold_q8_query:
        return fold_q8_query(_ptr(self.planes), _ptr(self.eta), _ptr(self.tau),
                             int(self.planes.shape[0]), int(self.planes.shape[1]),
                             _ptr(self.tau_v))


@dataclass
class V8Values:
    """8-bit values: E4M3 planes ``plane_p, plane_r`` (uint8, the BF16 value
    cache's element layout) under the scale ``2 ** scale_exp``."""
    plane_p: torch.Tensor
    plane_r: torch.Tensor
    scale_exp: int

    def view(self) -> fold_v8_values:
        return fold_v8_values(_ptr(self.plane_p), _ptr(self.plane_r), int(self.scale_exp))


def v8_empty_values(v_like: torch.Tensor, scale_exp: int) -> V8Values:
    return V8Values(torch.empty(v_like.shape, dtype=torch.uint8, device=v_like.device),
                    torch.empty(v_like.shape, dtype=torch.uint8, device=v_like.device),
                    scale_exp)


def fold_v8_write_values(kv: KV, v_src: torch.Tensor, tok_seq: torch.Tensor,
                         tok_pos: torch.Tensor, values: V8Values, stream=None) -> None:
    _need(v_src, "v_src", torch.bfloat16)
    _need(tok_seq, "tok_seq", torch.int32)
    _need(tok_pos, "tok_pos", torch.int32)
    _need(values.plane_p, "plane_p", torch.uint8)
    _need(values.plane_r, "plane_r", torch.uint8)
    _check(load_library().fold_v8_write_values(
        ctypes.byref(kv.view), _ptr(v_src), _ptr(tok_seq), _ptr(tok_pos), int(tok_seq.shape[0]),
        int(values.scale_exp), _ptr(values.plane_p), _ptr(values.plane_r), _stream(stream)))


def q8_empty_keys(k_like: torch.Tensor) -> Q8Keys:
    """Uninitialised planes and scales shaped like a BF16 key cache."""
    return Q8Keys(torch.empty(k_like.shape, dtype=torch.int8, device=k_like.device),
                  torch.empty(k_like.shape, dtype=torch.int8, device=k_like.device),
                  torch.empty(k_like.shape[:-1], dtype=torch.int16, device=k_like.device))


def fold_q8_write_keys(kv: KV, k_src: torch.Tensor, tok_seq: torch.Tensor, tok_pos: torch.Tensor,
                       keys: Q8Keys, stream=None) -> None:
    _need(k_src, "k_src", torch.bfloat16)
    _need(tok_seq, "tok_seq", torch.int32)
    _need(tok_pos, "tok_pos", torch.int32)
    for t, nm, dt in ((keys.plane_a, "plane_a", torch.int8), (keys.plane_b, "plane_b", torch.int8),
                      (keys.scale, "scale", torch.int16)):
        _need(t, nm, dt)
    _check(load_library().fold_q8_write_keys(
        ctypes.byref(kv.view), _ptr(k_src), _ptr(tok_seq), _ptr(tok_pos), int(tok_seq.shape[0]),
        _ptr(keys.plane_a), _ptr(keys.plane_b), _ptr(keys.scale), _stream(stream)))


def fold_q8_split_query(q: torch.Tensor, sm_scale: float, out: Q8Query,
                        req_lens: Optional[torch.Tensor] = None, kappa: float = -4.0,
                        kappa_v: float = -4.0, stream=None) -> Q8Query:
    qv = q_view(q)
    _need(out.planes, "planes", torch.int8)
    _need(out.eta, "eta", torch.float32)
    if req_lens is not None:
        _need(req_lens, "req_lens", torch.int32)
        _need(out.tau, "tau", torch.float32)
    if req_lens is not None and out.tau_v is not None:
        _need(out.tau_v, "tau_v", torch.float32)
    _check(load_library().fold_q8_split_query(
        ctypes.byref(qv.view), int(q.shape[-1]), sm_scale, _ptr(req_lens), kappa, kappa_v,
        _ptr(out.planes), _ptr(out.eta), None if req_lens is None else _ptr(out.tau),
        None if req_lens is None else _ptr(out.tau_v), _stream(stream)))
    return out


def q8_empty_query(q: torch.Tensor) -> Q8Query:
    b, h, d = q.shape
    return Q8Query(torch.empty(b, h, 2, d, dtype=torch.int8, device=q.device),
                   torch.empty(b, h, dtype=torch.float32, device=q.device),
                   torch.empty(b, dtype=torch.float32, device=q.device),
                   torch.empty(b, dtype=torch.float32, device=q.device))


def fold_q8_ref_estimate(kv: KV, keys: Q8Keys, q: Q8Query, z_out: torch.Tensor, params=None,
                         stream=None) -> torch.Tensor:
    _need(z_out, "z_out", torch.float32)
    p = None
    if params is not None:
        p = fold_est_params(params["sink"], params["recent"], params["strata"],
                            params["trim_lo"], params["trim_hi"])
    kk, qq = keys.view(), q.view()
    _check(load_library().fold_q8_ref_estimate(
        ctypes.byref(kv.view), ctypes.byref(kk), ctypes.byref(qq),
        None if p is None else ctypes.byref(p), _ptr(z_out), _stream(stream)))
    return z_out


def fold_q8_front(kv: KV, keys: Q8Keys, q: torch.Tensor, sm_scale: float, out: Q8Query,
                  z_out: torch.Tensor, req_lens: Optional[torch.Tensor] = None,
                  kappa: float = -4.0, kappa_v: float = -4.0, params=None,
                  stream=None) -> torch.Tensor:
    """fold_q8_split_query followed by fold_q8_ref_estimate, in one launch."""
    qv = q_view(q)
    _need(out.planes, "planes", torch.int8)
    _need(out.eta, "eta", torch.float32)
    _need(z_out, "z_out", torch.float32)
    if req_lens is not None:
        _need(req_lens, "req_lens", torch.int32)
        _need(out.tau, "tau", torch.float32)
    if req_lens is not None and out.tau_v is not None:
        _need(out.tau_v, "tau_v", torch.float32)
    p = None
    if params is not None:
        p = fold_est_params(params["sink"], params["recent"], params["strata"],
                            params["trim_lo"], params["trim_hi"])
    kk = keys.view()
    _check(load_library().fold_q8_front(
        ctypes.byref(kv.view), ctypes.byref(kk), ctypes.byref(qv.view), sm_scale,
        _ptr(req_lens), kappa, kappa_v, _ptr(out.planes), _ptr(out.eta),
        None if req_lens is None else _ptr(out.tau),
        None if req_lens is None else _ptr(out.tau_v),
        None if p is None else ctypes.byref(p), _ptr(z_out), _stream(stream)))
    return z_out


def fold_q8_decode_rows_per_group(kv: KV, q: Q8Query) -> int:
    qq = q.view()
    return load_library().fold_q8_decode_rows_per_group(ctypes.byref(kv.view), ctypes.byref(qq))


def fold_q8_decode_row_groups(kv: KV, q: Q8Query) -> int:
    qq = q.view()
    return load_library().fold_q8_decode_row_groups(ctypes.byref(kv.view), ctypes.byref(qq))


def fold_q8_stack_keys(kv: KV, keys: Q8Keys, k_f16: torch.Tensor, stream=None) -> torch.Tensor:
    """FP16 keys ``fp16(e (a + b/256))`` of a stacked level's kv sequences, in
    the element layout of the planes (written once per prefix)."""
    _need(k_f16, "k_f16", torch.float16)
    if tuple(k_f16.shape) != tuple(keys.plane_a.shape):
        raise ValueError(f"k_f16 must be shaped like the planes {tuple(keys.plane_a.shape)}")
    _need_device([("k_f16", k_f16), ("plane_a", keys.plane_a), ("plane_b", keys.plane_b),
                  ("scale", keys.scale)] + [(f"view tensor {i}", t) for i, t in
                                            enumerate(kv.tensors) if t is not None])
    kk = keys.view()
    _check(load_library().fold_q8_stack_keys(ctypes.byref(kv.view), ctypes.byref(kk),
                                             _ptr(k_f16), _stream(stream)))
    return k_f16


def fold_q8_decode_stacked(kv: KV, q: Q8Query, z: torch.Tensor, depth_T: float,
                           num_splits: int, slot_offset: int, part_A: torch.Tensor,
                           part_L: torch.Tensor, x_out: Optional[torch.Tensor] = None,
                           key_gate_out: Optional[torch.Tensor] = None,
                           page_gate_out: Optional[torch.Tensor] = None,
                           part_Lcut: Optional[torch.Tensor] = None, stream=None) -> None:
    """Split scan of a stacked level (more than 32 rows per kv sequence) over
    the FP16 keys of ``fold_q8_stack_keys`` (``kv.view.k``)."""
    _need(z, "z", torch.float32)
    _need(part_A, "part_A", torch.float32)
    _need(part_L, "part_L", torch.float32)
    if kv.tensors[0] is None or kv.tensors[0].dtype != torch.float16:
        raise ValueError("the view's k must be the FP16 keys of fold_q8_stack_keys")
    if part_Lcut is not None:
        _need(part_Lcut, "part_Lcut", torch.float32)
    b, h = int(q.planes.shape[0]), int(q.planes.shape[1])
    if part_A.dim() != 4 or tuple(part_A.shape[1:3]) != (b, h):
        raise ValueError(f"part_A must be [slots, {b}, {h}, D], got {tuple(part_A.shape)}")
    _need_device([("planes", q.planes), ("eta", q.eta), ("z", z), ("part_A", part_A),
                  ("part_L", part_L), ("part_Lcut", part_Lcut), ("x_out", x_out),
                  ("key_gate_out", key_gate_out), ("page_gate_out", page_gate_out)]
                 + [(f"view tensor {i}", t) for i, t in enumerate(kv.tensors)])
    dbg = None
    if x_out is not None or key_gate_out is not None or page_gate_out is not None:
        for t, nm, dt in ((x_out, "x_out", torch.float32), (key_gate_out, "key_gate_out", torch.uint8),
                          (page_gate_out, "page_gate_out", torch.uint8)):
            if t is not None:
                _need(t, nm, dt)
        dbg = fold_debug(_ptr(x_out), _ptr(key_gate_out), _ptr(page_gate_out))
    qq = q.view()
    _check(load_library().fold_q8_decode_stacked(
        ctypes.byref(kv.view), ctypes.byref(qq), _ptr(z), depth_T, num_splits, slot_offset,
        int(part_A.shape[0]), _ptr(part_A), _ptr(part_L), _ptr(part_Lcut),
        None if dbg is None else ctypes.byref(dbg), _stream(stream)))


def fold_q8_decode_split(kv: KV, keys: Q8Keys, q: Q8Query, z: torch.Tensor, depth_T: float,
                         num_splits: int, slot_offset: int, part_A: torch.Tensor,
                         part_L: torch.Tensor, x_out: Optional[torch.Tensor] = None,
                         xc_out: Optional[torch.Tensor] = None,
                         key_gate_out: Optional[torch.Tensor] = None,
                         page_gate_out: Optional[torch.Tensor] = None,
                         refine_gate_out: Optional[torch.Tensor] = None,
                         part_Lcut: Optional[torch.Tensor] = None,
                         values: Optional[V8Values] = None,
                         refine_v_gate_out: Optional[torch.Tensor] = None, stream=None) -> None:
    _need(z, "z", torch.float32)
    _need(part_A, "part_A", torch.float32)
    _need(part_L, "part_L", torch.float32)
    if part_Lcut is not None:
        _need(part_Lcut, "part_Lcut", torch.float32)
    outs = ((x_out, "x_out", torch.float32), (xc_out, "xc_out", torch.float32),
            (key_gate_out, "key_gate_out", torch.uint8),
            (page_gate_out, "page_gate_out", torch.uint8),
            (refine_gate_out, "refine_gate_out", torch.uint8),
            (refine_v_gate_out, "refine_v_gate_out", torch.uint8))
    dbg = None
    if any(t is not None for t, _, _ in outs):
        for t, nm, dt in outs:
            if t is not None:
                _need(t, nm, dt)
        dbg = fold_q8_debug(*(_ptr(t) for t, _, _ in outs))
    kk, qq = keys.view(), q.view()
    vals = None if values is None else values.view()
    _check(load_library().fold_q8_decode_split(
        ctypes.byref(kv.view), ctypes.byref(kk), ctypes.byref(qq),
        None if vals is None else ctypes.byref(vals), _ptr(z), depth_T, num_splits,
        slot_offset, int(part_A.shape[0]), _ptr(part_A), _ptr(part_L), _ptr(part_Lcut),
        None if dbg is None else ctypes.byref(dbg), _stream(stream)))
