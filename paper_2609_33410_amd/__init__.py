"""FoldAttention decode hot path for MI355X (gfx950).

The compute path is ``libfold.so`` (hand-written HIP kernels behind the C ABI
of ``include/fold.h``, ``include/fold_q8.h`` and ``include/fold_draft.h``);
:mod:`paper_2609_33410_amd.fold` is its ctypes
binding.  PyTorch supplies device memory and streams only.
"""

from .fold import (  # noqa: F401
    EXPORTED,
    FOLD_DTYPE_BF16,
    FOLD_DTYPE_F32,
    FOLD_E_HIP,
    FOLD_E_INVAL,
    FOLD_E_UNSUPPORTED,
    FOLD_OK,
    LIB_PATH,
    FoldError,
    FoldLibraryMissing,
    Q8Keys,
    Q8Query,
    DraftViews,
    V8Values,
    fold_append_kv,
    fold_cert_update,
    fold_certified_decode,
    fold_combine,
    fold_decode_fused,
    fold_decode_fused_noalloc,
    fold_decode,
    fold_draft_views,
    fold_decode_row_groups,
    fold_decode_rows_per_group,
    fold_decode_split,
    fold_q8_decode_row_groups,
    fold_q8_decode_rows_per_group,
    fold_q8_decode_split,
    fold_q8_front,
    fold_q8_ref_estimate,
    fold_q8_split_query,
    fold_q8_write_keys,
    fold_ref_estimate,
    fold_value_mean,
    fold_v8_write_values,
    fold_value_mean_append,
    kv_view,
    load_library,
    q8_empty_keys,
    q8_empty_query,
    v8_empty_values,
    q_view,
)
