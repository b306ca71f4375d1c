"""FP64 CPU oracle of the FoldAttention decode path (test infrastructure).

Only ``tests/``, ``__graft_entry__.smoke()`` and the benchmark's CPU-baseline
leg may import this package.  It shares no code with the HIP library.
"""

from .fold_oracle import (  # noqa: F401
    CERT_HI,
    CERT_LO,
    EST_DEFAULT,
    LOG2E,
    PAGE_GATE,
    TILE,
    bf16_bits_to_f64,
    block_means,
    combine,
    decode,
    decode_level,
    estimate_level,
    estimate_z,
    estimator_keys,
    fold,
    gather,
    live_mask,
    live_mask_imposed,
    lse_and_cert,
    read_gates,
    row_diagnostics,
    running_mean,
    scores,
    split_of_key,
    value_mean,
)
