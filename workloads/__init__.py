"""Seeded synthetic decode workloads (input data only).

This module builds the query rows, the BF16 key/value cache (paged or
contiguous), the block tables and the sequence lengths of the five decode
workloads used by the tests and the benchmark. It holds none of the
attention method's arithmetic: no scores, no weights, no reference, no
gating. Both the CPU oracle and the HIP path read the tensors it produces.
"""

from .synth import (  # noqa: F401
    CONFIG_NAMES,
    DraftWorkload,
    KVView,
    Workload,
    host_bits,
    make_cascade,
    make_config,
    chain_parents,
    make_custom,
    make_drafts,
)
