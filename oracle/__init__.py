"""Oracle (test infrastructure only).

A plain float64 CPU statement of the batched tree-verify step, used by the
tests, the package smoke check and the benchmark's CPU-baseline leg to
check and time the HIP library, and of the KV transfer buffer of sample
migration (``oracle.transfer``).  The product path never imports it.
"""

from . import transfer  # noqa: F401

from .verify import (  # noqa: F401
    attention,
    commit,
    forward,
    greedy_accept,
    prefill,
    rms_norm,
    rope,
    rope_cos_sin,
    tree_metadata,
    verify,
)
