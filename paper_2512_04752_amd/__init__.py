"""MI355X-native batched speculative-decoding tree-verify step.

The computation lives in the HIP library libspecverify.so (C ABI declared in
include/specverify.h); this package is its Python binding.  The library is
loaded on first use and its absence is an error.
"""

from .binding import (  # noqa: F401
    EXPORTS,
    CostModel,
    KVPool,
    SPEC_MAX_TREE,
    SpecError,
    Weights,
    lib,
    spec_kv_alloc,
    spec_kv_bytes,
    spec_kv_commit,
    spec_kv_free,
    spec_kv_pack,
    spec_kv_sample_layout,
    spec_kv_transfer_bytes,
    spec_kv_unpack,
    spec_profile_begin,
    spec_profile_end,
    spec_select_draft_count,
    spec_verify,
    spec_verify_sampled,
    spec_workspace_bytes,
    spec_workspace_bytes_sampled,
)
from .session import Verifier, flatten_trees  # noqa: F401
