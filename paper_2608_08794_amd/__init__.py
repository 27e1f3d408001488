"""MI355X-native A-PACK hot path: Python binding of libapack.so.

The functions below carry the C entry points' names and only marshal
arguments (tensor pointers, strides, host descriptors and the current HIP
stream) into the C ABI declared in include/apack.h; every step of the path
runs in the library's HIP kernels.  Importing this package loads nothing;
the first call loads ``libapack.so`` next to this file and raises
:class:`ApackError` if it is missing (build it with ``build.build()``).
"""

from ._lib import (  # noqa: F401
    APACK_AUDIO,
    APACK_BF16,
    APACK_F32,
    APACK_OTHER,
    APACK_VISUAL,
    ApackError,
    DynParams,
    apack_compact_kv,
    apack_compact_kv_inplace,
    apack_compact_kv_inplace_static,
    apack_compact_kv_inplace_status,
    apack_compact_kv_inplace_workspace,
    apack_dyn_params_default,
    apack_keep_count,
    apack_layer_flops,
    apack_prefill_flops,
    apack_prune_layer,
    apack_prune_layer_query,
    apack_schedule_lengths,
    apack_score_dynamics,
    apack_score_dynamics_query,
    apack_set_inplace_wait_limit,
    apack_visual_budget,
    library,
    library_path,
)
