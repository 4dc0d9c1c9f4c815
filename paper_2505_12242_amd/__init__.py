"""MI355X-native selective-update hot path of ZenFlow (arXiv 2505.12242).

Per bf16 weight gradient: per-input-channel squared norms, top-k channel
selection, in-place Adam on the selected channels' fp32 states with bf16
write-back, and S-step accumulation of the unselected channels in a packed
fp32 buffer handed over as a dense matrix.  All of it runs in the HIP
kernels of libzf.so (C ABI in include/zf.h); this package only binds it.
"""

from ._lib import (  # noqa: F401
    CHANNEL_MAJOR,
    LIB,
    LIB_PATH,
    ROW_MAJOR,
    STATIC_SCRATCH_BYTES,
    STATES_INIT,
    STATES_INPLACE,
    STATES_REMAP,
    AdamHparams,
    MatrixBuffers,
    Plan,
    Selection,
    StateSource,
    ZEN_TOTALS_BYTES,
    ZenTotals,
    ZfError,
    adam_selected,
    alloc_stored,
    colnorm,
    colnorm_noalloc,
    colnorm_workspace_bytes,
    host_adam_unselected,
    k_from_ratio,
    pack_accumulate,
    scatter_weights,
    topk_select,
    stream_probe,
    PROBE_READ,
    PROBE_COPY,
    PROBE_RMW,
    unpack,
    update_fused,
    update_fused_handover,
)
from .runner import SelectiveUpdateRunner, StepKind, schedule  # noqa: F401
