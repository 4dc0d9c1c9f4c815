"""Seeded synthetic workloads for the selective-update hot path.

This package only draws inputs (gradients, column scales, master weights,
stand-alone score vectors) and names the Llama-2-shaped gradient sets.  It
holds none of the method's arithmetic: no column norms, no selection, no
optimizer step, no packing.  Both the CPU oracle side of the tests and the
HIP path consume what it draws.
"""

from .configs import (  # noqa: F401
    AdamHyper,
    MatrixSpec,
    Workload,
    WORKLOADS,
    get_workload,
    llama_layer_shapes,
)
from .edges import edge_bf16, edge_f32, sprinkle_nonfinite  # noqa: F401
from .synth import (  # noqa: F401
    base_scales,
    derive_seed,
    gradient,
    gradient_iid,
    jittered_scales,
    master_weights,
    score_vector,
    space_all_pairs,
    space_boundary,
    step_scales,
)
