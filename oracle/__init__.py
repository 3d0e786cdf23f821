"""fp64 CPU reference of Kamera's chunk-reuse operator.

TEST INFRASTRUCTURE ONLY: imported by ``tests/``, the smoke check and the
benchmark's CPU-baseline leg, never by the product path.
"""

from .kamera_ref import (  # noqa: F401
    BLOCKED,
    INTERLEAVED,
    NEOX,
    Rope,
    add_patch,
    bf16_to_f64,
    form_patch,
    inv_freq,
    orbit_patch,
    pair_columns,
    pair_coordinate,
    paged_slot,
    positions_grid3,
    positions_linear,
    rehydrate_k,
    rehydrate_v,
    relocate_k,
    rope_angles,
    rotate,
    round_bf16,
    scatter_paged,
    shift_k,
)
