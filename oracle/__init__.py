"""CPU oracle of FadeMem's per-chunk cache step (test infrastructure only).

Only tests, the smoke check and the benchmark's CPU-baseline leg may import
this package.  The product library never does.
"""
from .fademem_oracle import (  # noqa: F401
    Entry,
    OracleCache,
    OPERATORS,
    TIE_RTOL,
    attend,
    band_correlations,
    bf16_bits,
    bf16_from_bits,
    chunk_step,
    dct2_ortho,
    decorrelation_horizons,
    exposed_kv_rope,
    fit_power_law,
    pearson,
    radial_band_of,
    round_to_bf16,
    round_to_f32,
    rope_angles,
    rope_rotate,
)
