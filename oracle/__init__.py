"""FluxBin oracle: plain CPU reference implementations in float64.

TEST INFRASTRUCTURE ONLY. Only ``tests/``, ``__graft_entry__.smoke()`` and ``bench.py``'s ``cpu_baseline`` leg may
import, call or run anything in this package. The product path (``paper_2608_15602_amd``) never imports it, and
it never imports the product path: the two share no code. Only the seeded input generators in ``synth/`` serve both.
"""
from .fluxbin_oracle import (  # noqa: F401
    abw,
    complexity,
    effective_tflops,
    f16_to_f64,
    gemv_dense,
    gemv_lut,
    lut_bsf,
    lut_indices,
    parity_check,
    pattern_signs,
    patterns,
    reconstruct_rows,
    sign_bits,
    sign_pm1,
    smem_bytes,
    storage_bits,
    vcm_dense_bits,
    vcm_gather,
)
from . import format_oracle  # noqa: F401
from . import rc_oracle  # noqa: F401
