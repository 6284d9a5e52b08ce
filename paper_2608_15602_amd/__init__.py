"""FluxBin LUT-GEMV hot path for AMD Instinct MI355X (gfx950).

The product is the C-ABI library ``libfluxbin.so`` (``include/fluxbin.h``); ``fluxbin`` is its thin ctypes binding.
"""
from . import fluxbin  # noqa: F401
from .fluxbin import (  # noqa: F401
    FluxbinError,
    PackedLayer,
    fluxbin_debug_indices,
    fluxbin_layer_from_header,
    fluxbin_lut_gemm_smallbatch,
    fluxbin_lut_gemv,
    fluxbin_pack,
    fluxbin_pack_query,
    fluxbin_unpack_canonical,
    fluxbin_workspace_init,
    fluxbin_workspace_query,
    make_shape,
    make_workspace,
)
