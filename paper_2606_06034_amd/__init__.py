"""MI355X (gfx950) MatMul-only chunk inversion for chunk-wise Gated DeltaNet.

Python binding of the C ABI in include/gdninv.h (libgdninv.so, built in this
directory by ``python paper_2606_06034_amd/csrc/build.py``).  Every function
here has the name of the C entry point it wraps and only marshals arguments:
it checks that tensors are contiguous device tensors of the right dtype and
shape, allocates outputs with torch when the caller passes none, and calls
the library on torch's current stream.  All computation runs in the HIP
kernels; there is no fallback.  Importing this package without the built
library raises ImportError.
"""

from ._binding import (  # noqa: F401
    GDN_BF16,
    GDN_F32,
    GDN_I8,
    GDN_INT_PLAIN,
    GdnError,
    LIB_PATH,
    abi_symbols,
    gdn_abi_version,
    gdn_build_A,
    gdn_chunk_forward,
    gdn_chunk_forward_noalloc,
    gdn_chunk_forward_prepare,
    GDN_FORWARD_SCRATCH_BYTES,
    gdn_chunk_forward_state,
    gdn_chunk_forward_varlen,
    gdn_chunk_forward_workspace,
    gdn_chunk_inverse_fwdsub,
    gdn_chunk_inverse_blockwise,
    gdn_chunk_inverse_neumann,
    gdn_chunk_inverse_neumann_i8,
    gdn_chunk_inverse_neumann_i8_fused,
    gdn_chunk_inverse_fwdsub_i16,
    gdn_chunk_inverse_fwdsub_i8,
    gdn_chunk_inverse_neumann_i16,
    gdn_chunk_inverse_neumann_i16_fused,
    gdn_chunk_wy_fused,
    gdn_chunk_wy_fused_blockwise,
    gdn_chunk_wy_fused_varlen,
    gdn_varlen_tables,
    gdn_default_order,
    gdn_quantize_tiles_i8,
    gdn_quantize_tiles_i16,
    gdn_status_string,
    gdn_wy_apply,
    lib,
)
