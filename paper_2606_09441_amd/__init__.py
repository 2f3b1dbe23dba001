"""SIFT sparse prefill attention for AMD Instinct MI355X (gfx950).

The compute path is libsift.so (HIP kernels + C ABI, include/sift.h); this
package only marshals torch tensors into it.  Importing the package does not
load the library; the first call does, and fails loudly if it is not built.
"""

from ._lib import (  # noqa: F401
    Plan,
    SiftError,
    decode_tiles,
    decode_workspace_bytes,
    default_scale,
    extract_bits,
    extract_sizes,
    header_functions,
    lib,
    rope_,
    sparse_prefill,
    sparse_prefill_ex,
    workspace_bytes,
)

__all__ = ["Plan", "SiftError", "decode_tiles", "decode_workspace_bytes", "sparse_prefill", "sparse_prefill_ex", "workspace_bytes", "extract_bits", "extract_sizes", "rope_", "lib",
           "header_functions", "default_scale"]
