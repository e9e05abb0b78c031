"""MI355X (gfx950) Sparse Steerable Convolution hot path (arXiv 2111.07383).

The computation lives in ``libssconv.so`` (HIP kernels behind the C ABI of
include/ssconv.h); ``binding`` only marshals torch tensors and streams into it.
"""
from ._abi import LIB_PATH, SSConvError, lib  # noqa: F401
from .binding import (  # noqa: F401
    Rulebook,
    backward,
    backward_workspace_size,
    basis_build,
    basis_desc,
    basis_info,
    build_rulebook,
    cached_bytes,
    debug_kernel_ms,
    debug_set,
    empty_cache,
    forward,
    forward_noalloc,
    forward_norm,
    NOALLOC_SCRATCH_BYTES,
    gate_backward,
    gate_forward,
    interpolate,
    interpolate_backward,
    layer_desc,
    make_fields,
    n_channels,
    norm_backward,
    norm_forward,
    pool_backward,
    pool_forward,
    steer,
    synth_kernel,
    voxelize,
    wigner_d,
)
