"""VideoMLA latent-attention hot path for AMD Instinct MI355X (gfx950).

The compute lives in libvideomla.so (hand-written HIP kernels behind a C ABI, declared in
include/videomla.h). This package is its thin Python binding: torch supplies device memory and
streams; importing it fails if the library has not been built.
"""
from ._lib import (  # noqa: F401
    EXPORTED,
    AttendOpts,
    Timer,
    VideomlaError,
    attend,
    attend_layer,
    attend_layer_workspace_bytes,
    attend_noalloc,
    attend_workspace_bytes,
    cache_bytes_per_token,
    cache_write,
    cache_write_prepared,
    dense_attend,
    dense_attend_workspace_bytes,
    dense_cache_bytes_per_token,
    dense_cache_write,
    layer_weights_bytes,
    make_dims,
    prepare_layer_weights,
    prepare_write_weights,
    slot_of,
    valid_tokens,
    window_advance,
    write_weights_bytes,
)
from ._lib import LIB_PATH, NOALLOC_SCRATCH_BYTES  # noqa: F401
from ._lib import (  # noqa: F401  (the diagnostic build: include/videomla_stamps.h)
    STAMP_KERNEL,
    STAMP_KERNELS,
    STAMP_POINTS,
    STAMP_WAVES,
    STAMP_WORKGROUPS,
    STAMPS,
    stamps_attach,
    stamps_buffer_bytes,
)
