"""DendSN layer scan on AMD Instinct MI355X (gfx950).

The forward temporal scan of a layer of dendritic spiking neurons and its
surrogate-gradient backward scan, as hand-written HIP kernels behind the C ABI
of include/dendsn.h.  This package is the Python binding of that library.
"""

from .binding import (  # noqa: F401
    EXPORTS,
    LIB_PATH,
    NOALLOC_SCRATCH_BYTES,
    DendSNConfig,
    DendSNError,
    backward,
    dendsn_backward,
    dendsn_backward_noalloc,
    dendsn_bwd_workspace_bytes,
    dendsn_ckpt_bytes,
    dendsn_forward,
    dendsn_last_error,
    dendsn_status_str,
    forward,
    lib,
)
