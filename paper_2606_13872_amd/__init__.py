"""Sparse Reference Attention (Avatar V) for AMD Instinct MI355X (gfx950).

The work runs in libsra.so (HIP kernels + host scheduler, C ABI in include/sra.h); this
package is its Python binding. Build the library with `python -m paper_2606_13872_amd.build`.
"""
from .sra import (  # noqa: F401
    SCHED_BWD_DKDV,
    SCHED_BWD_DQ,
    SCHED_FORWARD,
    Problem,
    SRAError,
    backward,
    forward,
    lib,
    pair_counts,
    release_caches,
    schedule_export,
    schedule_info,
    schedule_mask,
    useful_flops,
)
