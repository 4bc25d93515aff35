"""MI355X (gfx950) best-matching-unit search for sparse-binary self-organising maps.

The compute path is libsom.so (hand-written HIP kernels behind the C ABI of
include/som.h); ``paper_2608_24067_amd.som`` is a thin ctypes binding with the
same names. PyTorch supplies device memory and streams only.
"""
from .som import (  # noqa: F401
    SomError,
    alloc_workspace,
    alloc_workspace2,
    alloc_workspace_sf,
    bmu2_finalize,
    bmu2_search,
    bmu2_sweep,
    bmu_finalize,
    bmu_sf_finalize,
    bmu_sf_plan,
    bmu_sf_search,
    bmu_sf_sweep,
    bmu_plan,
    bmu_search,
    bmu_sweep,
    codebook_norms,
    input_flags,
    last_error,
    library_path,
    load,
    radius,
    sigma,
    update,
    update_workspace_bytes,
    validate_csr_host,
    workspace2_bytes,
    workspace_sf_bytes,
    workspace_bytes,
)
