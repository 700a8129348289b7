"""MI355X (gfx950) Barnes-Hut t-SNE gradient step and input similarities.

A thin ctypes binding over ``lib/libbhtsne.so`` (C ABI in ``include/bhtsne.h``).
PyTorch only provides device memory and the current stream; every step of
the computation runs in the library's HIP kernels.  The functions keep the C
names without the ``bhtsne_`` prefix.
"""
from ._binding import (  # noqa: F401
    BHTSNE_ECAPACITY,
    BHTSNE_EDEVICE,
    BHTSNE_EINPUT,
    BHTSNE_EINVAL,
    BHTSNE_ENONFINITE,
    BHTSNE_EWORKSPACE,
    BHTSNE_OK,
    PHASES,
    BhtsneError,
    Csr,
    CsrF64,
    Layout,
    LayoutF64,
    affinities,
    affinities_workspace_size,
    debug_sort,
    debug_sort_3d,
    debug_tree,
    debug_tree_3d,
    get_stats,
    gradient,
    gradient_3d,
    gradient_f64,
    layout_size,
    library_path,
    load_library,
    noalloc_max_bytes,
    status_string,
    step,
    step_3d,
    step_f64,
    step_noalloc,
    timing_enable,
    timing_phases,
    timing_read,
    workspace_size,
    workspace_size_3d,
    workspace_size_f64,
    z_exact,
    kl,
)
