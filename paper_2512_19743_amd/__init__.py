"""Sparse APML loss (arXiv:2512.19743) on AMD Instinct MI355X.

The computation lives in libapml.so (hand-written HIP for gfx950, C ABI in
include/apml.h); this package only binds it.
"""
from ._lib import (  # noqa: F401
    ApmlError,
    DensePlan,
    Plan,
    apml_backward,
    apml_dense_backward,
    apml_dense_forward,
    apml_forward,
    apml_forward_backward_noalloc,
    apml_get_memory_stats,
    apml_params,
    apml_params_default,
    apml_profile_enable,
    apml_profile_read,
    apml_profile_reset,
    apml_release_cached_memory,
    apml_reset_peak_memory,
    apml_set_allocator_default,
    apml_set_allocator_torch,
    load,
)
from .loss import APMLFunction, apml_loss, loss_params  # noqa: F401
