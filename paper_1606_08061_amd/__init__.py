"""Exact output-layer training step for very large sparse targets, on gfx950 (MI355X).

The HIP library liblst.so (C ABI in include/lst.h) implements the factored
step of Vincent, de Brebisson and Bouthillier (arXiv 1606.08061), the
numerical stabilisation of its section 5 and a naive O(D d) comparison path;
this package is its ctypes binding.
"""
from ._binding import (  # noqa: F401
    LIB_PATH, LOSSES, LST_E_ARG, LST_E_HIP, LST_E_INDEX, LST_E_NONFINITE, LST_E_NOT_SPD,
    LST_E_SHAPE, LST_E_STATE, LST_E_SYNC, LST_LOSS_SPHERICAL_SOFTMAX, LST_LOSS_SQUARED,
    LST_LOSS_TAYLOR_SOFTMAX, LST_OK, SIGNATURES,
    Factored, LstError, Naive, lib, library_path, lst_create, lst_destroy, lst_init_factored,
    lst_materialize_W, lst_naive_create, lst_naive_step, lst_profile_enable, lst_profile_read,
    lst_use_graphs, lst_restore_pristine, lst_refresh_uinvt, lst_power_iteration,
    lst_fix_singular_value, lst_singular_stabilize, lst_input_forward, lst_input_update,
    SparseInput, LST_OPT_ONLINE_KERNEL, LST_OPT_SPIN_LIMIT, lst_set_option, lst_workspace_bytes,
    lst_naive_workspace_bytes, lst_step_noalloc,
    lst_step, lst_sync_status, status_string, PHASES,
)
