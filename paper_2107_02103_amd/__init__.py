"""MI355X (gfx950) implementation of the compressed se_a descriptor of
DP Compress (arXiv:2107.02103): a C-ABI library (libdpc.so, HIP kernels and
a host table builder) and its thin Python binding.

Importing the package does not load the library (so that ``build`` can run
on a fresh tree); the first use of any binding name loads it and raises
ImportError if it has not been built."""
_BINDING = ("DPC_F32", "DPC_F32_ACC64", "DPC_F64", "DPC_OK", "DPC_EINVAL", "DPC_ERANGE",
            "DPC_EHIP", "DPC_ENOTSUP", "DPC_EOVERFLOW", "DPC_NLIST_NOALLOC_MAX_ATOMS", "DpcError", "build_tables", "dpc_build_table",
            "dpc_descriptor_bwd", "dpc_env_mat_a", "dpc_fitting_fwd_bwd", "dpc_fitting_net",
            "dpc_fitting_workspace_bytes", "dpc_force_a", "dpc_last_hip_error", "RocblasHandle",
            "dpc_nlist_reverse", "dpc_nlist_workspace_bytes", "dpc_nlist_build",
            "dpc_nlist_build_noalloc", "dpc_se_a_tab_bwd", "dpc_se_a_tab_bwd_from_dD", "dpc_se_a_tab_fwd", "dpc_strerror",
            "dpc_table_layout", "dpc_version", "make_ranges")


def __getattr__(name):
    if name in _BINDING:
        from . import binding
        return getattr(binding, name)
    if name == "SeATab":
        from .descriptor import SeATab
        return SeATab
    raise AttributeError(name)
