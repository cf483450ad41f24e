"""ResiSpec multi-candidate speculative verification on MI355X (gfx950).

The work is done by libresispec.so (HIP kernels behind the C ABI of
include/resispec.h); `native` is its Python binding and `synth` generates the
seeded synthetic workloads.  The binding is loaded on first use of an entry point.
"""

_API = ("resispec_verify", "resispec_verify_tree", "resispec_verify_tree_path",
        "resispec_verify_tree_path_group", "resispec_path_workspace_bytes",
        "resispec_path_group_size", "resispec_debug_set_group_waits", "resispec_verify_tree_group",
        "resispec_tree_group_workspace_bytes", "resispec_tree_group_size", "resispec_draft_candidates",
        "resispec_verify_tree_debug",
        "resispec_workspace_bytes", "resispec_validate_tree_host", "resispec_status_string",
        "resispec_abi_version")


def __getattr__(name):
    if name in _API:
        from . import native
        return getattr(native, name)
    raise AttributeError(name)
