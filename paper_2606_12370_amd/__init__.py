"""Speculative rejection-sampling verification and fused TV loss for AMD
MI355X (gfx950).

The compute path is the C-ABI library ``libspecverify.so`` built from
``csrc/``; :mod:`.binding` marshals torch tensors into its entry points.
Importing this package does not load the library or touch the GPU; the
first call of :func:`verify` or :func:`tv_loss_fwd_bwd` does.
"""

__all__ = ["verify", "tv_loss_fwd_bwd", "verify_workspace_size", "tv_workspace_size",
           "library_path", "load_library", "workspace", "SpecError"]


def __getattr__(name):
    if name in __all__:
        from . import binding
        return getattr(binding, name)
    raise AttributeError(name)
