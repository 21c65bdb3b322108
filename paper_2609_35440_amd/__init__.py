"""SOLO shared-readout local loss on MI355X (gfx950).

The hot path is a C-ABI shared library (``libsolo_readout.so``, declared in
``include/solo_readout.h``) of hand-written HIP kernels; this package holds its
sources (``csrc/``), the thin ctypes binding (``binding``), the build step
(``build``) and the FLOP/byte accounting (``costmodel``).
"""
from . import costmodel  # noqa: F401

__all__ = ["costmodel", "readout_fwd_bwd", "workspace_size", "load_library", "SoloError"]


def __getattr__(name):
    # the binding loads the HIP library; import it only when asked for
    if name in ("readout_fwd_bwd", "workspace_size", "load_library", "SoloError", "binding"):
        import importlib

        binding = importlib.import_module(__name__ + ".binding")
        return binding if name == "binding" else getattr(binding, name)
    raise AttributeError(name)
