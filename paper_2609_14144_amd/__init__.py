"""Gated early-exit batch-1 decode on MI355X (gfx950).

The compute path is the HIP library libee.so (C ABI in include/ee.h); this
package only marshals arguments to it. There is no CPU fallback: accessing the
binding without the built library raises. The binding is loaded on first use,
so `paper_2609_14144_amd.build` can run before the library exists."""

_EXPORTS = ("EEError", "Engine", "lib", "lib_path", "EE_F32", "EE_BF16", "EE_CAL_EXIT_RATE",
            "EE_CAL_MEDIAN", "EE_CAL_NUCLEUS", "EE_CONF_MAXPROB", "EE_CONF_MARGIN", "EE_CONF_NEGENTROPY",
            "EE_FILL_EAGER", "EE_FILL_LAZY")

__all__ = list(_EXPORTS)


def __getattr__(name):
    if name in _EXPORTS:
        from . import _binding
        return getattr(_binding, name)
    raise AttributeError(name)
