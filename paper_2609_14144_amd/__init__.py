"""Gated early-exit batch-1 decode on MI355X (gfx950).

The compute path is the HIP library libee.so (C ABI in include/ee.h); this
package only marshals arguments to it. There is no CPU fallback: importing
the binding without the built library raises."""
from ._binding import (EEError, Engine, lib, lib_path, EE_F32, EE_BF16, EE_CAL_EXIT_RATE,
                       EE_CAL_MEDIAN)

__all__ = ["EEError", "Engine", "lib", "lib_path", "EE_F32", "EE_BF16", "EE_CAL_EXIT_RATE",
           "EE_CAL_MEDIAN"]
