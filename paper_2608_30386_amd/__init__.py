"""DASC state-checkpoint hot path for MI355X (gfx950).

Everything runs in the HIP library libdasc.so (built in-tree by
``python paper_2608_30386_amd/build.py``); this package only marshals arguments
to its C ABI (include/dasc.h).  Importing it without the built library raises
ImportError -- there is no CPU fallback.
"""

from .dasc import (  # noqa: F401
    DascError,
    Shape,
    dasc_matched_slots,
    dasc_pack,
    dasc_pack_padded,
    dasc_pack_q8,
    dasc_plan,
    dasc_refresh,
    dasc_refresh_noalloc,
    dasc_refresh_select,
    dasc_refresh_workspace_bytes,
    dasc_restore,
    dasc_restore_padded,
    dasc_restore_q8,
    dasc_restore_refresh,
    dasc_static_log_decay,
    dasc_tp_permutation,
)
