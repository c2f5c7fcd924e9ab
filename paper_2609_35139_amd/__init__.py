"""CacheRepair repair forward pass on MI355X (gfx950).

The product is the HIP C-ABI library ``libcacherepair.so`` (declared in
``include/cacherepair.h``).  ``binding`` is its thin ctypes binding with the
same function names; ``repairer.Repairer`` adds torch device-buffer
marshalling.  There is no CPU or fallback implementation: if the library is
not built, loading it raises.
"""
from .binding import (  # noqa: F401
    CR_DTYPE_BF16, CR_DTYPE_F32, CrError, cr_chunk_schedule, cr_dims, cr_kv_layout,
    cr_prepare_weights, cr_prepared_bytes, cr_repair, cr_status_string, cr_version,
    cr_weights_layout, cr_workspace_bytes, cr_workspace_view, layer_major_layout, load,
    make_dims,
)


def __getattr__(name):
    if name == "Repairer":
        from .repairer import Repairer
        return Repairer
    raise AttributeError(name)
