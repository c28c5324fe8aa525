"""Nested-Winograd stride-1 2D convolution for MI355X (gfx950).

The compute lives in the HIP library ``libnwg.so`` (C ABI in
``include/nwg.h``); ``paper_2102_13272_amd.nwg`` binds it with ctypes.
"""
from .nwg import (NWG_EHIP, NWG_EINVAL, NWG_ENOMEM, NWG_EUNSUPPORTED, NWG_OK,  # noqa: F401
                  NWG_TILE_F2X2_3X3, NwgError, Plan, load_library, plan_geometry)
