"""MI355X-native exact grammar-constrained next-token masks (GRID's cold path).

The compute path lives in libgrid.so (HIP kernels for gfx950 plus the host
compiler behind a C ABI, include/grid.h); this package is the Python binding.
"""

from .grid import (Grid, GridError, apply, mask_noalloc, from_workload, lib, CONFIG_DTYPE, ROW_OK,  # noqa: F401
                   ROW_EMPTY, ROW_BAD_CONFIG, ROW_OVERFLOW, ROW_NOT_VIABLE, ROW_FINISHED, EXPORTS, CACHE_LOOKUP, CACHE_INSERT)
