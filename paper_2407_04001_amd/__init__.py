"""PaSE strategy search (FindBestStrategy) on MI355X: C-ABI library + binding.

The search runs in ``libpase.so`` (host planner in C++, DP-table fill in HIP
kernels for gfx950); this package only loads it and marshals arguments.
"""
from .pase import (EXPORTS, LIB_PATH, OPT_KEEP_TABLES, OPT_KERNEL, OPT_KEY_TYPE,  # noqa: F401
                   OPT_MEMORY_BUDGET, OPT_PROFILE, OPT_SCHEDULE, OPT_TILE_COLS, OPT_TILE_ROWS,
                   OPT_TILE_PARTS, OPT_C_SPLITS, OPT_LATENCY_WORKERS, OPT_CONFIG_SET, OPT_ORDER, OPT_TRANSFER, OPT_GRAD_SYNC, OPT_DIRECT_CELLS, OPT_BULK_US,
                   Graph, PaseError, load)
