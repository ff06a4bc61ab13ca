"""PaSE strategy search (FindBestStrategy) on MI355X: C-ABI library + binding.

The search runs in ``libpase.so`` (host planner in C++, DP-table fill in HIP
kernels for gfx950); this package only loads it and marshals arguments.
"""
from .pase import (EXPORTS, LIB_PATH, OPT_BULK_US, OPT_C_SPLITS, OPT_CONFIG_SET,  # noqa: F401
                   OPT_DIRECT_CELLS, OPT_FUSED_MIN, OPT_GRAD_SYNC, OPT_HALO, OPT_KEEP_TABLES, OPT_KERNEL,
                   OPT_HOIST_ELEMS, OPT_KEY_TYPE, OPT_MEMORY_BUDGET, OPT_ORDER, OPT_PROFILE, OPT_SCHEDULE, OPT_TILE_COLS,
                   OPT_TILE_PARTS, OPT_TILE_ROWS, OPT_TRANSFER, SCHEDULE_BULK, SCHEDULE_LEVEL,
                   SCHEDULE_SEQUENTIAL, SCHEDULE_SPLIT, Graph, PaseError, load)
