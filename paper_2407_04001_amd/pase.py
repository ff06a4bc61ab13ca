"""Python binding of libpase (ctypes).

Argument marshalling only: every step of the strategy search runs inside
libpase.so (host planner + gfx950 kernels).  Functions carry the names of the
C ABI in ``include/pase.h``; ``Graph`` bundles them for convenience.  PyTorch,
when present, supplies the stream and the device workspace.
"""
from __future__ import annotations

import ctypes as C
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libpase.so")
MAX_DIMS = 8

OK, INVALID_ARGUMENT, NOT_CONNECTED, BAD_STATE, OVERFLOW, TOO_LARGE, OUT_OF_MEMORY, HIP, INTERNAL = range(9)
STATUS_NAMES = {0: "OK", 1: "INVALID_ARGUMENT", 2: "NOT_CONNECTED", 3: "BAD_STATE", 4: "OVERFLOW",
                5: "TOO_LARGE", 6: "OUT_OF_MEMORY", 7: "HIP", 8: "INTERNAL"}
(OPT_KEEP_TABLES, OPT_MEMORY_BUDGET, OPT_KERNEL, OPT_KEY_TYPE, OPT_PROFILE, OPT_SCHEDULE,
 OPT_TILE_COLS, OPT_TILE_ROWS, OPT_TILE_PARTS, OPT_C_SPLITS) = range(1, 11)
(OPT_CONFIG_SET, OPT_ORDER, OPT_TRANSFER, OPT_GRAD_SYNC, OPT_DIRECT_CELLS, OPT_BULK_US) = range(12, 18)
OPT_HALO = 19
OPT_FUSED_MIN = 20
OPT_HOIST_ELEMS = 21
SCHEDULE_LEVEL, SCHEDULE_SEQUENTIAL, SCHEDULE_BULK, SCHEDULE_SPLIT = 0, 1, 4, 5


class VertexDesc(C.Structure):
    _fields_ = [("ndims", C.c_uint32), ("size", C.c_uint64 * MAX_DIMS), ("reduce_mask", C.c_uint32),
                ("flops_per_point", C.c_uint64), ("weight_mask", C.c_uint32), ("weight_per_point", C.c_uint64),
                ("input_mask", C.c_uint32), ("halo", C.c_uint32 * MAX_DIMS)]


class EdgeDesc(C.Structure):
    _fields_ = [("src", C.c_uint32), ("dst", C.c_uint32), ("rank", C.c_uint32),
                ("src_dim", C.c_int32 * MAX_DIMS), ("dst_dim", C.c_int32 * MAX_DIMS),
                ("elems", C.c_uint64)]


class CostParams(C.Structure):
    _fields_ = [("comm_weight", C.c_uint64), ("seq_rule", C.c_uint32)]


class RunStats(C.Structure):
    _fields_ = [("cells", C.c_uint64), ("table_entries", C.c_uint64), ("workspace_bytes", C.c_uint64),
                ("max_dep", C.c_uint32), ("key_type", C.c_uint32), ("launches", C.c_uint32),
                ("rows_vertices", C.c_uint32), ("rows_cells", C.c_uint64), ("host_plan_ms", C.c_double),
                ("wall_ms", C.c_double), ("fill_ms", C.c_double), ("rows_fill_ms", C.c_double),
                ("rows_launches", C.c_uint32), ("slots", C.c_uint32), ("stream_cells", C.c_uint64),
                ("stream_fill_ms", C.c_double), ("stream_launches", C.c_uint32), ("schedule", C.c_uint32),
                ("pad0", C.c_uint32), ("seq_ms", C.c_double), ("plan_ms", C.c_double), ("setup_ms", C.c_double),
                ("cost_tables_ms", C.c_double), ("fill_span_ms", C.c_double), ("backtrack_ms", C.c_double),
                ("assign_ms", C.c_double)]

    def as_dict(self):
        return {k: getattr(self, k) for k, _ in self._fields_}


class VertexInfo(C.Structure):
    _fields_ = [("position", C.c_uint32), ("kernel", C.c_uint32), ("num_configs", C.c_uint32),
                ("dep_count", C.c_uint32), ("entries", C.c_uint64), ("cells", C.c_uint64),
                ("column", C.c_int32), ("outer", C.c_uint32), ("rows", C.c_uint32),
                ("tile_cols", C.c_uint32), ("tile_rows", C.c_uint32), ("splits", C.c_uint32),
                ("row_terms", C.c_uint32), ("lookups", C.c_uint32), ("parts", C.c_uint32),
                ("fill_ms", C.c_double), ("level", C.c_uint32), ("lane", C.c_uint32),
                ("key_bound", C.c_uint64), ("table_bound", C.c_uint64), ("key_type", C.c_uint32),
                ("fused", C.c_uint32), ("prep_after", C.c_int32), ("prep_lane", C.c_uint32)]

    def as_dict(self):
        return {k: getattr(self, k) for k, _ in self._fields_}


EXPORTS = ["pase_graph_create", "pase_graph_destroy", "pase_last_error", "pase_enumerate_configs",
           "pase_num_configs", "pase_config_splits", "pase_get_sequence", "pase_get_dependent_set",
           "pase_set_option", "pase_override_costs", "pase_workspace_size", "pase_set_workspace",
           "pase_find_best_strategy", "pase_table_entry", "pase_table_fingerprint",
           "pase_layer_costs", "pase_edge_costs", "pase_stats", "pase_vertex_info_get",
           "pase_find_best_strategy_noalloc", "pase_plan_check", "pase_assign_devices"]

_lib = None


def load(path: str | None = None):
    """Load libpase.so (``LIB_PATH`` unless a path is given); raises if the
    HIP library has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    path = path or LIB_PATH
    if not os.path.exists(path):
        raise ImportError(f"libpase.so not found at {path}: build it with "
                          "`python -c 'import __graft_entry__ as g; g.build()'`")
    L = C.CDLL(path)
    P, U32, U64 = C.c_void_p, C.c_uint32, C.c_uint64
    st = C.c_int
    sig = {
        "pase_graph_create": (st, [P, U32, P, U32, P, P]),
        "pase_graph_destroy": (None, [P]),
        "pase_last_error": (C.c_char_p, [P]),
        "pase_enumerate_configs": (st, [P, U32]),
        "pase_num_configs": (st, [P, U32, P]),
        "pase_config_splits": (st, [P, U32, U32, P]),
        "pase_get_sequence": (st, [P, P]),
        "pase_get_dependent_set": (st, [P, U32, P, U32, P]),
        "pase_set_option": (st, [P, C.c_int, U64]),
        "pase_override_costs": (st, [P, P, P]),
        "pase_workspace_size": (st, [P, P]),
        "pase_set_workspace": (st, [P, P, U64]),
        "pase_find_best_strategy": (st, [P, P, P, P]),
        "pase_find_best_strategy_noalloc": (st, [P, P, P, P]),
        "pase_plan_check": (st, [P, P]),
        "pase_assign_devices": (st, [P, P, P, P, P]),
        "pase_table_entry": (st, [P, U32, P, P, P]),
        "pase_table_fingerprint": (st, [P, U32, P, P]),
        "pase_layer_costs": (st, [P, U32, P]),
        "pase_edge_costs": (st, [P, U32, P]),
        "pase_stats": (st, [P, P]),
        "pase_vertex_info_get": (st, [P, U32, P]),
    }
    for name, (res, args) in sig.items():
        f = getattr(L, name)
        f.restype = res
        f.argtypes = args
    _lib = L
    return L


class PaseError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"{STATUS_NAMES.get(status, status)}: {msg}")
        self.status = status


def _ptr(a: np.ndarray):
    return a.ctypes.data_as(C.c_void_p)


def _check(h, rc):
    if rc != OK:
        msg = load().pase_last_error(h).decode() if h else ""
        raise PaseError(rc, msg)


# ------------------------------------------------------------------ C-ABI mirrors
def pase_graph_create(vertices, edges, comm_weight: int = 8, seq_rule: int = 0):
    """vertices: list of dicts {dims, reduce, flops_per_point}; edges: list of
    dicts {src, dst, src_dim, dst_dim, elems} (the layout of workloads.gen)."""
    L = load()
    nv, ne = len(vertices), len(edges)
    V = (VertexDesc * max(nv, 1))()
    for i, v in enumerate(vertices):
        V[i].ndims = len(v["dims"])
        for k, n in enumerate(v["dims"]):
            V[i].size[k] = int(n)
        V[i].reduce_mask = sum(1 << int(k) for k in v["reduce"])
        V[i].flops_per_point = int(v["flops_per_point"])
        V[i].weight_mask = sum(1 << int(k) for k in v.get("weight_dims", []))
        V[i].weight_per_point = int(v.get("weight_per_point", 0))
        V[i].input_mask = sum(1 << int(k) for k in v.get("input_dims", []))
        for k, w in enumerate(v.get("halo", [])):
            V[i].halo[k] = int(w)
    E = (EdgeDesc * max(ne, 1))()
    for i, e in enumerate(edges):
        E[i].src, E[i].dst, E[i].rank = int(e["src"]), int(e["dst"]), len(e["src_dim"])
        for k in range(MAX_DIMS):
            E[i].src_dim[k] = int(e["src_dim"][k]) if k < len(e["src_dim"]) else -1
            E[i].dst_dim[k] = int(e["dst_dim"][k]) if k < len(e["dst_dim"]) else -1
        E[i].elems = int(e["elems"])
    params = CostParams(int(comm_weight), int(seq_rule))
    h = C.c_void_p()
    rc = L.pase_graph_create(C.byref(V), nv, C.byref(E) if ne else None, ne, C.byref(params), C.byref(h))
    _check(None, rc)
    return h.value


def pase_graph_destroy(h):
    load().pase_graph_destroy(h)


def pase_enumerate_configs(h, p: int):
    _check(h, load().pase_enumerate_configs(h, int(p)))


def pase_num_configs(h, v: int) -> int:
    k = C.c_uint32()
    _check(h, load().pase_num_configs(h, int(v), C.byref(k)))
    return k.value


def pase_config_splits(h, v: int, idx: int, ndims: int):
    out = np.zeros(MAX_DIMS, np.uint32)
    _check(h, load().pase_config_splits(h, int(v), int(idx), _ptr(out)))
    return out[:ndims].tolist()


def pase_get_sequence(h, nv: int):
    out = np.zeros(nv, np.uint32)
    _check(h, load().pase_get_sequence(h, _ptr(out)))
    return out.tolist()


def pase_get_dependent_set(h, v: int, cap: int = 64):
    out = np.zeros(cap, np.uint32)
    n = C.c_uint32()
    _check(h, load().pase_get_dependent_set(h, int(v), _ptr(out), cap, C.byref(n)))
    return out[:n.value].tolist()


def pase_set_option(h, opt: int, value: int):
    _check(h, load().pase_set_option(h, int(opt), int(value)))


def pase_override_costs(h, layer, edge):
    lf = np.ascontiguousarray(np.concatenate([np.asarray(a, np.uint64).ravel() for a in layer]))
    ef = (np.ascontiguousarray(np.concatenate([np.asarray(a, np.uint64).ravel() for a in edge]))
          if len(edge) else np.zeros(1, np.uint64))
    _check(h, load().pase_override_costs(h, _ptr(lf), _ptr(ef)))


def pase_workspace_size(h) -> int:
    b = C.c_uint64()
    _check(h, load().pase_workspace_size(h, C.byref(b)))
    return b.value


def pase_set_workspace(h, device_ptr: int, nbytes: int):
    _check(h, load().pase_set_workspace(h, C.c_void_p(device_ptr) if device_ptr else None, int(nbytes)))


def pase_find_best_strategy(h, nv: int, stream: int = 0):
    mc = C.c_uint64()
    cfg = np.zeros(nv, np.uint32)
    _check(h, load().pase_find_best_strategy(h, C.c_void_p(stream) if stream else None, C.byref(mc),
                                             _ptr(cfg)))
    return mc.value, cfg.tolist()


def pase_find_best_strategy_noalloc(h, nv: int, stream: int = 0):
    mc = C.c_uint64()
    cfg = np.zeros(nv, np.uint32)
    _check(h, load().pase_find_best_strategy_noalloc(h, C.c_void_p(stream) if stream else None, C.byref(mc),
                                                     _ptr(cfg)))
    return mc.value, cfg.tolist()


NOALLOC_WORKSPACE_BYTES = 64 << 20


def pase_table_entry(h, v: int, dep_cfg):
    d = np.ascontiguousarray(np.asarray(list(dep_cfg) or [0], np.uint32))
    cost, arg = C.c_uint64(), C.c_uint32()
    _check(h, load().pase_table_entry(h, int(v), _ptr(d), C.byref(cost), C.byref(arg)))
    return cost.value, arg.value


def pase_table_fingerprint(h, v: int):
    a, b = C.c_uint64(), C.c_uint64()
    _check(h, load().pase_table_fingerprint(h, int(v), C.byref(a), C.byref(b)))
    return a.value, b.value


def pase_layer_costs(h, v: int, k: int):
    out = np.zeros(k, np.uint64)
    _check(h, load().pase_layer_costs(h, int(v), _ptr(out)))
    return out


def pase_edge_costs(h, e: int, ku: int, kv: int):
    out = np.zeros((ku, kv), np.uint64)
    _check(h, load().pase_edge_costs(h, int(e), _ptr(out)))
    return out


def pase_stats(h) -> dict:
    s = RunStats()
    _check(h, load().pase_stats(h, C.byref(s)))
    return s.as_dict()


def pase_vertex_info_get(h, v: int) -> dict:
    x = VertexInfo()
    _check(h, load().pase_vertex_info_get(h, int(v), C.byref(x)))
    return x.as_dict()


def pase_plan_check(h) -> int:
    b = C.c_uint64()
    _check(h, load().pase_plan_check(h, C.byref(b)))
    return b.value


def pase_assign_devices(h, config_idx, nv: int, ne: int, p: int):
    cfg = np.ascontiguousarray(np.asarray(config_idx, np.uint32))
    if cfg.shape != (nv,):
        raise ValueError(f"strategy of {cfg.size} configurations for {nv} vertices")
    dev = np.zeros((nv, p), np.int32)
    loc = np.zeros(max(ne, 1), np.uint64)
    xfer = np.zeros(max(ne, 1), np.uint64)
    _check(h, load().pase_assign_devices(h, _ptr(cfg), _ptr(dev), _ptr(loc), _ptr(xfer)))
    return dev, loc[:ne], xfer[:ne]


# ------------------------------------------------------------------ convenience wrapper
class Graph:
    """A computation graph handle.  ``graph`` is a dict in the layout of
    ``workloads.gen`` (vertices, edges, comm_weight)."""

    def __init__(self, graph: dict, seq_rule: int = 0):
        self.nv = len(graph["vertices"])
        self.ne = len(graph["edges"])
        self.graph = graph
        self.h = pase_graph_create(graph["vertices"], graph["edges"], graph.get("comm_weight", 8),
                                   seq_rule)
        self._ws = None
        self._K = None

    def close(self):
        if getattr(self, "h", None):
            pase_graph_destroy(self.h)
            self.h = None
            self._ws = None

    def __del__(self):
        try:
            self.close()
        except (TypeError, AttributeError):   # interpreter shutdown: module globals are gone
            pass

    def enumerate_configs(self, p: int, all_integers: bool | None = None):
        """Enumerate configurations and plan the search for p devices; the
        per-vertex configuration counts are read lazily through `K`.
        all_integers (when given) sets OPT_CONFIG_SET first: every positive
        integer split instead of the power-of-two ones."""
        if all_integers is not None:
            pase_set_option(self.h, OPT_CONFIG_SET, 1 if all_integers else 0)
        pase_enumerate_configs(self.h, p)
        self.p = int(p)
        self._K = None

    @property
    def K(self):
        if self._K is None:
            self._K = [pase_num_configs(self.h, v) for v in range(self.nv)]
        return self._K

    def set_option(self, opt: int, value: int):
        pase_set_option(self.h, opt, value)

    def override_costs(self, layer, edge):
        pase_override_costs(self.h, layer, edge)

    def sequence(self):
        return pase_get_sequence(self.h, self.nv)

    def dependent_set(self, v: int):
        return pase_get_dependent_set(self.h, v)

    def config_splits(self, v: int, idx: int):
        return pase_config_splits(self.h, v, idx, len(self.graph["vertices"][v]["dims"]))

    def workspace_size(self) -> int:
        return pase_workspace_size(self.h)

    def find_best_strategy(self, stream=None, torch_workspace: bool = True):
        """Run the search on the current HIP device.  With torch available the
        workspace is a torch allocation and the stream torch's current one."""
        s = 0
        try:
            import torch
            if torch.cuda.is_available():
                if stream is None:
                    stream = torch.cuda.current_stream()
                s = stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream)
                if torch_workspace:
                    need = self.workspace_size()
                    if self._ws is None or self._ws.numel() < need:
                        self._ws = torch.empty(max(need, 256), dtype=torch.uint8, device="cuda")
                        pase_set_workspace(self.h, self._ws.data_ptr(), self._ws.numel())
        except ImportError:
            s = int(stream or 0)
        return pase_find_best_strategy(self.h, self.nv, s)

    def table_entry(self, v: int, dep_cfg):
        return pase_table_entry(self.h, v, dep_cfg)

    def fingerprint(self, v: int):
        return pase_table_fingerprint(self.h, v)

    def layer_costs(self, v: int):
        return pase_layer_costs(self.h, v, self.K[v])

    def edge_costs(self, e: int):
        ed = self.graph["edges"][e]
        return pase_edge_costs(self.h, e, self.K[ed["src"]], self.K[ed["dst"]])

    def stats(self) -> dict:
        return pase_stats(self.h)

    def vertex_info(self, v: int) -> dict:
        return pase_vertex_info_get(self.h, v)

    def plan_check(self) -> int:
        return pase_plan_check(self.h)

    def assign_devices(self, strategy):
        """Greedy device assignment of a strategy: (devices [nv, p] = part on
        each device or -1, edge locality [ne], edge r * t_x [ne])."""
        return pase_assign_devices(self.h, strategy, self.nv, self.ne, self.p)
