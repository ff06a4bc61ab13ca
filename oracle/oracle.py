"""ctypes wrapper of the plain-C oracle (``pase_oracle.c``).

TEST INFRASTRUCTURE ONLY: imported by the tests, the smoke check and the
benchmark's CPU-baseline leg, never by the HIP library or its binding.  This
module only marshals a graph dict into flat arrays and reads results back; all
of the method's arithmetic lives in the C file.
"""
from __future__ import annotations

import ctypes as C
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "pase_oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")
MAXD = 8
_libs = {}


def build(force: bool = True, src: str = _SRC, out: str = _LIB) -> str:
    """Compile the oracle with gcc -O2 (no SIMD intrinsics) and OpenMP."""
    if force or not os.path.exists(out):
        tmp = out + ".tmp"
        subprocess.run(["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-Wall", "-o", tmp, src],
                       check=True)
        os.replace(tmp, out)
    return out


def _load(path: str | None = None):
    path = path or _LIB
    if path in _libs:
        return _libs[path]
    if path == _LIB and not os.path.exists(_LIB):
        build()
    L = C.CDLL(path)
    P, I, U64, U32 = C.c_void_p, C.c_int, C.c_uint64, C.c_uint32
    L.oracle_new.restype = P
    L.oracle_new.argtypes = [I, P, P, P, P, I, P, P, P, P, P, P, U64]
    L.oracle_free.argtypes = [P]
    L.oracle_error.restype = C.c_char_p
    L.oracle_error.argtypes = [P]
    L.oracle_configs.argtypes = [P, I]
    L.oracle_configs_all.argtypes = [P, I]
    L.oracle_set_transfer_model.argtypes = [P, I]
    L.oracle_set_weights.argtypes = [P, P, P]
    L.oracle_set_grad_sync.argtypes = [P, I]
    L.oracle_set_halo.argtypes = [P, P, P]
    L.oracle_assign_devices.argtypes = [P, P, P, P, P]
    L.oracle_set_halo_model.argtypes = [P, I]
    L.oracle_set_costs.argtypes = [P, P, P]
    L.oracle_solve.argtypes = [P, I, P, U64, I]
    L.oracle_solve_bf.argtypes = [P, U64, I]
    L.oracle_num_configs.argtypes = [P, I]
    L.oracle_config_splits.argtypes = [P, I, I, P]
    L.oracle_layer_costs.argtypes = [P, I, P]
    L.oracle_edge_costs.argtypes = [P, I, P]
    L.oracle_sequence.argtypes = [P, P]
    L.oracle_dependent_set.argtypes = [P, I, P]
    L.oracle_table_size.restype = U64
    L.oracle_table_size.argtypes = [P, I]
    L.oracle_table.argtypes = [P, I, P, P]
    L.oracle_entry.argtypes = [P, I, U64, P, P]
    L.oracle_result.argtypes = [P, P, P]
    L.oracle_cells.restype = U64
    L.oracle_cells.argtypes = [P]
    L.oracle_cells_done.restype = U64
    L.oracle_cells_done.argtypes = [P]
    L.oracle_seconds.restype = C.c_double
    L.oracle_seconds.argtypes = [P]
    L.oracle_fingerprint.argtypes = [P, I, P, P]
    _ = U32
    _libs[path] = L
    return L


def _ptr(a: np.ndarray):
    return a.ctypes.data_as(C.c_void_p)


class OracleError(RuntimeError):
    pass


class Oracle:
    """One graph, its configurations, cost tables and DP tables (CPU)."""

    def __init__(self, graph: dict, lib_path: str | None = None):
        self._L = L = _load(lib_path)
        vs, es = graph["vertices"], graph["edges"]
        nv, ne = len(vs), len(es)
        self.nv, self.ne = nv, ne
        self._keep = []
        ndims = np.array([len(v["dims"]) for v in vs], dtype=np.int32)
        sizes = np.zeros((nv, MAXD), dtype=np.uint64)
        red = np.zeros(nv, dtype=np.uint32)
        fpp = np.array([v["flops_per_point"] for v in vs], dtype=np.uint64)
        for i, v in enumerate(vs):
            sizes[i, :len(v["dims"])] = v["dims"]
            for k in v["reduce"]:
                red[i] |= np.uint32(1 << k)
        src = np.array([e["src"] for e in es] or [0], dtype=np.int32)
        dst = np.array([e["dst"] for e in es] or [0], dtype=np.int32)
        rank = np.array([len(e["src_dim"]) for e in es] or [0], dtype=np.int32)
        sdim = np.full((max(ne, 1), MAXD), -1, dtype=np.int32)
        ddim = np.full((max(ne, 1), MAXD), -1, dtype=np.int32)
        elems = np.array([e["elems"] for e in es] or [0], dtype=np.uint64)
        for i, e in enumerate(es):
            sdim[i, :len(e["src_dim"])] = e["src_dim"]
            ddim[i, :len(e["dst_dim"])] = e["dst_dim"]
        self.src, self.dst = src[:ne].copy(), dst[:ne].copy()
        self._h = L.oracle_new(nv, _ptr(ndims), _ptr(sizes), _ptr(red), _ptr(fpp), ne, _ptr(src),
                               _ptr(dst), _ptr(rank), _ptr(sdim), _ptr(ddim), _ptr(elems),
                               int(graph.get("comm_weight", 8)))
        if not self._h:
            raise OracleError("oracle_new rejected the graph")
        wmask = np.zeros(nv, dtype=np.uint32)
        wpp = np.zeros(nv, dtype=np.uint64)
        for i, v in enumerate(vs):
            for k in v.get("weight_dims", []):
                wmask[i] |= np.uint32(1 << k)
            wpp[i] = v.get("weight_per_point", 0)
        self._check(L.oracle_set_weights(self._h, _ptr(wmask), _ptr(wpp)))
        halo = np.zeros((nv, MAXD), dtype=np.uint32)
        imask = np.zeros(nv, dtype=np.uint32)
        for i, v in enumerate(vs):
            for k, w in enumerate(v.get("halo", [])):
                halo[i, k] = w
            for k in v.get("input_dims", []):
                imask[i] |= np.uint32(1 << k)
        self._check(L.oracle_set_halo(self._h, _ptr(halo), _ptr(imask)))
        self.ndims = ndims
        self.p = None

    def __del__(self):
        if getattr(self, "_h", None):
            self._L.oracle_free(self._h)
            self._h = None

    def _check(self, rc):
        if rc == 1:
            raise OracleError(self._L.oracle_error(self._h).decode())
        return rc

    # -- configurations and costs
    def configs(self, p: int, all_integers: bool = False, volume: bool = False, grad_sync: bool = False,
                halo: bool = False):
        """C(v) for p devices: power-of-two splits (p = 2^L), or with
        all_integers every tuple of positive integers with product <= p; the
        transfer costs follow the split-match model, or with `volume` the
        volume-intersection model; grad_sync adds the weight-gradient
        all-reduce to the layer costs, halo the halo exchange of
        convolutions."""
        self._check(self._L.oracle_set_transfer_model(self._h, 1 if volume else 0))
        self._check(self._L.oracle_set_grad_sync(self._h, 1 if grad_sync else 0))
        self._check(self._L.oracle_set_halo_model(self._h, 1 if halo else 0))
        fn = self._L.oracle_configs_all if all_integers else self._L.oracle_configs
        self._check(fn(self._h, int(p)))
        self.p = p
        self.K = np.array([self._L.oracle_num_configs(self._h, v) for v in range(self.nv)])
        return self.K

    def splits(self, v: int) -> np.ndarray:
        """Split factors of every configuration of v, in index order."""
        out = np.zeros((int(self.K[v]), int(self.ndims[v])), dtype=np.uint32)
        buf = np.zeros(MAXD, dtype=np.uint32)
        for c in range(int(self.K[v])):
            self._check(self._L.oracle_config_splits(self._h, v, c, _ptr(buf)))
            out[c] = buf[:self.ndims[v]]
        return out

    def exponents(self, v: int) -> np.ndarray:
        """log2 of the split factors (power-of-two configurations)."""
        sp = self.splits(v)
        ex = np.log2(sp).astype(np.uint8)
        assert np.array_equal(np.left_shift(1, ex.astype(np.uint32)), sp), "not powers of two"
        return ex

    def layer_costs(self, v: int) -> np.ndarray:
        out = np.zeros(int(self.K[v]), dtype=np.uint64)
        self._check(self._L.oracle_layer_costs(self._h, v, _ptr(out)))
        return out

    def edge_costs(self, e: int) -> np.ndarray:
        out = np.zeros((int(self.K[self.src[e]]), int(self.K[self.dst[e]])), dtype=np.uint64)
        self._check(self._L.oracle_edge_costs(self._h, e, _ptr(out)))
        return out

    def set_costs(self, layer, edge):
        lf = np.ascontiguousarray(np.concatenate([np.asarray(a, np.uint64).ravel() for a in layer]))
        ef = np.ascontiguousarray(np.concatenate([np.asarray(a, np.uint64).ravel() for a in edge]
                                                 or [np.zeros(0, np.uint64)]))
        if lf.size == 0:
            lf = np.zeros(1, np.uint64)
        if ef.size == 0:
            ef = np.zeros(1, np.uint64)
        self._check(self._L.oracle_set_costs(self._h, _ptr(lf), _ptr(ef)))

    # -- search
    def solve(self, rule: int = 0, order=None, max_cells: int = 0, threads: int = 1) -> int:
        ordp = None
        if order is not None:
            ord_arr = np.ascontiguousarray(np.asarray(order, dtype=np.int32))
            self._keep.append(ord_arr)
            ordp = _ptr(ord_arr)
        rc = self._L.oracle_solve(self._h, int(rule), ordp, int(max_cells), int(threads))
        return self._check(rc)

    def solve_bf(self, max_cells: int = 0, threads: int = 1) -> int:
        """The breadth-first recurrence (eq. 2): breadth-first order from
        vertex 0, tables B over D_B(i); read back with the same getters."""
        return self._check(self._L.oracle_solve_bf(self._h, int(max_cells), int(threads)))

    def sequence(self) -> list:
        out = np.zeros(self.nv, dtype=np.int32)
        self._check(self._L.oracle_sequence(self._h, _ptr(out)))
        return out.tolist()

    def dependent_set(self, i: int) -> list:
        """D(i) of the vertex at *position* i, sorted by vertex id."""
        out = np.zeros(self.nv, dtype=np.int32)
        n = self._L.oracle_dependent_set(self._h, i, _ptr(out))
        if n < 0:
            raise OracleError("no sequence")
        return out[:n].tolist()

    def table_size(self, i: int) -> int:
        return int(self._L.oracle_table_size(self._h, i))

    def table(self, i: int):
        n = self.table_size(i)
        T = np.zeros(n, dtype=np.uint64)
        A = np.zeros(n, dtype=np.uint16)
        self._check(self._L.oracle_table(self._h, i, _ptr(T), _ptr(A)))
        return T, A

    def entry(self, i: int, idx: int):
        t = np.zeros(1, np.uint64)
        a = np.zeros(1, np.uint32)
        self._check(self._L.oracle_entry(self._h, i, int(idx), _ptr(t), _ptr(a)))
        return int(t[0]), int(a[0])

    def result(self):
        mc = np.zeros(1, np.uint64)
        st = np.zeros(self.nv, np.int32)
        self._check(self._L.oracle_result(self._h, _ptr(mc), _ptr(st)))
        return int(mc[0]), st.tolist()

    def assign_devices(self, strategy):
        """Greedy device assignment of `strategy` (configuration per vertex id):
        (dev [nv, p] -- the part of each vertex on each device, -1 for none --,
        locality [ne] in elements, r * t_x [ne] under the assignment)."""
        cfg = np.ascontiguousarray(np.asarray(strategy, dtype=np.int32))
        dev = np.zeros((self.nv, int(self.p)), dtype=np.int32)
        loc = np.zeros(max(len(self.src), 1), dtype=np.uint64)
        xfer = np.zeros(max(len(self.src), 1), dtype=np.uint64)
        self._check(self._L.oracle_assign_devices(self._h, _ptr(cfg), _ptr(dev), _ptr(loc), _ptr(xfer)))
        ne = len(self.src)
        return dev, loc[:ne], xfer[:ne]

    def fingerprint(self, i: int):
        a = np.zeros(1, np.uint64)
        b = np.zeros(1, np.uint64)
        self._check(self._L.oracle_fingerprint(self._h, i, _ptr(a), _ptr(b)))
        return int(a[0]), int(b[0])

    def cells(self) -> int:
        return int(self._L.oracle_cells(self._h))

    def cells_done(self) -> int:
        return int(self._L.oracle_cells_done(self._h))

    def seconds(self) -> float:
        return float(self._L.oracle_seconds(self._h))


def solve_graph(graph: dict, p: int | None = None, rule: int = 0, threads: int = 1,
                costs=None, lib_path: str | None = None) -> Oracle:
    o = Oracle(graph, lib_path)
    o.configs(p if p is not None else graph["p"])
    if costs is not None:
        o.set_costs(*costs)
    o.solve(rule=rule, threads=threads)
    return o
