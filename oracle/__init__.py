"""CPU oracle for batched backward dataflow enumeration (ctypes wrapper).

TEST INFRASTRUCTURE ONLY: the tests, the smoke check and the benchmark's
CPU-baseline leg may use this package; the product library never imports,
links or calls it.  The oracle is a plain per-location dynamic program over
the back-projection of Sec. 3.4 (see dg_oracle.cpp for the definition and
the readings taken where the paper is silent).

Parity status: every op kind is pinned by tests that do not reuse the
oracle's own loops: perturbation of real PyTorch fp64 ops (footprint sets),
autograd of linearised PyTorch graphs (path counts), literal tree expansion
of res (the dynamic program), closed forms of the five workloads, and the
worked example of the paper.
"""

from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "dg_oracle.cpp")
_LIB = os.path.join(_HERE, "libdgoracle.so")
_lib = None


def build(force: bool = True) -> str:
    """Compile the oracle with g++ (host only)."""
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp"
        subprocess.check_call(["g++", "-O2", "-std=c++17", "-shared", "-fPIC", "-pthread",
                               _SRC, "-o", tmp])
        os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB):
        build()
    lib = ctypes.CDLL(_LIB)
    P = ctypes.c_void_p
    i64 = ctypes.c_int64
    lib.dgo_error.restype = ctypes.c_char_p
    lib.dgo_parse.argtypes = [ctypes.c_char_p, i64]
    lib.dgo_parse.restype = P
    lib.dgo_free.argtypes = [P]
    lib.dgo_output_numel.argtypes = [P]
    lib.dgo_output_numel.restype = i64
    lib.dgo_num_leaves.argtypes = [P]
    lib.dgo_num_tensors.argtypes = [P]
    lib.dgo_output_tensor.argtypes = [P]
    lib.dgo_leaf_total.argtypes = [P]
    lib.dgo_leaf_total.restype = ctypes.c_uint64
    lib.dgo_tensor_info.argtypes = [P, ctypes.c_int, ctypes.c_char_p, ctypes.c_int, P, P, P, P]
    lib.dgo_enumerate.argtypes = [P, P, i64, ctypes.c_int, ctypes.c_int]
    lib.dgo_enumerate.restype = P
    lib.dgo_result_total.argtypes = [P]
    lib.dgo_result_total.restype = i64
    lib.dgo_result_copy.argtypes = [P, P, P, P]
    lib.dgo_result_copy_wide.argtypes = [P, P, P, P]
    lib.dgo_result_free.argtypes = [P]
    lib.dgo_compare.argtypes = [P, P, P, i64, ctypes.c_int, P]
    lib.dgo_tensor_gid.argtypes = [P, ctypes.c_int]
    lib.dgo_tensor_gid.restype = ctypes.c_uint64
    lib.dgo_dag_build.argtypes = [P, P, i64, ctypes.c_int]
    lib.dgo_dag_build.restype = P
    lib.dgo_dag_totals.argtypes = [P, P, P]
    lib.dgo_dag_copy.argtypes = [P, P, P, P, P, P, P]
    lib.dgo_dag_free.argtypes = [P]
    lib.dgo_reads.argtypes = [P, ctypes.c_int, i64, P, P, P, i64]
    lib.dgo_reads.restype = i64
    lib.dgo_order_prefix.argtypes = [P, i64, i64, P, i64]
    lib.dgo_order_prefix.restype = i64
    lib.dgo_permutation.argtypes = [i64, ctypes.c_uint64, i64, i64, P]
    lib.dgo_feistel.argtypes = [i64, ctypes.c_uint64, ctypes.c_int, P, i64, P]
    lib.dgo_splitmix.argtypes = [ctypes.c_uint64, i64, P]
    lib.dgo_merge.argtypes = [P, P, ctypes.c_int, ctypes.c_char_p, i64, P]
    lib.dgo_merge.restype = i64
    _lib = lib
    return lib


class OracleError(RuntimeError):
    pass


class TensorInfo:
    def __init__(self, name, shape, leaf_index, base):
        self.name = name
        self.shape = tuple(shape)
        self.leaf_index = leaf_index
        self.base = base

    @property
    def numel(self):
        n = 1
        for s in self.shape:
            n *= s
        return n


class Graph:
    """A parsed dgir graph held by the oracle."""

    def __init__(self, text: str):
        lib = _load()
        data = text.encode()
        self._h = lib.dgo_parse(data, len(data))
        if not self._h:
            raise OracleError(lib.dgo_error().decode())
        self.tensors = []
        for t in range(lib.dgo_num_tensors(self._h)):
            name = ctypes.create_string_buffer(128)
            shape = (ctypes.c_int64 * 8)()
            rank = ctypes.c_int()
            li = ctypes.c_int()
            base = ctypes.c_uint64()
            lib.dgo_tensor_info(self._h, t, name, 128, ctypes.addressof(shape), ctypes.addressof(rank),
                                ctypes.addressof(li), ctypes.addressof(base))
            self.tensors.append(TensorInfo(name.value.decode(), shape[: rank.value], li.value, base.value))
        self.output = lib.dgo_output_tensor(self._h)
        self.leaves = [t for t in self.tensors if t.leaf_index >= 0]
        self.leaf_total = lib.dgo_leaf_total(self._h)

    def __del__(self):
        if getattr(self, "_h", None):
            _load().dgo_free(self._h)
            self._h = None

    @property
    def output_shape(self):
        return self.tensors[self.output].shape

    @property
    def output_numel(self):
        return self.tensors[self.output].numel

    def tensor_index(self, name: str) -> int:
        for i, t in enumerate(self.tensors):
            if t.name == name:
                return i
        raise KeyError(name)

    def enumerate(self, locs, threads: int = 1, wide: bool = False):
        """CSR of the footprints: (offsets int64[n+1], ids, counts), ids and
        counts uint32 (wide=False) or uint64 (wide=True)."""
        lib = _load()
        locs = np.ascontiguousarray(np.asarray(locs, dtype=np.int64))
        r = lib.dgo_enumerate(self._h, locs.ctypes.data, len(locs), threads, int(wide))
        if not r:
            raise OracleError(lib.dgo_error().decode())
        try:
            total = lib.dgo_result_total(r)
            offsets = np.empty(len(locs) + 1, dtype=np.int64)
            dt = np.uint64 if wide else np.uint32
            ids = np.empty(total, dtype=dt)
            counts = np.empty(total, dtype=dt)
            copy = lib.dgo_result_copy_wide if wide else lib.dgo_result_copy
            copy(r, offsets.ctypes.data, ids.ctypes.data, counts.ctypes.data)
        finally:
            lib.dgo_result_free(r)
        return offsets, ids, counts

    def row(self, loc: int):
        """{global id: path count} of one location."""
        off, ids, cnt = self.enumerate([loc])
        return dict(zip(ids.tolist(), cnt.tolist()))

    def gid(self, tensor: int) -> int:
        """Global id of element 0 of a tensor: its leaf base, or for an op
        output leaf_total plus the element counts of the earlier ops."""
        return _load().dgo_tensor_gid(self._h, tensor)

    def dag(self, locs, threads: int = 1):
        """Expression DAGs of res(y[l]) per location, as a dict of arrays:
        node_offsets, edge_offsets (int64[n+1]); nodes, node_edge, edges,
        mults (uint64).  Nodes are the non-leaf cone elements (ops in reverse
        SSA order, elements ascending); node_edge is each node's first edge
        relative to its location's first edge; edges are child global ids
        in equation order with their multiplicities."""
        lib = _load()
        locs = np.ascontiguousarray(np.asarray(locs, dtype=np.int64))
        h = lib.dgo_dag_build(self._h, locs.ctypes.data, len(locs), threads)
        if not h:
            raise OracleError(lib.dgo_error().decode())
        try:
            nn, ne = ctypes.c_int64(), ctypes.c_int64()
            lib.dgo_dag_totals(h, ctypes.byref(nn), ctypes.byref(ne))
            r = {"node_offsets": np.empty(len(locs) + 1, np.int64), "edge_offsets": np.empty(len(locs) + 1, np.int64),
                 "nodes": np.empty(nn.value, np.uint64), "node_edge": np.empty(nn.value, np.uint64),
                 "edges": np.empty(ne.value, np.uint64), "mults": np.empty(ne.value, np.uint64)}
            lib.dgo_dag_copy(h, *(r[k].ctypes.data for k in ("node_offsets", "edge_offsets", "nodes", "node_edge",
                                                             "edges", "mults")))
        finally:
            lib.dgo_dag_free(h)
        return r

    def reads(self, tensor: int, loc: int):
        """R_k(l) of the op writing ``tensor``: list of (tensor, flat index, multiplicity)."""
        lib = _load()
        cap = 1 << 16
        while True:
            t = np.empty(cap, dtype=np.int32)
            i = np.empty(cap, dtype=np.int64)
            m = np.empty(cap, dtype=np.uint64)
            n = lib.dgo_reads(self._h, tensor, loc, t.ctypes.data, i.ctypes.data, m.ctypes.data, cap)
            if n < 0:
                raise OracleError(lib.dgo_error().decode())
            if n <= cap:
                return list(zip(t[:n].tolist(), i[:n].tolist(), m[:n].tolist()))
            cap = n


def compare(a: Graph, b: Graph, locs, threads: int = 1) -> np.ndarray:
    """Per-location status: 0 equal, 1 footprints differ, 2 only counts differ."""
    lib = _load()
    locs = np.ascontiguousarray(np.asarray(locs, dtype=np.int64))
    status = np.empty(len(locs), dtype=np.uint8)
    if lib.dgo_compare(a._h, b._h, locs.ctypes.data, len(locs), threads, status.ctypes.data) != 0:
        raise OracleError(lib.dgo_error().decode())
    return status


# ---- location order (Sec. 4, "Search Heuristic") ------------------------------
def order_prefix(g: Graph, threads: int = 256, warp: int = 32) -> list[int]:
    """Corner locations of every op (later ops first), then the first and
    last output location, each once (see dg_oracle.cpp)."""
    lib = _load()
    n = lib.dgo_order_prefix(g._h, threads, warp, None, 0)
    if n < 0:
        raise OracleError(lib.dgo_error().decode())
    out = np.empty(max(1, n), dtype=np.int64)
    lib.dgo_order_prefix(g._h, threads, warp, out.ctypes.data, n)
    return out[:n].tolist()


def permutation(n: int, seed: int, first: int = 0, count: int | None = None) -> np.ndarray:
    """Positions [first, first + count) of the keyed permutation of [0, n)."""
    count = n - first if count is None else count
    out = np.empty(max(1, count), dtype=np.int64)
    _load().dgo_permutation(n, seed & ((1 << 64) - 1), first, count, out.ctypes.data)
    return out[:count]


def feistel(n: int, seed: int, x, inverse: bool = False) -> np.ndarray:
    """The Feistel network of the permutation of [0, n) without cycle walking."""
    x = np.ascontiguousarray(np.asarray(x, dtype=np.uint64))
    out = np.empty(max(1, len(x)), dtype=np.uint64)
    _load().dgo_feistel(n, seed & ((1 << 64) - 1), 1 if inverse else 0, x.ctypes.data, len(x), out.ctypes.data)
    return out[:len(x)]


def splitmix64(seed: int, count: int) -> list[int]:
    out = np.empty(count, dtype=np.uint64)
    _load().dgo_splitmix(seed & ((1 << 64) - 1), count, out.ctypes.data)
    return [int(v) for v in out]


def location_order(g: Graph, seed: int, threads: int = 256, warp: int = 32) -> np.ndarray:
    """The full order: the prefix, then the permutation without its locations."""
    prefix = order_prefix(g, threads, warp)
    rest = permutation(g.output_numel, seed)
    if prefix:
        rest = rest[~np.isin(rest, np.asarray(prefix, dtype=np.int64))]
    return np.concatenate([np.asarray(prefix, dtype=np.int64), rest])


# ---- MERGE (Sec. 3.2) -------------------------------------------------------------
def merge(a: Graph, b: Graph, trim: bool = True) -> tuple[str, str, int]:
    """Matched inputs and (with trim) the common op prefix trimmed: (text of
    a, text of b, number of prefix ops)."""
    lib = _load()
    k = ctypes.c_int()
    n = lib.dgo_merge(a._h, b._h, 1 if trim else 0, None, 0, ctypes.byref(k))
    if n < 0:
        raise OracleError(lib.dgo_error().decode())
    buf = ctypes.create_string_buffer(n)
    lib.dgo_merge(a._h, b._h, 1 if trim else 0, buf, n, ctypes.byref(k))
    ta, tb = buf.raw[:n].split(b"\0")
    return ta.decode(), tb.decode(), k.value
