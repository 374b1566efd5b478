"""Wrapper of the host-emulation test library (one-thread blocks on the CPU
running the library's compiled plans and block code)."""

import ctypes
import os

import numpy as np

LIB = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "paper_2609_19611_amd", "lib",
                   "libdirigo_hostemu.so")
_lib = None


class HostEmuError(RuntimeError):
    def __init__(self, code, msg):
        super().__init__(f"{code}: {msg}")
        self.code = code


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB):
            from paper_2609_19611_amd import build
            build.build_hostemu()
        _lib = ctypes.CDLL(LIB)
        _lib.dgh_error.restype = ctypes.c_char_p
        P, i64 = ctypes.c_void_p, ctypes.c_int64
        _lib.dgh_sizes.argtypes = [ctypes.c_char_p, i64, P, i64, P]
        _lib.dgh_fill.argtypes = [ctypes.c_char_p, i64, P, i64, P, P, P]
        _lib.dgh_compare.argtypes = [ctypes.c_char_p, i64, ctypes.c_char_p, i64, P, i64, P]
        _lib.dgh_jit_source.argtypes = [ctypes.c_char_p, i64, ctypes.c_int, ctypes.c_char_p, i64]
        _lib.dgh_jit_wide_source.argtypes = [ctypes.c_char_p, i64, ctypes.c_int, ctypes.c_char_p, i64]
        _lib.dgh_jit_dag_source.argtypes = [ctypes.c_char_p, i64, ctypes.c_int, ctypes.c_char_p, i64]
        _lib.dgh_dag_bounds.argtypes = [ctypes.c_char_p, i64, ctypes.c_int, P]
        _lib.dgh_jit_compare_source.argtypes = [ctypes.c_char_p, i64, ctypes.c_char_p, i64, ctypes.c_int,
                                                ctypes.c_char_p, i64]
        _lib.dgh_jit_options.argtypes = [ctypes.c_char_p, i64]
        _lib.dgh_dag_sizes.argtypes = [ctypes.c_char_p, i64, P, i64, P, P]
        _lib.dgh_dag_fill.argtypes = [ctypes.c_char_p, i64, P, i64, P, P, P, P, P, P]
        _lib.dgh_dag_groups.argtypes = [ctypes.c_char_p, i64, P, i64]
        _lib.dgh_box_unique.argtypes = [ctypes.c_int, P, P, ctypes.c_uint32, ctypes.c_uint32]
        _lib.dgh_box_unique.restype = i64
    return _lib


def box_unique(shape, cand, ws_words):
    """The DAG frontier dedup through the bounding-box bitmap: (sorted unique
    candidates, True), or (None, False) when the bitmap does not apply."""
    L = lib()
    shp = np.ascontiguousarray(np.asarray(shape, dtype=np.int64))
    c = np.ascontiguousarray(np.asarray(cand, dtype=np.uint32)).copy()
    k = L.dgh_box_unique(len(shape), shp.ctypes.data, c.ctypes.data, len(c), ws_words)
    return (c[:k].copy(), True) if k >= 0 else (None, False)


def enumerate(text, locs):
    L = lib()
    t = text.encode()
    locs = np.ascontiguousarray(np.asarray(locs, dtype=np.int64))
    off = np.zeros(len(locs) + 1, dtype=np.int64)
    rc = L.dgh_sizes(t, len(t), locs.ctypes.data, len(locs), off.ctypes.data)
    if rc:
        raise HostEmuError(rc, L.dgh_error().decode())
    ids = np.zeros(max(1, off[-1]), dtype=np.uint32)
    cnt = np.zeros(max(1, off[-1]), dtype=np.uint32)
    rc = L.dgh_fill(t, len(t), locs.ctypes.data, len(locs), off.ctypes.data, ids.ctypes.data, cnt.ctypes.data)
    if rc:
        raise HostEmuError(rc, L.dgh_error().decode())
    return off, ids[: off[-1]], cnt[: off[-1]]


def dag(text, locs):
    """Expression DAGs from the library's block code on one host thread, in
    the layout of oracle.Graph.dag (ids as uint64 for comparison)."""
    L = lib()
    t = text.encode()
    locs = np.ascontiguousarray(np.asarray(locs, dtype=np.int64))
    noff = np.zeros(len(locs) + 1, dtype=np.int64)
    eoff = np.zeros(len(locs) + 1, dtype=np.int64)
    rc = L.dgh_dag_sizes(t, len(t), locs.ctypes.data, len(locs), noff.ctypes.data, eoff.ctypes.data)
    if rc:
        raise HostEmuError(rc, L.dgh_error().decode())
    nodes = np.zeros(max(1, noff[-1]), dtype=np.uint32)
    node_edge = np.zeros(max(1, noff[-1]), dtype=np.uint32)
    edges = np.zeros(max(1, eoff[-1]), dtype=np.uint32)
    mults = np.zeros(max(1, eoff[-1]), dtype=np.uint32)
    rc = L.dgh_dag_fill(t, len(t), locs.ctypes.data, len(locs), noff.ctypes.data, eoff.ctypes.data,
                        nodes.ctypes.data, node_edge.ctypes.data, edges.ctypes.data, mults.ctypes.data)
    if rc:
        raise HostEmuError(rc, L.dgh_error().decode())
    return {"node_offsets": noff, "edge_offsets": eoff, "nodes": nodes[: noff[-1]].astype(np.uint64),
            "node_edge": node_edge[: noff[-1]].astype(np.uint64), "edges": edges[: eoff[-1]].astype(np.uint64),
            "mults": mults[: eoff[-1]].astype(np.uint64)}


def dag_groups(text):
    """How the DAG program takes each read group, as (op index, pointwise op,
    per-variable group, list variables) rows."""
    L = lib()
    t = text.encode()
    out = np.zeros((256, 4), dtype=np.int32)
    k = L.dgh_dag_groups(t, len(t), out.ctypes.data, 256)
    if k < 0:
        raise HostEmuError(k, L.dgh_error().decode())
    return [tuple(int(v) for v in r) for r in out[:k]]


def dag_bounds(text, block=64):
    """Static bounds of one location's DAG: (nodes, edges, largest frontier,
    LDS bytes)."""
    out = np.zeros(4, dtype=np.int64)
    t = text.encode()
    rc = lib().dgh_dag_bounds(t, len(t), block, out.ctypes.data)
    if rc:
        raise HostEmuError(rc, lib().dgh_error().decode())
    return tuple(int(v) for v in out)


def compare(text_a, text_b, locs):
    L = lib()
    a, b = text_a.encode(), text_b.encode()
    locs = np.ascontiguousarray(np.asarray(locs, dtype=np.int64))
    st = np.zeros(max(1, len(locs)), dtype=np.uint8)
    rc = L.dgh_compare(a, len(a), b, len(b), locs.ctypes.data, len(locs), st.ctypes.data)
    if rc:
        raise HostEmuError(rc, L.dgh_error().decode())
    return st[: len(locs)]
