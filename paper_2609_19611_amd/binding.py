"""ctypes binding of libdirigo_rocm.so.

The functions named ``dg_*`` take the C ABI's arguments (device buffers as
torch tensors, streams as torch streams) and only marshal them; every step
of the enumeration runs in the library's HIP kernels.  ``enumerate_locations``
and ``compare_locations`` are conveniences that allocate the outputs with torch and call
the ``dg_*`` functions in order.

Importing this module fails loudly if the library has not been built.
"""

from __future__ import annotations

import ctypes
import os
import re

import torch

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "lib", "libdirigo_rocm.so")
HEADER = os.path.join(os.path.dirname(HERE), "include", "dirigo_rocm.h")

DG_OK = 0
STATUS_NAMES = {
    -1: "DG_E_INVALID_ARG", -2: "DG_E_PARSE", -3: "DG_E_SHAPE", -4: "DG_E_UNSUPPORTED_OP", -5: "DG_E_RANGE",
    -6: "DG_E_OVERFLOW", -7: "DG_E_SIGNATURE", -8: "DG_E_WORKSPACE", -9: "DG_E_HIP", -10: "DG_E_CAPACITY",
    -11: "DG_E_BUFFER", -12: "DG_E_STOPPED",
}
MAX_RANK = 8


class DgError(RuntimeError):
    def __init__(self, code: int, message: str):
        super().__init__(f"{STATUS_NAMES.get(code, code)}: {message}")
        self.code = code
        self.name = STATUS_NAMES.get(code, str(code))


class GraphInfo(ctypes.Structure):
    _fields_ = [
        ("n_leaves", ctypes.c_int32),
        ("output_rank", ctypes.c_int32),
        ("output_shape", ctypes.c_int64 * MAX_RANK),
        ("output_numel", ctypes.c_int64),
        ("leaf_total", ctypes.c_uint64),
        ("max_row_size", ctypes.c_int64),
        ("count_bound", ctypes.c_uint64),
        ("n_instructions", ctypes.c_int32),
        ("lds_bytes", ctypes.c_int32),
        ("lds_wide_bytes", ctypes.c_int32),
        ("block_threads", ctypes.c_int32),
        ("max_leaf_terms", ctypes.c_int32),
        ("n_tensors", ctypes.c_int32),
        ("specialized", ctypes.c_int32),
        ("dag_specialized", ctypes.c_int32),
        ("dag_block_threads", ctypes.c_int32),
        ("dag_lds_bytes", ctypes.c_int32),
        ("dag_edge_bound", ctypes.c_int64),
    ]


class LeafInfo(ctypes.Structure):
    _fields_ = [
        ("name", ctypes.c_char * 64),
        ("rank", ctypes.c_int32),
        ("shape", ctypes.c_int64 * MAX_RANK),
        ("base", ctypes.c_uint64),
        ("numel", ctypes.c_int64),
    ]


class TensorInfo(ctypes.Structure):
    _fields_ = [
        ("name", ctypes.c_char * 64),
        ("rank", ctypes.c_int32),
        ("shape", ctypes.c_int64 * MAX_RANK),
        ("numel", ctypes.c_int64),
        ("gid", ctypes.c_uint64),
        ("leaf", ctypes.c_int32),
        ("producer", ctypes.c_int32),
        ("kind", ctypes.c_char * 32),
    ]


class TensorDesc(ctypes.Structure):
    _fields_ = [("name", ctypes.c_char_p), ("rank", ctypes.c_int32), ("shape", ctypes.POINTER(ctypes.c_int64))]


class OpDesc(ctypes.Structure):
    _fields_ = [("name", ctypes.c_char_p), ("kind", ctypes.c_char_p), ("n_inputs", ctypes.c_int32),
                ("inputs", ctypes.POINTER(ctypes.c_int32)), ("attrs", ctypes.c_char_p)]


# dg_chunk_fn(user, first, n, d_offsets, d_ids, d_counts, total, stream)
CHUNK_FN = ctypes.CFUNCTYPE(ctypes.c_int32, ctypes.c_void_p, ctypes.c_int64, ctypes.c_int64, ctypes.c_void_p,
                            ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p)


def _load():
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is not built: run `python -m paper_2609_19611_amd.build` "
                           "(or __graft_entry__.build()) first")
    lib = ctypes.CDLL(LIB_PATH)
    P, i32, i64, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t
    sig = {
        "dg_graph_parse": ([ctypes.c_char_p, sz, ctypes.POINTER(P)], i32),
        "dg_graph_build": ([P, i32, P, i32, i32, ctypes.POINTER(P)], i32),
        "dg_graph_destroy": ([P], None),
        "dg_graph_info": ([P, ctypes.POINTER(GraphInfo)], i32),
        "dg_graph_leaf": ([P, i32, ctypes.POINTER(LeafInfo)], i32),
        "dg_workspace_size": ([P, i64, ctypes.POINTER(sz)], i32),
        "dg_enumerate_sizes": ([P, P, i64, P, P, ctypes.POINTER(i64), P], i32),
        "dg_enumerate_fill": ([P, P, i64, P, P, P, P, P], i32),
        "dg_enumerate": ([P, P, i64, P, P, P, i64, P, ctypes.POINTER(i64), P], i32),
        "dg_compare": ([P, P, P, i64, P, P, ctypes.POINTER(i64), P, P], i32),
        "dg_enumerate_range": ([P, i64, i64, P, P, P, i64, P, ctypes.POINTER(i64), P], i32),
        "dg_compare_range": ([P, P, i64, i64, i64, P, P, ctypes.POINTER(i64), P, P], i32),
        "dg_enumerate_stream": ([P, i64, i64, P, sz, i64, CHUNK_FN, P, P, P], i32),
        "dg_enumerate_wide": ([P, P, i64, P, P, P, i64, P, ctypes.POINTER(i64), P], i32),
        "dg_enumerate_noalloc": ([P, P, i64, P, P, P, i64, ctypes.POINTER(i64), P], i32),
        "dg_graph_tensor": ([P, i32, P], i32),
        "dg_dag_sizes": ([P, P, i64, P, P, P, ctypes.POINTER(i64), ctypes.POINTER(i64), P], i32),
        "dg_dag_fill": ([P, P, i64, P, P, P, P, P, P, P, P], i32),
        "dg_dag": ([P, P, i64, P, P, P, P, P, P, i64, i64, P, ctypes.POINTER(i64), ctypes.POINTER(i64), P], i32),
        "dg_order_prefix": ([P, i32, i32, P, i64, ctypes.POINTER(i64)], i32),
        "dg_graph_text": ([P, ctypes.c_char_p, sz, ctypes.POINTER(sz)], i32),
        "dg_graph_merge": ([P, P, i32, ctypes.POINTER(P), ctypes.POINTER(P), ctypes.POINTER(i32)], i32),
        "dg_order_workspace_size": ([i64, ctypes.POINTER(sz)], i32),
        "dg_order_permute": ([i64, ctypes.c_uint64, P, i64, i64, i64, P, ctypes.POINTER(i64), P, sz, P], i32),
        "dg_last_error": ([], ctypes.c_char_p),
    }
    for name, (args, res) in sig.items():
        fn = getattr(lib, name)
        fn.argtypes = args
        fn.restype = res
    return lib


_lib = _load()


def _check(rc: int) -> None:
    if rc != DG_OK:
        raise DgError(rc, _lib.dg_last_error().decode())


def header_symbols() -> list[str]:
    """Names of the functions include/dirigo_rocm.h declares."""
    text = open(HEADER).read()
    return sorted(set(re.findall(r"^\s*(?:dg_status|void|const char\*)\s+(dg_\w+)\s*\(", text, re.M)))


def _ptr(t: torch.Tensor | None) -> int | None:
    return None if t is None else t.data_ptr()


def _stream(stream) -> int | None:
    if stream is None:
        stream = torch.cuda.current_stream()
    return stream.cuda_stream


class Graph:
    """An owned dg_graph handle."""

    def __init__(self, handle):
        self._h = handle

    def __del__(self):
        h = getattr(self, "_h", None)
        # (At interpreter exit the module's globals may already be gone.)
        if h and _lib is not None:
            _lib.dg_graph_destroy(h)
            self._h = None

    @property
    def handle(self):
        return self._h


def dg_graph_parse(text: str) -> Graph:
    data = text.encode()
    h = ctypes.c_void_p()
    _check(_lib.dg_graph_parse(data, len(data), ctypes.byref(h)))
    return Graph(h)


def dg_graph_build(leaves, ops, output: int) -> Graph:
    """leaves: [(name, shape)]; ops: [(name, kind, [input indices], attrs)]."""
    keep = []
    td = (TensorDesc * len(leaves))()
    for i, (name, shape) in enumerate(leaves):
        arr = (ctypes.c_int64 * len(shape))(*shape)
        keep.append(arr)
        td[i] = TensorDesc(name.encode(), len(shape), arr)
    od = (OpDesc * max(1, len(ops)))()
    for i, (name, kind, ins, attrs) in enumerate(ops):
        arr = (ctypes.c_int32 * max(1, len(ins)))(*ins)
        keep.append(arr)
        od[i] = OpDesc(name.encode(), kind.encode(), len(ins), arr, (attrs or "").encode())
    h = ctypes.c_void_p()
    _check(_lib.dg_graph_build(td, len(leaves), od, len(ops), output, ctypes.byref(h)))
    return Graph(h)


def dg_graph_info(g: Graph) -> dict:
    info = GraphInfo()
    _check(_lib.dg_graph_info(g.handle, ctypes.byref(info)))
    return {
        "n_leaves": info.n_leaves,
        "output_shape": tuple(info.output_shape[: info.output_rank]),
        "output_numel": info.output_numel,
        "leaf_total": info.leaf_total,
        "max_row_size": info.max_row_size,
        "count_bound": info.count_bound,
        "n_instructions": info.n_instructions,
        "lds_bytes": info.lds_bytes,
        "lds_wide_bytes": info.lds_wide_bytes,
        "block_threads": info.block_threads,
        "max_leaf_terms": info.max_leaf_terms,
        "n_tensors": info.n_tensors,
        "specialized": info.specialized,
        "dag_specialized": info.dag_specialized,
        "dag_block_threads": info.dag_block_threads,
        "dag_lds_bytes": info.dag_lds_bytes,
        "dag_edge_bound": info.dag_edge_bound,
    }


def dg_graph_leaf(g: Graph, i: int) -> dict:
    li = LeafInfo()
    _check(_lib.dg_graph_leaf(g.handle, i, ctypes.byref(li)))
    return {"name": li.name.decode(), "shape": tuple(li.shape[: li.rank]), "base": li.base, "numel": li.numel}


def dg_graph_tensor(g: Graph, i: int) -> dict:
    ti = TensorInfo()
    _check(_lib.dg_graph_tensor(g.handle, i, ctypes.byref(ti)))
    return {"name": ti.name.decode(), "shape": tuple(ti.shape[: ti.rank]), "numel": ti.numel, "gid": ti.gid,
            "leaf": ti.leaf, "producer": ti.producer, "kind": ti.kind.decode()}


def dg_workspace_size(g: Graph, n_locs: int) -> int:
    b = ctypes.c_size_t()
    _check(_lib.dg_workspace_size(g.handle, n_locs, ctypes.byref(b)))
    return b.value


def _dev_i64(t: torch.Tensor, what: str) -> None:
    if not t.is_cuda or t.dtype != torch.int64 or not t.is_contiguous():
        raise ValueError(f"{what} must be a contiguous int64 device tensor")


def dg_enumerate_sizes(g: Graph, d_locs: torch.Tensor, d_offsets: torch.Tensor, d_ws: torch.Tensor,
                       stream=None) -> int:
    n = d_locs.numel()
    _dev_i64(d_locs, "locations")
    _dev_i64(d_offsets, "offsets")
    if d_offsets.numel() < n + 1:
        raise ValueError("offsets needs n + 1 entries")
    total = ctypes.c_int64()
    _check(_lib.dg_enumerate_sizes(g.handle, _ptr(d_locs), n, _ptr(d_offsets), _ptr(d_ws), ctypes.byref(total),
                                   _stream(stream)))
    return total.value


def dg_enumerate_fill(g: Graph, d_locs: torch.Tensor, d_offsets: torch.Tensor, d_ids: torch.Tensor,
                      d_counts: torch.Tensor, d_ws: torch.Tensor, stream=None) -> None:
    n = d_locs.numel()
    for t, what in ((d_ids, "ids"), (d_counts, "counts")):
        if not t.is_cuda or t.dtype not in (torch.int32, torch.uint32) or not t.is_contiguous():
            raise ValueError(f"{what} must be a contiguous 32-bit device tensor")
    _check(_lib.dg_enumerate_fill(g.handle, _ptr(d_locs), n, _ptr(d_offsets), _ptr(d_ids), _ptr(d_counts),
                                  _ptr(d_ws), _stream(stream)))


def dg_enumerate(g: Graph, d_locs: torch.Tensor, d_offsets: torch.Tensor, d_ids: torch.Tensor,
                 d_counts: torch.Tensor, d_ws: torch.Tensor, stream=None) -> int:
    """Single pass: offsets and rows; capacity is the size of d_ids/d_counts.
    Returns the total; raises DgError(DG_E_BUFFER) if the rows do not fit
    (the offsets are then valid)."""
    n = d_locs.numel()
    _dev_i64(d_locs, "locations")
    _dev_i64(d_offsets, "offsets")
    if d_offsets.numel() < n + 1:
        raise ValueError("offsets needs n + 1 entries")
    cap = min(d_ids.numel(), d_counts.numel())
    for t, what in ((d_ids, "ids"), (d_counts, "counts")):
        if not t.is_cuda or t.dtype not in (torch.int32, torch.uint32) or not t.is_contiguous():
            raise ValueError(f"{what} must be a contiguous 32-bit device tensor")
    total = ctypes.c_int64()
    _check(_lib.dg_enumerate(g.handle, _ptr(d_locs), n, _ptr(d_offsets), _ptr(d_ids), _ptr(d_counts), cap,
                             _ptr(d_ws), ctypes.byref(total), _stream(stream)))
    return total.value


NOALLOC_MAX_LOCATIONS = 2097152


def dg_enumerate_noalloc(g: Graph, d_locs: torch.Tensor, d_offsets: torch.Tensor, d_ids: torch.Tensor,
                         d_counts: torch.Tensor, stream=None) -> int:
    """dg_enumerate with the library's own device scratch instead of a
    workspace (no allocation; the graph must be resident on the device from
    an earlier enumeration call).  Returns the total."""
    n = d_locs.numel()
    _dev_i64(d_locs, "locations")
    _dev_i64(d_offsets, "offsets")
    if d_offsets.numel() < n + 1:
        raise ValueError("offsets needs n + 1 entries")
    cap = min(d_ids.numel(), d_counts.numel())
    for t, what in ((d_ids, "ids"), (d_counts, "counts")):
        if not t.is_cuda or t.dtype not in (torch.int32, torch.uint32) or not t.is_contiguous():
            raise ValueError(f"{what} must be a contiguous 32-bit device tensor")
    total = ctypes.c_int64()
    _check(_lib.dg_enumerate_noalloc(g.handle, _ptr(d_locs), n, _ptr(d_offsets), _ptr(d_ids), _ptr(d_counts), cap,
                                     ctypes.byref(total), _stream(stream)))
    return total.value


def dg_compare(a: Graph, b: Graph, d_locs: torch.Tensor, d_status: torch.Tensor, d_mismatch: torch.Tensor,
               d_ws: torch.Tensor, stream=None) -> int:
    n = d_locs.numel()
    _dev_i64(d_locs, "locations")
    if d_status.dtype != torch.uint8 or d_status.numel() < n:
        raise ValueError("status must be a uint8 device tensor of n entries")
    _dev_i64(d_mismatch, "mismatch")
    nm = ctypes.c_int64()
    _check(_lib.dg_compare(a.handle, b.handle, _ptr(d_locs), n, _ptr(d_status), _ptr(d_mismatch),
                           ctypes.byref(nm), _ptr(d_ws), _stream(stream)))
    return nm.value


def dg_enumerate_wide(g: Graph, d_locs: torch.Tensor, d_offsets: torch.Tensor, d_ids: torch.Tensor,
                      d_counts: torch.Tensor, d_ws: torch.Tensor, stream=None) -> int:
    """dg_enumerate with 64-bit ids and counts (int64 or uint64 device
    tensors; int64 ones hold the uint64 values' bits).  Returns the total;
    raises DgError(DG_E_BUFFER) if the rows do not fit (the offsets are then
    valid)."""
    n = d_locs.numel()
    _dev_i64(d_locs, "locations")
    _dev_i64(d_offsets, "offsets")
    if d_offsets.numel() < n + 1:
        raise ValueError("offsets needs n + 1 entries")
    for t, what in ((d_ids, "ids"), (d_counts, "counts")):
        if not t.is_cuda or t.dtype not in (torch.int64, torch.uint64) or not t.is_contiguous():
            raise ValueError(f"{what} must be a contiguous 64-bit device tensor")
    cap = min(d_ids.numel(), d_counts.numel())
    total = ctypes.c_int64()
    _check(_lib.dg_enumerate_wide(g.handle, _ptr(d_locs), n, _ptr(d_offsets), _ptr(d_ids), _ptr(d_counts), cap,
                                  _ptr(d_ws), ctypes.byref(total), _stream(stream)))
    return total.value


def dg_enumerate_range(g: Graph, first: int, n: int, d_offsets: torch.Tensor, d_ids: torch.Tensor,
                       d_counts: torch.Tensor, d_ws: torch.Tensor, stream=None) -> int:
    """Single pass over the flat locations first .. first + n - 1."""
    _dev_i64(d_offsets, "offsets")
    if d_offsets.numel() < n + 1:
        raise ValueError("offsets needs n + 1 entries")
    cap = min(d_ids.numel(), d_counts.numel())
    for t, what in ((d_ids, "ids"), (d_counts, "counts")):
        if not t.is_cuda or t.dtype not in (torch.int32, torch.uint32) or not t.is_contiguous():
            raise ValueError(f"{what} must be a contiguous 32-bit device tensor")
    total = ctypes.c_int64()
    _check(_lib.dg_enumerate_range(g.handle, first, n, _ptr(d_offsets), _ptr(d_ids), _ptr(d_counts), cap,
                                   _ptr(d_ws), ctypes.byref(total), _stream(stream)))
    return total.value


def dg_compare_range(a: Graph, b: Graph, first: int, n: int, d_status: torch.Tensor, d_mismatch: torch.Tensor,
                     d_ws: torch.Tensor, max_mismatch: int = 0, stream=None) -> int:
    """Compare over the flat locations first .. first + n - 1; with
    max_mismatch > 0 locations not started once that many mismatches were
    found get status 3.  Returns the number of mismatch positions written."""
    if d_status.dtype != torch.uint8 or d_status.numel() < n or not d_status.is_cuda:
        raise ValueError("status must be a uint8 device tensor of n entries")
    _dev_i64(d_mismatch, "mismatch")
    if d_mismatch.numel() < n:
        raise ValueError("mismatch needs n entries")
    nm = ctypes.c_int64()
    _check(_lib.dg_compare_range(a.handle, b.handle, first, n, max_mismatch, _ptr(d_status), _ptr(d_mismatch),
                                 ctypes.byref(nm), _ptr(d_ws), _stream(stream)))
    return nm.value


class _DeviceArray:
    """A device pointer viewed as a torch tensor (no copy)."""

    def __init__(self, ptr: int, n: int, typestr: str):
        self.__cuda_array_interface__ = {"shape": (n,), "typestr": typestr, "data": (ptr, False), "version": 3}


def device_view(ptr: int, n: int, dtype: torch.dtype) -> torch.Tensor:
    typestr = {torch.int64: "<i8", torch.int32: "<i4", torch.uint8: "|u1"}[dtype]
    if n == 0:
        return torch.empty(0, dtype=dtype, device="cuda")
    return torch.as_tensor(_DeviceArray(ptr, n, typestr), device="cuda")


def dg_enumerate_stream(g: Graph, first: int, n: int, d_buf: torch.Tensor, max_chunk: int, consume,
                        streams=None) -> None:
    """Streams rows of locations first .. first + n - 1 through d_buf.
    consume(first, offsets, ids, counts, stream) gets each chunk as device
    tensors (views into d_buf) right after its work was enqueued on
    `stream`, which is current during the call: work it enqueues there sees
    the finished chunk, and the views stay valid until that work is done.
    A truthy return stops."""
    if not d_buf.is_cuda or not d_buf.is_contiguous():
        raise ValueError("the buffer must be a contiguous device tensor")
    sa, sb = streams if streams is not None else (torch.cuda.Stream(), torch.cuda.Stream())
    by_handle = {int(sa.cuda_stream): sa, int(sb.cuda_stream): sb}
    errors = []

    def trampoline(user, first_, n_, d_off, d_ids, d_cnt, total, stream):
        try:
            off = device_view(d_off, n_ + 1, torch.int64)
            ids = device_view(d_ids, total, torch.int32)
            cnt = device_view(d_cnt, total, torch.int32)
            s = by_handle.get(int(stream or 0))
            with torch.cuda.stream(s):
                return 1 if consume(first_, off, ids, cnt, s) else 0
        except Exception as e:  # reported after the call returns
            errors.append(e)
            return 1

    cb = CHUNK_FN(trampoline)
    rc = _lib.dg_enumerate_stream(g.handle, first, n, _ptr(d_buf), d_buf.numel() * d_buf.element_size(), max_chunk,
                                  cb, None, sa.cuda_stream, sb.cuda_stream)
    if errors:
        raise errors[0]
    _check(rc)


def dg_last_error() -> str:
    return _lib.dg_last_error().decode()


# ---------------------------------------------------------------- helpers --
def workspace(g: Graph, n: int, device=None) -> torch.Tensor:
    return torch.empty(max(1, dg_workspace_size(g, n)), dtype=torch.uint8, device=device or "cuda")


def enumerate_locations(g: Graph, locs, stream=None):
    """(offsets int64[n+1], ids int32[total], counts int32[total]) on the device.
    ids and counts hold uint32 values in int32 storage."""
    d_locs = locs if isinstance(locs, torch.Tensor) else torch.as_tensor(locs, dtype=torch.int64)
    d_locs = d_locs.to(device="cuda", dtype=torch.int64).contiguous()
    n = d_locs.numel()
    ws = workspace(g, n, d_locs.device)
    offsets = torch.empty(n + 1, dtype=torch.int64, device=d_locs.device)
    total = dg_enumerate_sizes(g, d_locs, offsets, ws, stream)
    ids = torch.empty(max(1, total), dtype=torch.int32, device=d_locs.device)
    cnt = torch.empty(max(1, total), dtype=torch.int32, device=d_locs.device)
    dg_enumerate_fill(g, d_locs, offsets, ids, cnt, ws, stream)
    return offsets, ids[:total], cnt[:total]


def _dev_u32(t: torch.Tensor, what: str) -> None:
    if not t.is_cuda or t.dtype not in (torch.int32, torch.uint32) or not t.is_contiguous():
        raise ValueError(f"{what} must be a contiguous 32-bit device tensor")


def dg_dag_sizes(g: Graph, d_locs: torch.Tensor, d_node_offsets: torch.Tensor, d_edge_offsets: torch.Tensor,
                 d_ws: torch.Tensor, stream=None):
    """Expression DAG sizes: fills both offset arrays (n + 1 entries);
    returns (total nodes, total edges)."""
    n = d_locs.numel()
    _dev_i64(d_locs, "locations")
    for t, what in ((d_node_offsets, "node offsets"), (d_edge_offsets, "edge offsets")):
        _dev_i64(t, what)
        if t.numel() < n + 1:
            raise ValueError(f"{what} needs n + 1 entries")
    nn, ne = ctypes.c_int64(), ctypes.c_int64()
    _check(_lib.dg_dag_sizes(g.handle, _ptr(d_locs), n, _ptr(d_node_offsets), _ptr(d_edge_offsets), _ptr(d_ws),
                             ctypes.byref(nn), ctypes.byref(ne), _stream(stream)))
    return nn.value, ne.value


def dg_dag_fill(g: Graph, d_locs: torch.Tensor, d_node_offsets: torch.Tensor, d_edge_offsets: torch.Tensor,
                d_nodes: torch.Tensor, d_node_edge: torch.Tensor, d_edges: torch.Tensor, d_mults: torch.Tensor,
                d_ws: torch.Tensor, stream=None) -> None:
    n = d_locs.numel()
    _dev_i64(d_locs, "locations")
    _dev_i64(d_node_offsets, "node offsets")
    _dev_i64(d_edge_offsets, "edge offsets")
    for t, what in ((d_nodes, "nodes"), (d_node_edge, "node edges"), (d_edges, "edges"), (d_mults, "mults")):
        _dev_u32(t, what)
    _check(_lib.dg_dag_fill(g.handle, _ptr(d_locs), n, _ptr(d_node_offsets), _ptr(d_edge_offsets), _ptr(d_nodes),
                            _ptr(d_node_edge), _ptr(d_edges), _ptr(d_mults), _ptr(d_ws), _stream(stream)))


def dg_dag(g: Graph, d_locs: torch.Tensor, d_node_offsets: torch.Tensor, d_edge_offsets: torch.Tensor,
           d_nodes: torch.Tensor, d_node_edge: torch.Tensor, d_edges: torch.Tensor, d_mults: torch.Tensor,
           d_ws: torch.Tensor, stream=None):
    """Expression DAGs in one call into buffers sized beforehand (their
    lengths are the capacities); returns (total nodes, total edges).
    Raises DgError (DG_E_BUFFER) when a total exceeds its buffer; the
    offsets are then written."""
    n = d_locs.numel()
    _dev_i64(d_locs, "locations")
    for t, what in ((d_node_offsets, "node offsets"), (d_edge_offsets, "edge offsets")):
        _dev_i64(t, what)
        if t.numel() < n + 1:
            raise ValueError(f"{what} needs n + 1 entries")
    for t, what in ((d_nodes, "nodes"), (d_node_edge, "node edges"), (d_edges, "edges"), (d_mults, "mults")):
        _dev_u32(t, what)
    if d_nodes.numel() != d_node_edge.numel() or d_edges.numel() != d_mults.numel():
        raise ValueError("nodes and node edges, and edges and mults, need equal lengths")
    nn, ne = ctypes.c_int64(), ctypes.c_int64()
    _check(_lib.dg_dag(g.handle, _ptr(d_locs), n, _ptr(d_node_offsets), _ptr(d_edge_offsets), _ptr(d_nodes),
                       _ptr(d_node_edge), _ptr(d_edges), _ptr(d_mults), d_nodes.numel(), d_edges.numel(),
                       _ptr(d_ws), ctypes.byref(nn), ctypes.byref(ne), _stream(stream)))
    return nn.value, ne.value


def dag_locations(g: Graph, locs, stream=None) -> dict:
    """Expression DAGs of res(y[l]) for the given locations, on the device:
    node_offsets, edge_offsets (int64[n+1]); nodes, node_edge, edges, mults
    (uint32 values in int32 storage)."""
    d_locs = locs if isinstance(locs, torch.Tensor) else torch.as_tensor(locs, dtype=torch.int64)
    d_locs = d_locs.to(device="cuda", dtype=torch.int64).contiguous()
    n = d_locs.numel()
    ws = workspace(g, n, d_locs.device)
    noff = torch.empty(n + 1, dtype=torch.int64, device=d_locs.device)
    eoff = torch.empty(n + 1, dtype=torch.int64, device=d_locs.device)
    nn, ne = dg_dag_sizes(g, d_locs, noff, eoff, ws, stream)
    out = {"node_offsets": noff, "edge_offsets": eoff}
    for k, m in (("nodes", nn), ("node_edge", nn), ("edges", ne), ("mults", ne)):
        out[k] = torch.empty(max(1, m), dtype=torch.int32, device=d_locs.device)
    dg_dag_fill(g, d_locs, noff, eoff, out["nodes"], out["node_edge"], out["edges"], out["mults"], ws, stream)
    for k, m in (("nodes", nn), ("node_edge", nn), ("edges", ne), ("mults", ne)):
        out[k] = out[k][:m]
    return out


def dg_graph_text(g: Graph) -> str:
    """The graph as dgir v1 text."""
    n = ctypes.c_size_t()
    _check(_lib.dg_graph_text(g.handle, None, 0, ctypes.byref(n)))
    buf = ctypes.create_string_buffer(n.value + 1)
    _check(_lib.dg_graph_text(g.handle, buf, n.value + 1, ctypes.byref(n)))
    return buf.value.decode()


def dg_graph_merge(a: Graph, b: Graph, trim_prefix: bool = True) -> tuple[Graph, Graph, int]:
    """MERGE: the two graphs with matched inputs and (by default) the common
    prefix trimmed, and the number of trimmed ops."""
    ha, hb, k = ctypes.c_void_p(), ctypes.c_void_p(), ctypes.c_int32()
    _check(_lib.dg_graph_merge(a.handle, b.handle, 1 if trim_prefix else 0, ctypes.byref(ha), ctypes.byref(hb),
                               ctypes.byref(k)))
    return Graph(ha.value), Graph(hb.value), k.value


def dg_order_prefix(g: Graph, block_threads: int = 256, warp: int = 32) -> list[int]:
    """The ranked prefix of the location order (corners, then the first and
    last output location); host only."""
    n = ctypes.c_int64()
    _check(_lib.dg_order_prefix(g.handle, block_threads, warp, None, 0, ctypes.byref(n)))
    buf = (ctypes.c_int64 * max(1, n.value))()
    _check(_lib.dg_order_prefix(g.handle, block_threads, warp, buf, n.value, ctypes.byref(n)))
    return list(buf[: n.value])


def dg_order_workspace_size(n_exclude: int) -> int:
    b = ctypes.c_size_t()
    _check(_lib.dg_order_workspace_size(n_exclude, ctypes.byref(b)))
    return b.value


def dg_order_permute(n_out: int, seed: int, exclude, first: int, count: int, d_out: torch.Tensor,
                     d_ws: torch.Tensor, stream=None) -> int:
    """Positions [first, first + count) of the keyed permutation of
    [0, n_out) without the values in `exclude` (host ints), into d_out;
    returns the number written."""
    _dev_i64(d_out, "out")
    ex = list(exclude or [])
    if d_out.numel() < count - len(set(ex)):
        raise ValueError("out needs room for count values less the excluded ones")
    buf = (ctypes.c_int64 * max(1, len(ex)))(*ex)
    w = ctypes.c_int64()
    _check(_lib.dg_order_permute(n_out, seed & ((1 << 64) - 1), buf, len(ex), first, count, _ptr(d_out),
                                 ctypes.byref(w), _ptr(d_ws), d_ws.numel() * d_ws.element_size(), _stream(stream)))
    return w.value


def order_locations(g: Graph, seed: int, block_threads: int = 256, warp: int = 32, device=None) -> torch.Tensor:
    """The full location order of g's output on the device: the prefix, then
    the permutation without the prefix's locations."""
    device = device or torch.device("cuda", torch.cuda.current_device())
    n = dg_graph_info(g)["output_numel"]
    prefix = dg_order_prefix(g, block_threads, warp)
    k = len(prefix)
    out = torch.empty(max(1, n), dtype=torch.int64, device=device)
    if k:
        out[:k] = torch.tensor(prefix, dtype=torch.int64)
    ws = torch.empty(max(1, dg_order_workspace_size(k)), dtype=torch.uint8, device=device)
    w = dg_order_permute(n, seed, prefix, 0, n, out[k:], ws) if n > k else 0
    if k + w != n:
        raise RuntimeError(f"order has {k + w} of {n} locations")
    return out[:n]


def compare_locations(a: Graph, b: Graph, locs, stream=None):
    """(status uint8[n], mismatch positions int64[k]) on the device."""
    d_locs = locs if isinstance(locs, torch.Tensor) else torch.as_tensor(locs, dtype=torch.int64)
    d_locs = d_locs.to(device="cuda", dtype=torch.int64).contiguous()
    n = d_locs.numel()
    ws = torch.empty(max(dg_workspace_size(a, n), dg_workspace_size(b, n), 1), dtype=torch.uint8,
                     device=d_locs.device)
    status = torch.empty(max(1, n), dtype=torch.uint8, device=d_locs.device)
    mism = torch.empty(max(1, n), dtype=torch.int64, device=d_locs.device)
    k = dg_compare(a, b, d_locs, status, mism, ws, stream)
    return status[:n], mism[:k]
