"""CPU checks of the C ABI library: it loads, exports every symbol the header
declares, and its host-only calls (parse, build, info, leaf, workspace size)
behave, including every error path that needs no device."""

import ctypes

import numpy as np
import pytest

import oracle
import tiny_graphs
from paper_2609_19611_amd import binding as B
from paper_2609_19611_amd import workloads as W

CAT = tiny_graphs.catalogue()


def test_library_exports_every_header_symbol():
    names = B.header_symbols()
    assert len(names) == 25
    lib = ctypes.CDLL(B.LIB_PATH)
    for n in names:
        assert hasattr(lib, n), n


@pytest.mark.parametrize("name", ["c1", "c2", "c3", "c4", "c5"])
def test_info_of_workloads(name):
    text = W.CONFIGS[name]["text"]()
    g = B.dg_graph_parse(text)
    info = B.dg_graph_info(g)
    og = oracle.Graph(text)
    assert info["output_shape"] == og.output_shape
    assert info["output_numel"] == og.output_numel
    assert info["leaf_total"] == og.leaf_total
    assert info["n_leaves"] == len(og.leaves)
    for i, leaf in enumerate(og.leaves):
        li = B.dg_graph_leaf(g, i)
        assert (li["name"], li["shape"], li["base"], li["numel"]) == (leaf.name, leaf.shape, leaf.base, leaf.numel)
    # Static bounds hold for sampled rows.
    locs = W.config_locations(name)[:: max(1, len(W.config_locations(name)) // 5)][:5]
    off, ids, cnt = og.enumerate(locs, threads=4)
    assert info["max_row_size"] >= int(np.diff(off).max())
    assert info["count_bound"] >= int(cnt.max())
    assert info["lds_bytes"] <= 160 * 1024
    assert info["block_threads"] in (64, 256)
    # No DAG call yet: no DAG program, no DAG kernels.
    assert (info["dag_block_threads"], info["dag_lds_bytes"], info["dag_edge_bound"]) == (0, 0, 0)


def test_build_matches_parse():
    leaves = [("x", [16, 3, 32, 32]), ("W", [16, 3, 3, 3]), ("conv_b", [16]), ("bias", [16, 1, 1])]
    ops = [("t1", "conv", [0, 1, 2], "stride=1,1 pad=1,1 dilation=1,1 groups=1"),
           ("t2", "add", [4, 3], ""), ("t3", "gelu", [5], ""),
           ("y", "max_pool", [6], "kernel=2,2 stride=2,2")]
    gb = B.dg_graph_build(leaves, ops, 7)
    gp = B.dg_graph_parse(W.c2_text())
    assert B.dg_graph_info(gb) == B.dg_graph_info(gp)


@pytest.mark.parametrize("text,code", [
    ("leaf x 2\noutput x 2\n", "DG_E_PARSE"),
    ("dgir 1\nleaf x 2,0\noutput x 2,0\n", "DG_E_SHAPE"),
    ("dgir 1\nleaf x 2\nop y frobnicate x\noutput y 2\n", "DG_E_UNSUPPORTED_OP"),
    ("dgir 1\nleaf x 2,3\nleaf z 4\nop y add x z\noutput y 2,3\n", "DG_E_SHAPE"),
    ("dgir 1\nleaf x 2\nop y relu q\noutput y 2\n", "DG_E_PARSE"),
    ("dgir 1\nleaf x 2\nop y relu x\noutput y 3\n", "DG_E_SHAPE"),
    ("dgir 1\nleaf x 2\nop y relu x\n", "DG_E_PARSE"),
    ("dgir 1\nleaf x 1073741824,1073741824,8\noutput x 1073741824,1073741824,8\n", "DG_E_OVERFLOW"),
    ("dgir 1\nleaf x 2,3\nop y affine_gather x ; shape=2 idx0=o0+,o1\noutput y 2\n", "DG_E_PARSE"),
    ("dgir 1\nleaf x 2,3\nop y affine_gather x ; shape=2 idx0=o0\noutput y 2\n", "DG_E_SHAPE"),
    ("dgir 1\nleaf x 2,3\nop y conv x x\noutput y 2\n", "DG_E_SHAPE"),
])
def test_parse_errors(text, code):
    with pytest.raises(B.DgError) as e:
        B.dg_graph_parse(text)
    assert e.value.name == code
    assert B.dg_last_error()


def test_unrefinable_reshape_is_rejected():
    with pytest.raises(B.DgError) as e:
        B.dg_graph_parse(tiny_graphs.UNREFINABLE_RESHAPE)
    assert e.value.name == "DG_E_UNSUPPORTED_OP" and "refinement" in str(e.value)


@pytest.mark.parametrize("name", sorted(tiny_graphs.MERGED_DIMS))
def test_graphs_with_merged_dims_are_accepted(name):
    """Grouped transposed convolutions and reshapes that merge or split
    dims build; their plans view the coupled dims merged."""
    info = B.dg_graph_info(B.dg_graph_parse(CAT[name][0]))
    assert info["n_instructions"] > 0


def test_static_overflow_rejected():
    # Ten nested layer norms over 65536 elements: the bound passes 2^63.
    ops = []
    prev = "x"
    for i in range(10):
        ops.append((f"n{i}", "layer_norm", [prev], dict(ndims=1)))
        prev = f"n{i}"
    txt = tiny_graphs._g([("x", [1, 65536])], ops, prev, [1, 65536])
    with pytest.raises(B.DgError) as e:
        B.dg_graph_parse(txt)
    assert e.value.name == "DG_E_OVERFLOW"


def test_workspace_size_grows_with_n():
    g = B.dg_graph_parse(W.c1_text())
    a, b, c = (B.dg_workspace_size(g, n) for n in (0, 1000, 1_000_000))
    assert 0 < a <= b <= c
    assert c >= 8 * 1_000_001


def test_header_documents_every_status():
    text = open(B.HEADER).read()
    for code in B.STATUS_NAMES.values():
        assert code in text


def test_ranges_outside_the_output_are_rejected_before_any_work():
    g = B.dg_graph_parse(W.c1_text())  # output [8]
    fake = ctypes.c_void_p(0x1000)  # never dereferenced: the range is checked first
    total = ctypes.c_int64()
    for first, n in ((-1, 2), (7, 2), (9, 0), (0, 9)):
        rc = B._lib.dg_enumerate_range(g.handle, first, n, fake, fake, fake, 16, fake, ctypes.byref(total), None)
        assert B.STATUS_NAMES[rc] == "DG_E_RANGE", (first, n)
        rc = B._lib.dg_compare_range(g.handle, g.handle, first, n, 0, fake, fake, ctypes.byref(total), fake, None)
        assert B.STATUS_NAMES[rc] == "DG_E_RANGE", (first, n)
    rc = B._lib.dg_compare_range(g.handle, g.handle, 0, 4, -1, fake, fake, ctypes.byref(total), fake, None)
    assert B.STATUS_NAMES[rc] == "DG_E_INVALID_ARG"


def test_graphs_with_64_bit_ids_parse_and_32_bit_calls_refuse_them():
    """2^32 leaf elements: the graph builds; the 32-bit enumeration calls
    report DG_E_OVERFLOW before any device work, the 64-bit call exists."""
    g = B.dg_graph_parse("dgir 1\nleaf x 65536,65536\nop y relu x\noutput y 65536,65536\n")
    assert B.dg_graph_info(g)["leaf_total"] == 1 << 32
    fake = ctypes.c_void_p(0x1000)  # never dereferenced
    total = ctypes.c_int64()
    rc = B._lib.dg_enumerate(g.handle, fake, 1, fake, fake, fake, 16, fake, ctypes.byref(total), None)
    assert B.STATUS_NAMES[rc] == "DG_E_OVERFLOW"
    rc = B._lib.dg_enumerate_range(g.handle, 0, 1, fake, fake, fake, 16, fake, ctypes.byref(total), None)
    assert B.STATUS_NAMES[rc] == "DG_E_OVERFLOW"
    assert "64 bits" in B.dg_last_error()


@pytest.mark.parametrize("name", sorted(tiny_graphs.catalogue()))
def test_static_bounds_hold_everywhere(name):
    """count_bound and max_row_size bound the oracle's rows at every output
    location of the small graphs (the 32-bit kernels skip their run-time
    overflow checks when count_bound fits 32 bits, so it must be sound)."""
    text = tiny_graphs.catalogue()[name][0]
    info = B.dg_graph_info(B.dg_graph_parse(text))
    og = oracle.Graph(text)
    off, ids, cnt = og.enumerate(range(og.output_numel), threads=4, wide=True)
    assert info["max_row_size"] >= int(np.diff(off).max())
    assert info["count_bound"] >= int(cnt.max())


def test_static_bound_of_nested_norms_is_tight():
    """Three nested layer norms over 4096 elements: the exact largest count
    is about 1.15e18; the bound stays below 2^63, so the graph is accepted."""
    info = B.dg_graph_info(B.dg_graph_parse(tiny_graphs.nested_layer_norms(4096)))
    exact = max(tiny_graphs.nested_layer_norm_counts(4096, 0))
    assert exact <= info["count_bound"] <= 1.01 * exact


@pytest.mark.parametrize("name", ["c1", "c3", "c4", "c5"])
def test_tensor_ids_match_the_oracle(name):
    """Element ids of every tensor (leaves keep their base; op outputs follow
    in SSA order), as the expression DAGs name them."""
    text = W.CONFIGS[name]["text"]()
    g = B.dg_graph_parse(text)
    og = oracle.Graph(text)
    info = B.dg_graph_info(g)
    assert info["n_tensors"] == len(og.tensors)
    for t in range(info["n_tensors"]):
        ti = B.dg_graph_tensor(g, t)
        assert ti["name"] == og.tensors[t].name and ti["shape"] == og.tensors[t].shape
        assert ti["gid"] == og.gid(t)
        assert (ti["leaf"] >= 0) == (og.tensors[t].leaf_index >= 0)


@pytest.mark.parametrize("text", tiny_graphs.OVERFLOWING_SHAPES)
def test_element_counts_past_2_62_are_rejected(text):
    """A leaf or an op result with more than 2^62 elements (including
    products that wrap 64 bits) is DG_E_OVERFLOW, not a wrapped count."""
    with pytest.raises(B.DgError) as e:
        B.dg_graph_parse(text)
    assert e.value.name == "DG_E_OVERFLOW"


def test_calls_over_2_31_locations_are_rejected_before_any_work():
    """A call takes at most 2^31 locations; more is DG_E_INVALID_ARG, checked
    before any device work (no device is needed here)."""
    g = B.dg_graph_parse("dgir 1\nleaf x 65536,65536\nop y relu x\noutput y 65536,65536\n")  # 2^32 outputs
    fake = ctypes.c_void_p(0x1000)  # never dereferenced
    total = ctypes.c_int64()
    n = (1 << 31) + 1
    calls = [
        lambda: B._lib.dg_enumerate_sizes(g.handle, fake, n, fake, fake, ctypes.byref(total), None),
        lambda: B._lib.dg_enumerate_fill(g.handle, fake, n, fake, fake, fake, fake, None),
        lambda: B._lib.dg_enumerate(g.handle, fake, n, fake, fake, fake, 16, fake, ctypes.byref(total), None),
        lambda: B._lib.dg_enumerate_range(g.handle, 0, n, fake, fake, fake, 16, fake, ctypes.byref(total), None),
        lambda: B._lib.dg_compare(g.handle, g.handle, fake, n, fake, fake, ctypes.byref(total), fake, None),
        lambda: B._lib.dg_compare_range(g.handle, g.handle, 0, n, 0, fake, fake, ctypes.byref(total), fake, None),
    ]
    for call in calls:
        assert B.STATUS_NAMES[call()] == "DG_E_INVALID_ARG"


def test_one_call_dag_rejects_bad_arguments_before_any_work():
    """dg_dag checks its arguments before any device work (no device is
    needed here): too many locations, negative capacities, missing output
    buffers for a non-zero capacity, missing totals, and no workspace."""
    g = B.dg_graph_parse(W.CONFIGS["c1"]["text"]())
    fake = ctypes.c_void_p(0x1000)  # never dereferenced
    nn, ne = ctypes.c_int64(), ctypes.c_int64()

    def call(n=4, ncap=8, ecap=8, nodes=fake, edges=fake, ws=fake, tot=True):
        return B.STATUS_NAMES[B._lib.dg_dag(g.handle, fake, n, fake, fake, nodes, nodes, edges, edges, ncap, ecap, ws,
                                            ctypes.byref(nn) if tot else None, ctypes.byref(ne), None)]
    assert call(n=(1 << 31) + 1) == "DG_E_INVALID_ARG"
    assert call(n=-1) == "DG_E_INVALID_ARG"
    assert call(ncap=-1) == "DG_E_INVALID_ARG"
    assert call(ecap=-1) == "DG_E_INVALID_ARG"
    assert call(nodes=None) == "DG_E_INVALID_ARG"
    assert call(edges=None) == "DG_E_INVALID_ARG"
    assert call(tot=False) == "DG_E_INVALID_ARG"
    assert call(ws=None) == "DG_E_WORKSPACE"


def test_count_bound_is_an_exact_integer():
    """The static path-count bound is reported as an integer: above 2^53,
    where a double would round, it is still a sound bound of the exact
    counts (three nested layer norms over 4,096 elements)."""
    text = tiny_graphs.nested_layer_norms(4096)
    info = B.dg_graph_info(B.dg_graph_parse(text))
    assert isinstance(info["count_bound"], int) and info["count_bound"] > 2 ** 53
    exact = max(tiny_graphs.nested_layer_norm_counts(4096, 0))
    assert exact <= info["count_bound"] < 2 ** 63
