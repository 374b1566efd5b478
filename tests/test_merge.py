"""MERGE (Sec. 3.2): the oracle's input matching and prefix trimming pinned
by the paper's worked example (the two whole programs of the running
example, merged, give the rows and the verdict the paper prints), by
trimming identical programs entirely, and by the one-way implication that
trimming keeps (equal after trimming => equal before); then the library's
merge against the oracle's, and its error paths."""

import json
import os

import numpy as np
import pytest

import oracle
import tiny_graphs
from paper_2609_19611_amd import workloads as W
from paper_2609_19611_amd.workloads import GraphText

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "paper_example.json")


def _rows(g, locs):
    off, ids, cnt = g.enumerate(locs, threads=4)
    return [sorted(zip(ids[off[i]:off[i + 1]].tolist(), cnt[off[i]:off[i + 1]].tolist())) for i in range(len(locs))]


# ---- oracle pins --------------------------------------------------------------------
def test_paper_programs_merge_to_the_worked_example():
    gold = json.load(open(GOLDEN))
    a, b, k = oracle.merge(oracle.Graph(W.paper_program_text(False)), oracle.Graph(W.paper_program_text(True)))
    assert k == 1  # the shared convolution
    ga, gb = oracle.Graph(a), oracle.Graph(b)
    assert [t.name for t in ga.leaves] == ["x", "Wt", "conv_b", "b", "M"] == [t.name for t in gb.leaves]
    assert list(ga.leaves[-1].shape) == gold["M_shape"] and list(ga.output_shape) == gold["Y_shape"]
    loc = gold["location_flat"]
    ra, rb = _rows(ga, [loc])[0], _rows(gb, [loc])[0]
    assert len(ra) == gold["reference_row_size"] and len(rb) == gold["kernel_row_size"]
    assert {c for _, c in ra} == {c for _, c in rb} == {gold["all_counts"]}
    # The row is M[11, :, :, 12] (by the footprint the paper prints) and b[5].
    mbase = ga.leaves[-1].base
    n, c, w = gold["location_multi_index"]
    want = sorted(mbase + ((n * 16 + cc) * 64 + h) * 64 + w for cc in range(16) for h in range(64))
    assert [i for i, _ in ra] == sorted(want + [ga.leaves[3].base + c])
    assert oracle.compare(ga, gb, [loc])[0] == gold["compare_status"]


def test_identical_programs_are_trimmed_entirely():
    text = W.c4_text()
    a, b, k = oracle.merge(oracle.Graph(text), oracle.Graph(text))
    assert k == 6 and a == b
    g = oracle.Graph(a)
    assert [t.name for t in g.leaves][-1] == "y"  # the output became an input
    assert (oracle.compare(g, oracle.Graph(b), range(g.output_numel)) == 0).all()


def _shared_prefix_pair(n=2, c=3, hw=5):
    """Two programs sharing conv -> relu, then different tails (one
    transposes before its reduction, one has an off-by-one window)."""
    def prog(tail):
        g = GraphText()
        g.leaf("x", [n, c, hw, hw])
        g.leaf("w", [4, c, 3, 3])
        g.op("t", "conv", "x", "w", stride=[1, 1], pad=[1, 1], dilation=[1, 1], groups=1)
        g.op("r", "relu", "t")
        tail(g)
        g.output("y", [n, 4, hw])
        return g.text()

    def ta(g):
        g.op("y", "sum", "r", dims=2, keepdim=0)

    def tb(g):
        g.op("y", "affine_gather", "r", shape=[n, 4, hw], window=[hw - 1], idx0=["o0", "o1", "w0", "o2"], mult=[1])
    return prog(ta), prog(tb)


def test_equal_after_trimming_implies_equal_before():
    for a_text, b_text in [_shared_prefix_pair(),
                           (W.paper_program_text(False, N=2, Cin=2, C=3, H=4, W=2),
                            W.paper_program_text(True, N=2, Cin=2, C=3, H=4, W=2, h_limit=4)),
                           (W.paper_program_text(False, N=2, Cin=2, C=3, H=4, W=2),
                            W.paper_program_text(True, N=2, Cin=2, C=3, H=4, W=2, h_limit=2))]:
        A, Bg = oracle.Graph(a_text), oracle.Graph(b_text)
        ta, tb, k = oracle.merge(A, Bg)
        assert k >= 1
        locs = list(range(A.output_numel))
        after = oracle.compare(oracle.Graph(ta), oracle.Graph(tb), locs)
        # The untrimmed obligation: b over a's inputs, no op trimmed (by
        # hand, and by the merge without trimming).
        ua, ub = _untrimmed(a_text, b_text)
        ma, mb, k0 = oracle.merge(A, Bg, trim=False)
        assert k0 == 0 and _canonical(ma) == _canonical(ua) and _canonical(mb) == _canonical(ub)
        before = oracle.compare(oracle.Graph(ua), oracle.Graph(ub), locs)
        assert ((after != 0) | (before == 0)).all()


def _untrimmed(a_text, b_text):
    """b rewritten over a's inputs (same names and order) with no op trimmed,
    by hand: the kernel programs of these tests declare the same inputs."""
    A = oracle.Graph(a_text)
    names = [t.name for t in A.leaves]
    lines = b_text.strip().split("\n")
    leaf_lines = [l for l in lines if l.startswith("leaf ")]
    rest = [l for l in lines[1:] if not l.startswith("leaf ")]
    # Pair b's leaves with a's by shape in declaration order.
    a_shapes = [(t.name, ",".join(map(str, t.shape))) for t in A.leaves]
    ren, free = {}, list(a_shapes)
    for l in leaf_lines:
        _, nm, shape = l.split()
        j = next(i for i, (_, s) in enumerate(free) if s == shape)
        ren[nm] = free.pop(j)[0]
    def fix(line):
        return " ".join(ren.get(w, w) for w in line.split())
    head = ["dgir 1"] + [f"leaf {n} {s}" for n, s in a_shapes]
    return a_text, "\n".join(head + [fix(l) for l in rest]) + "\n"


def test_inputs_matched_by_name_then_by_shape():
    a_text = W.c4_text()
    lines = a_text.strip().split("\n")
    leaves = [l for l in lines if l.startswith("leaf ")]
    other = [l for l in lines[1:] if not l.startswith("leaf ")]
    # Reversed declaration order, x renamed: gamma/beta/bias keep their names
    # (matched by name), x_in pairs with x by shape.
    b_text = "\n".join(["dgir 1"] + leaves[::-1] + other).replace(" x ", " x_in ").replace("leaf x ", "leaf x_in ")
    b_text = b_text.replace("matmul x W", "matmul x_in W").replace("slice x ;", "slice x_in ;") + "\n"
    with pytest.raises(oracle.OracleError):
        oracle.compare(oracle.Graph(a_text), oracle.Graph(b_text), [0])
    a, b, k = oracle.merge(oracle.Graph(a_text), oracle.Graph(b_text))
    assert k == 6 and a == b


def test_unmatched_inputs_are_errors():
    g = GraphText()
    g.leaf("x", [3, 4])
    g.op("y", "relu", "x")
    g.output("y", [3, 4])
    h = GraphText()
    h.leaf("x", [4, 3])
    h.op("t", "permute", "x", dims=[1, 0])
    h.op("y", "relu", "t")
    h.output("y", [3, 4])
    with pytest.raises(oracle.OracleError):
        oracle.merge(oracle.Graph(g.text()), oracle.Graph(h.text()))


# ---- library against the oracle ----------------------------------------------------------
def _pairs():
    small_a = W.paper_program_text(False, N=2, Cin=2, C=3, H=4, W=2)
    small_b = W.paper_program_text(True, N=2, Cin=2, C=3, H=4, W=2, h_limit=2)
    pairs = [("paper", W.paper_program_text(False), W.paper_program_text(True)),
             ("paper_small", small_a, small_b), ("shared", *_shared_prefix_pair()),
             ("c5", W.c5_reference_text(n=1, c=4, hw=5, co=3), W.c5_variant_text(n=1, c=4, hw=5, co=3)),
             ("same_c4", W.c4_text(), W.c4_text()), ("same_c2", W.c2_text(), W.c2_text())]
    cat = tiny_graphs.catalogue()
    for name in sorted(cat)[:10]:
        pairs.append(("cat_" + name, cat[name][0], cat[name][0]))
    return pairs


@pytest.fixture(scope="module")
def B():
    from paper_2609_19611_amd import binding
    return binding


@pytest.mark.parametrize("name,a_text,b_text", _pairs(), ids=[p[0] for p in _pairs()])
def test_library_merge_matches_oracle(B, name, a_text, b_text):
    for trim in (True, False):
        ta, tb, k = B.dg_graph_merge(B.dg_graph_parse(a_text), B.dg_graph_parse(b_text), trim)
        oa, ob, ok = oracle.merge(oracle.Graph(a_text), oracle.Graph(b_text), trim)
        assert k == ok
        for lib_text, orc_text in ((B.dg_graph_text(ta), oa), (B.dg_graph_text(tb), ob)):
            assert _canonical(lib_text) == _canonical(orc_text)


def _canonical(text):
    """Statements with attribute values split into lists (attribute order and
    formatting are not part of a graph)."""
    out = []
    for line in text.strip().split("\n"):
        w = line.split()
        if w[0] == "op" and ";" in w:
            i = w.index(";")
            attrs = tuple(sorted((kv.split("=", 1)[0], tuple(kv.split("=", 1)[1].split(","))) for kv in w[i + 1:]))
            out.append(tuple(w[:i]) + attrs)
        else:
            out.append(tuple(w))
    return out


def test_library_merge_errors(B):
    g = GraphText()
    g.leaf("x", [3, 4])
    g.op("y", "relu", "x")
    g.output("y", [3, 4])
    h = GraphText()
    h.leaf("x", [4, 3])
    h.op("t", "permute", "x", dims=[1, 0])
    h.op("y", "relu", "t")
    h.output("y", [3, 4])
    with pytest.raises(B.DgError) as e:
        B.dg_graph_merge(B.dg_graph_parse(g.text()), B.dg_graph_parse(h.text()))
    assert e.value.name == "DG_E_SIGNATURE"
    with pytest.raises(B.DgError) as e:
        B.dg_graph_merge(B.dg_graph_parse(W.c1_text()), B.dg_graph_parse(W.c4_text()))
    assert e.value.name == "DG_E_SIGNATURE"


def test_graph_text_round_trips(B):
    for text in [W.c1_text(), W.c2_text(), W.c3_text(), W.c4_text(), W.c5_variant_text()]:
        g = B.dg_graph_parse(text)
        t = B.dg_graph_text(g)
        assert _canonical(t) == _canonical(text)
        assert B.dg_graph_text(B.dg_graph_parse(t)) == t
