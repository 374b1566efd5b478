"""Pins of the CPU oracle against facts that do not come from the oracle.

* perturbation of the real PyTorch fp64 program: the footprint set
  (semantic footprint is always a subset of the syntactic one, Sec. 3.4;
  equality on graphs without an invariance);
* autograd of the linearised program: path counts with PyTorch's index
  semantics, softmax and norms through their primitive decompositions;
* literal tree expansion of res (Sec. 3.4, "Back-projection"), which checks
  the oracle's dynamic program against the substitution definition;
* closed forms of the five workloads at their real shapes;
* the worked example of the paper (fig:checker, Sec. 2).
"""

import collections
import json
import math
import os

import numpy as np
import pytest

import oracle
import tiny_graphs
import torch_eval
from paper_2609_19611_amd import workloads as W

CAT = tiny_graphs.catalogue()
GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def oracle_rows(text, locs):
    g = oracle.Graph(text)
    off, ids, cnt = g.enumerate(locs)
    return {l: dict(zip(ids[off[i]:off[i + 1]].tolist(), cnt[off[i]:off[i + 1]].tolist()))
            for i, l in enumerate(locs)}


# -------------------------------------------------------------- path counts
@pytest.mark.parametrize("name", sorted(CAT))
def test_counts_match_linearised_autograd(name):
    text = CAT[name][0]
    g = oracle.Graph(text)
    locs = list(range(g.output_numel))
    assert oracle_rows(text, locs) == torch_eval.path_counts(text, locs)


# ----------------------------------------------------------- footprint sets
# Graphs where a semantic invariance removes leaves from the semantic
# footprint for every input: (leaf name, reason).
INVARIANT = {
    # softmax is shift invariant along its dim, and the bias adds the same
    # mean(b) to every element of a softmax row.
    "c3_small": ("b", "softmax shift invariance"),
    # each softmax row is one channel's flattened map: b[c] shifts the whole row.
    "conv_flatten_softmax": ("b", "softmax shift invariance"),
    # min(max(x, z), x) == x.
    "select_absorb": ("z", "select absorbed"),
}


@pytest.mark.parametrize("name", sorted(CAT))
def test_footprint_matches_perturbation(name):
    text, masks = CAT[name]
    g = oracle.Graph(text)
    n = g.output_numel
    syn = {l: set(r) for l, r in oracle_rows(text, list(range(n))).items()}
    if masks:
        sem = torch_eval.perturbation_footprints(text, draws=10, deltas=(0.5, -0.5, 30.0, -30.0))
    else:
        sem = torch_eval.perturbation_footprints(text, draws=2, deltas=(0.5, -10.0))
    for l in range(n):
        assert sem[l] <= syn[l], f"location {l}: semantic footprint escapes the syntactic one"
    hidden = set()
    if name in INVARIANT:
        leaf = next(t for t in g.leaves if t.name == INVARIANT[name][0])
        hidden = set(range(leaf.base, leaf.base + leaf.numel))
    for l in range(n):
        assert sem[l] == syn[l] - hidden, f"location {l}: {sorted(syn[l] - hidden - sem[l])[:8]} unobserved"


# ------------------------------------------------------------ tree expansion
def _expand(g, t, loc, memo_free_budget):
    """res(T[l]) as a multiset of leaf ids, by literal substitution (no
    sharing of sub-results)."""
    info = g.tensors[t]
    if info.leaf_index >= 0:
        return collections.Counter({info.base + loc: 1})
    out = collections.Counter()
    for tt, idx, m in g.reads(t, loc):
        memo_free_budget[0] -= 1
        assert memo_free_budget[0] > 0, "tree too large for literal expansion"
        sub = _expand(g, tt, idx, memo_free_budget)
        for k, v in sub.items():
            out[k] += v * m
    return out


@pytest.mark.parametrize("name", ["diamond", "self_product", "c1", "c2_small", "c4_small", "softmax",
                                  "group_norm", "c5_small_var", "paper_kernel_small", "reductions", "views"])
def test_dynamic_program_matches_tree_expansion(name):
    text = CAT[name][0]
    g = oracle.Graph(text)
    locs = list(range(min(g.output_numel, 12)))
    rows = oracle_rows(text, locs)
    for l in locs:
        tree = _expand(g, g.output, l, [2_000_000])
        assert dict(tree) == rows[l]


# --------------------------------------------------------------- closed forms
def _row_by_leaf(g, row):
    out = {}
    for t in g.leaves:
        out[t.name] = {gid - t.base: c for gid, c in row.items() if t.base <= gid < t.base + t.numel}
    return out


def test_c1_closed_form():
    g = oracle.Graph(W.c1_text())
    off, ids, cnt = g.enumerate(range(8))
    assert off[-1] == 1152
    for i in range(8):
        row = _row_by_leaf(g, dict(zip(ids[off[i]:off[i + 1]].tolist(), cnt[off[i]:off[i + 1]].tolist())))
        # y[i] = sum_j relu(sum_k A[i,k] B[k,j]): A[i,k] on 8 paths, B[k,j] on one.
        assert row["A"] == {i * 16 + k: 8 for k in range(16)}
        assert row["B"] == {f: 1 for f in range(128)}


def _pool_conv_counts(p, n_in):
    """1-D count of input position i for pooled output p of maxpool(2,2)
    over conv(k3, s1, p1): the number of (pool offset a, tap t) pairs with
    i = 2p + a - 1 + t in range."""
    c = collections.Counter()
    for a in range(2):
        for t in range(3):
            i = 2 * p + a - 1 + t
            if 0 <= i < n_in:
                c[i] += 1
    return c


def _pool_tap_counts(p, n_in):
    c = collections.Counter()
    for a in range(2):
        for t in range(3):
            if 0 <= 2 * p + a - 1 + t < n_in:
                c[t] += 1
    return c


def test_c2_closed_form():
    g = oracle.Graph(W.c2_text())
    locs = W.config_locations("c2")
    assert len(locs) == 4096
    sample = locs[:40] + [0, 15, 255, 65535, 16 * 256 + 17]
    rows = oracle_rows(W.c2_text(), sample)
    for l in sample:
        n, c, ph, pw = np.unravel_index(l, (16, 16, 16, 16))
        row = _row_by_leaf(g, rows[l])
        ch, cw = _pool_conv_counts(ph, 32), _pool_conv_counts(pw, 32)
        th, tw = _pool_tap_counts(ph, 32), _pool_tap_counts(pw, 32)
        exp_x = {((n * 3 + ci) * 32 + i) * 32 + j: ch[i] * cw[j] for ci in range(3) for i in ch for j in cw}
        exp_w = {((c * 3 + ci) * 3 + a) * 3 + b: th[a] * tw[b] for ci in range(3) for a in th for b in tw}
        assert row["x"] == exp_x
        assert row["W"] == exp_w
        assert row["conv_b"] == {c: 4} and row["bias"] == {c: 4}
        r = lambda q: 3 if q in (0, 15) else 4
        assert len(rows[l]) == 29 + 3 * r(ph) * r(pw)
        assert set(ch.values()) <= {1, 2}


def test_c3_closed_form():
    g = oracle.Graph(W.c3_text())
    locs = W.config_locations("c3")
    assert len(locs) == 65536 and locs == sorted(set(locs))
    picks = [0, 1 * 4096 + 1 * 64 + 1, 31 * 4096 + 63 * 64 + 63, 29 * 4096 + 61 * 64 + 5,
             30 * 4096 + 2 * 64 + 62, 13 * 4096 + 40 * 64 + 0, 7 * 131072 + 17 * 4096 + 33 * 64 + 9]
    rows = oracle_rows(W.c3_text(), picks)
    for l in picks:
        n, d, h, w = np.unravel_index(l, (8, 32, 64, 64))
        td = 2 if (d % 2 == 1 and d <= 29) else 1
        th = 2 if (h % 2 == 1 and h <= 61) else 1
        row = _row_by_leaf(g, rows[l])
        assert len(rows[l]) == 7168 * td * th + 64
        # bias: 64 softmax-row elements, plus the numerator once more.
        assert row["b"] == {co: 65 for co in range(64)}
        T = lambda iw: {v for v in (2 * iw - 1, 2 * iw, 2 * iw + 1) if 0 <= v < 64}
        for f, cnt in row["x"].items():
            iw = f % 32
            assert cnt == 64 * (len(T(iw)) + (w in T(iw)))
        S = {0: {2 * i - 1 for i in range(1, 32)}, 1: {2 * i for i in range(32)}, 2: {2 * i + 1 for i in range(32)}}
        for f, cnt in row["W"].items():
            kw = f % 3
            assert cnt == len(S[kw]) + (w in S[kw])
        assert set(row["x"].values()) <= {128, 192, 256}


def test_c4_closed_form():
    g = oracle.Graph(W.c4_text())
    picks = [0, 1, 511, 512 * 37 + 200, 65535]
    rows = oracle_rows(W.c4_text(), picks)
    for l in picks:
        n, c = divmod(l, 512)
        grp = c // 64
        row = _row_by_leaf(g, rows[l])
        assert len(rows[l]) == 66626
        # GroupNorm over |S| = 64 features: h2[n, c'] counts 64 + 2 + [c' = c].
        assert row["x"] == {n * 1024 + k: 64 * 66 + 1 + (k == c) for k in range(1024)}
        assert row["W"] == {k * 512 + cc: 66 + (cc == c) for k in range(1024) for cc in range(grp * 64, grp * 64 + 64)}
        assert row["bias"] == {cc: 66 + (cc == c) for cc in range(grp * 64, grp * 64 + 64)}
        assert row["gamma"] == {c: 1} and row["beta"] == {c: 1}


def test_c5_closed_form_and_clean_variant():
    ref = oracle.Graph(W.c5_reference_text())
    var = oracle.Graph(W.c5_variant_text())
    locs = W.config_locations("c5")
    assert len(locs) == 1048576
    picks = locs[:6] + [0, 63, 64 * 5 + 7, 33554431]
    rr = oracle_rows(W.c5_reference_text(), picks)
    for l in picks:
        n, co, h, w = np.unravel_index(l, (64, 128, 64, 64))
        r = lambda q: 2 if q in (0, 63) else 3
        assert len(rr[l]) == 128 * r(h) * r(w) + 3
        assert set(rr[l].values()) == {1}
    # Split-K and channels-last change neither the footprint nor the counts.
    assert not oracle.compare(ref, var, picks).any()


def test_c5_faults_are_detected_or_neutral():
    faults = W.c5_faults()
    assert len(faults) == 16 and len(set(faults)) == 16
    ref = oracle.Graph(W.c5_reference_text(n=2, c=4, hw=6, co=3))
    locs = list(range(2 * 3 * 6 * 6))
    for f in faults:
        var = oracle.Graph(W.c5_variant_text(fault=f, n=2, c=4, hw=6, co=3))
        st = oracle.compare(ref, var, locs)
        # An index-map fault always moves some read of this shape somewhere.
        assert st.any(), f


# ---------------------------------------------------------- paper example
def test_paper_worked_example():
    gold = json.load(open(os.path.join(GOLDEN, "paper_example.json")))
    ref = oracle.Graph(W.paper_reference_text())
    ker = oracle.Graph(W.paper_kernel_text())
    assert list(ref.output_shape) == gold["Y_shape"]
    loc = int(np.ravel_multi_index(gold["location_multi_index"], gold["Y_shape"]))
    assert loc == gold["location_flat"]
    for g, key, size_key in ((ref, "reference_footprint", "reference_row_size"),
                             (ker, "kernel_footprint", "kernel_row_size")):
        row = g.row(loc)
        assert len(row) == gold[size_key]
        assert set(row.values()) == {gold["all_counts"]}
        fp = gold[key]
        M = next(t for t in g.leaves if t.name == "M")
        b = next(t for t in g.leaves if t.name == "b")
        exp = {M.base + int(np.ravel_multi_index((fp["M"]["n"], c, h, fp["M"]["w"]), gold["M_shape"]))
               for c in range(*fp["M"]["c_range"]) for h in range(*fp["M"]["h_range"])}
        exp |= {b.base + i for i in fp["b"]}
        assert set(row) == exp
    sec2 = int(np.ravel_multi_index(gold["sec2_location_multi_index"], gold["Y_shape"]))
    assert list(oracle.compare(ker, ref, [loc, sec2])) == [gold["compare_status"]] * 2


def test_paper_example_fixed_kernel_is_equivalent():
    # With the loop bound fixed (s >= 32) the kernel sums every h.
    ref = oracle.Graph(W.paper_reference_text(N=4, C=3, H=8, W=5))
    fixed = oracle.Graph(W.paper_kernel_text(N=4, C=3, H=8, W=5, h_limit=8))
    assert not oracle.compare(fixed, ref, range(4 * 3 * 5)).any()


# ----------------------------------------------------------------- compare
def test_compare_status_codes():
    a = oracle.Graph(CAT["self_product"][0])  # y = (x*x + x) * w: x counts 3
    txt_b = tiny_graphs._g([("x", [3, 2]), ("w", [2])],
                           [("a", "add", ["x", "x"], {}), ("y", "mul", ["a", "w"], {})], "y", [3, 2])
    txt_c = tiny_graphs._g([("x", [3, 2]), ("w", [2])],
                           [("a", "neg", ["w"], {}), ("y", "mul", ["x", "a"], {})], "y", [3, 2])
    b, c = oracle.Graph(txt_b), oracle.Graph(txt_c)
    assert list(oracle.compare(a, a, range(6))) == [0] * 6
    assert list(oracle.compare(a, b, range(6))) == [2] * 6  # same ids, counts 3 vs 2
    assert list(oracle.compare(b, c, range(6))) == [2] * 6  # 2 vs 1
    d = oracle.Graph(tiny_graphs._g([("x", [3, 2]), ("w", [2])], [("y", "relu", ["x"], {})], "y", [3, 2]))
    assert list(oracle.compare(a, d, range(6))) == [1] * 6
    e = oracle.Graph(tiny_graphs._g([("x", [3, 2]), ("v", [2])], [("y", "relu", ["x"], {})], "y", [3, 2]))
    with pytest.raises(oracle.OracleError):
        oracle.compare(d, e, range(6))


def test_threads_do_not_change_results():
    text = W.c2_text()
    g = oracle.Graph(text)
    locs = W.config_locations("c2")[:300]
    a = g.enumerate(locs, threads=1)
    b = g.enumerate(locs, threads=4)
    for x, y in zip(a, b):
        assert np.array_equal(x, y)


# ------------------------------------------------------------- error paths
@pytest.mark.parametrize("text,msg", [
    ("leaf x 2\noutput x 2\n", "header"),
    ("dgir 1\nleaf x 2,0\noutput x 2,0\n", "positive"),
    ("dgir 1\nleaf x 2\nop y frobnicate x\noutput y 2\n", "unsupported"),
    ("dgir 1\nleaf x 2,3\nleaf z 4\nop y add x z\noutput y 2,3\n", "broadcast"),
    ("dgir 1\nleaf x 2\nop y relu q\noutput y 2\n", "unknown operand"),
    ("dgir 1\nleaf x 2\nop y relu x\noutput y 3\n", "declared shape"),
    ("dgir 1\nleaf x 2\nop y relu x\n", "output"),
    ("dgir 1\nleaf x 2,3\nop y affine_gather x ; shape=2 idx0=o0+,o1\noutput y 2\n", "expression"),
])
def test_parse_errors(text, msg):
    with pytest.raises(oracle.OracleError) as e:
        oracle.Graph(text)
    assert msg in str(e.value)


def test_location_out_of_range_and_overflow():
    g = oracle.Graph(W.c1_text())
    with pytest.raises(oracle.OracleError):
        g.enumerate([8])
    with pytest.raises(oracle.OracleError):
        g.enumerate([-1])
    # Nested layer norms over 4096 elements: counts pass 2**32.
    with pytest.raises(oracle.OracleError) as e:
        oracle.Graph(tiny_graphs.nested_layer_norms(4096)).enumerate([0])
    assert "32 bits" in str(e.value)


@pytest.mark.parametrize("n,loc", [(5, 3), (4096, 0), (4096, 4095)])
def test_wide_counts_closed_form(n, loc):
    """64-bit path counts past 2^32 (n = 4096 gives about 1.2e18)."""
    off, ids, cnt = oracle.Graph(tiny_graphs.nested_layer_norms(n)).enumerate([loc], wide=True)
    assert ids.dtype == np.uint64 and cnt.dtype == np.uint64
    assert off.tolist() == [0, n]
    assert ids.tolist() == list(range(n))
    assert cnt.tolist() == tiny_graphs.nested_layer_norm_counts(n, loc)
    if n == 4096:
        assert int(cnt.min()) > 2 ** 32


def test_wide_equals_narrow_where_both_fit():
    for name in ("c1", "c2", "c3"):
        g = oracle.Graph(W.CONFIGS[name]["text"]())
        locs = W.config_locations(name)[:64]
        o32, i32, c32 = g.enumerate(locs)
        o64, i64, c64 = g.enumerate(locs, wide=True)
        assert (o32 == o64).all()
        assert (i32.astype(np.uint64) == i64).all() and (c32.astype(np.uint64) == c64).all()


def test_leaf_total_limit():
    """Graphs up to 2^62 leaf elements parse; 32-bit ids refuse more than
    2^32 - 1 of them; 64-bit ids name a leaf past 2^32 as its base plus its
    flat index (leaves in declaration order)."""
    with pytest.raises(oracle.OracleError) as e:
        oracle.Graph("dgir 1\nleaf x 1073741824,1073741824,8\noutput x 1073741824,1073741824,8\n")
    assert "2^62" in str(e.value)
    g = oracle.Graph("dgir 1\nleaf a 65536,65536\nleaf x 8\nop y relu x\noutput y 8\n")
    assert g.leaf_total == 2 ** 32 + 8
    with pytest.raises(oracle.OracleError) as e:
        g.enumerate([0])
    assert "64 bits" in str(e.value)
    off, ids, cnt = g.enumerate([0, 5, 7], wide=True)
    assert off.tolist() == [0, 1, 2, 3]
    assert ids.tolist() == [2 ** 32, 2 ** 32 + 5, 2 ** 32 + 7]
    assert cnt.tolist() == [1, 1, 1]



@pytest.mark.parametrize("text", tiny_graphs.OVERFLOWING_SHAPES)
def test_element_counts_past_2_62_are_rejected(text):
    with pytest.raises(oracle.OracleError) as e:
        oracle.Graph(text)
    assert "2^62" in str(e.value)
