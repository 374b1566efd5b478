"""CPU checks of the library's compiler and block code.

The host-emulation test library runs the compiled per-location plans and
the same block code as the GPU kernels with a block of one host thread; its
rows must equal the oracle's bit for bit.  (The GPU parity tests in
test_gpu_parity.py check the real kernels.)
"""

import numpy as np
import pytest

import hostemu
import oracle
import tiny_graphs
from paper_2609_19611_amd import workloads as W

CAT = tiny_graphs.catalogue()
SEPARABLE = sorted(CAT)


def assert_same(a, b):
    for x, y in zip(a, b):
        assert np.array_equal(np.asarray(x), np.asarray(y))


@pytest.mark.parametrize("name", SEPARABLE)
def test_catalogue_matches_oracle(name):
    text = CAT[name][0]
    g = oracle.Graph(text)
    locs = list(range(g.output_numel))
    assert_same(hostemu.enumerate(text, locs), g.enumerate(locs))


def test_unrefinable_reshape_rejected():
    """A reshape between two factorisations of one block with no common
    refinement is refused (the oracle takes it)."""
    with pytest.raises(hostemu.HostEmuError) as e:
        hostemu.enumerate(tiny_graphs.UNREFINABLE_RESHAPE, [0])
    assert e.value.code == -4
    assert oracle.Graph(tiny_graphs.UNREFINABLE_RESHAPE).output_numel == 24


@pytest.mark.parametrize("name,a,b", tiny_graphs.merged_view_pairs())
def test_compare_pairs_viewed_with_different_merged_dims(name, a, b):
    """Graphs over the same leaves, one reading a leaf through merged dims:
    the comparison views both over the joined dims, against the oracle."""
    n = oracle.Graph(a).output_numel
    want = oracle.compare(oracle.Graph(a), oracle.Graph(b), range(n))
    assert np.array_equal(hostemu.compare(a, b, range(n)), want)
    assert np.array_equal(hostemu.compare(b, a, range(n)), want)
    assert set(want.tolist()) == {{"same_footprint": 0, "sliced": 1}.get(name, 2)}


@pytest.mark.parametrize("name", ["c1", "c2", "c3", "c4", "c5"])
def test_workload_samples_match_oracle(name):
    text = W.CONFIGS[name]["text"]()
    locs = W.config_locations(name)
    rng = np.random.default_rng(7)
    k = {"c1": 8, "c2": 64, "c3": 6, "c4": 3, "c5": 24}[name]
    pick = sorted(set(rng.choice(locs, size=min(k, len(locs)), replace=False).tolist()) | {locs[0], locs[-1]})
    assert_same(hostemu.enumerate(text, pick), oracle.Graph(text).enumerate(pick, threads=4))


def test_unsorted_and_duplicate_locations():
    text = W.c2_text()
    locs = [65535, 3, 3, 40000, 0, 3]
    assert_same(hostemu.enumerate(text, locs), oracle.Graph(text).enumerate(locs))


def test_compare_clean_and_faults():
    ref = W.c5_reference_text(n=2, c=4, hw=6, co=3)
    locs = list(range(2 * 3 * 6 * 6))
    assert not hostemu.compare(ref, W.c5_variant_text(n=2, c=4, hw=6, co=3), locs).any()
    g_ref = oracle.Graph(ref)
    for f in W.c5_faults():
        var = W.c5_variant_text(fault=f, n=2, c=4, hw=6, co=3)
        assert np.array_equal(hostemu.compare(ref, var, locs), oracle.compare(g_ref, oracle.Graph(var), locs)), f


def test_compare_status_two():
    a = CAT["self_product"][0]
    b = tiny_graphs._g([("x", [3, 2]), ("w", [2])], [("a", "add", ["x", "x"], {}), ("y", "mul", ["a", "w"], {})],
                       "y", [3, 2])
    assert list(hostemu.compare(a, b, range(6))) == [2] * 6
    assert list(hostemu.compare(a, a, range(6))) == [0] * 6


@pytest.mark.parametrize("shape", [[1, 6, 12], [2, 6, 12]])
def test_compare_counts_near_2_32(shape):
    """Both static bounds below 2^32, so the comparison's tables and sums
    are 32-bit; counts reach 2,101,864,255."""
    a = tiny_graphs.large_count_norms(shape)
    n = oracle.Graph(a).output_numel
    for v in ("permuted", "mid_1d"):
        b = tiny_graphs.large_count_norms(shape, v)
        want = oracle.compare(oracle.Graph(a), oracle.Graph(b), range(n))
        assert np.array_equal(hostemu.compare(a, b, list(range(n))), want)
        assert set(want.tolist()) == ({0} if v == "permuted" else {2})


def test_paper_example():
    st = hostemu.compare(W.paper_kernel_text(), W.paper_reference_text(), [11596, 0, 131071])
    assert list(st) == [1, 1, 1]


def test_range_and_overflow_errors():
    with pytest.raises(hostemu.HostEmuError) as e:
        hostemu.enumerate(W.c1_text(), [8])
    assert e.value.code == -5
    txt = tiny_graphs._g([("x", [1, 4096])],
                         [("a", "layer_norm", ["x"], dict(ndims=1)), ("b", "layer_norm", ["a"], dict(ndims=1)),
                          ("y", "layer_norm", ["b"], dict(ndims=1))], "y", [1, 4096])
    with pytest.raises(hostemu.HostEmuError) as e:
        hostemu.enumerate(txt, [0])
    assert e.value.code == -6


# ---- expression DAGs (the library's DAG block code on one host thread) ----
_CAT = tiny_graphs.catalogue()
_SEP = sorted(_CAT)


def _dag_equal(a, b):
    for k in ("node_offsets", "edge_offsets", "nodes", "node_edge", "edges", "mults"):
        assert np.array_equal(np.asarray(a[k]), np.asarray(b[k])), k


@pytest.mark.parametrize("name", _SEP)
def test_dag_catalogue(name):
    text = _CAT[name][0]
    g = oracle.Graph(text)
    n = g.output_numel
    locs = list(range(n)) if n <= 256 else sorted(set(np.linspace(0, n - 1, 96).astype(int).tolist()))
    _dag_equal(hostemu.dag(text, locs), g.dag(locs))


@pytest.mark.parametrize("name,count", [("c1", 8), ("c2", 64), ("c3", 2), ("c4", 3), ("c5", 8)])
def test_dag_workloads(name, count):
    text = W.CONFIGS[name]["text"]()
    locs = W.config_locations(name)
    locs = [locs[i] for i in np.linspace(0, len(locs) - 1, count).astype(int)]
    _dag_equal(hostemu.dag(text, locs), oracle.Graph(text).dag(locs, threads=4))


_DAGCAT = tiny_graphs.dag_catalogue()


@pytest.mark.parametrize("name", sorted(_DAGCAT))
def test_dag_extra_catalogue(name):
    """Coupled window indices (point by point), an oversized list table,
    grouped conv-transpose, boundary reads, coupled reads of a non-leaf."""
    text = _DAGCAT[name]
    g = oracle.Graph(text)
    locs = list(range(g.output_numel))[::-1]
    _dag_equal(hostemu.dag(text, locs), g.dag(locs))


def test_dag_paths_taken():
    """Each way of taking a group is exercised: by progressions (with and
    without an exact division), point by point (two window variables in one
    index, floor division of a window variable), pointwise."""
    rows = {name: hostemu.dag_groups(text) for name, text in _DAGCAT.items()}
    assert any(r[1] == 0 and r[2] == 0 for r in rows["gather_coupled"])
    assert any(r[1] == 0 and r[2] == 0 for r in rows["gather_coupled_nonleaf"])
    assert any(r[1] == 0 and r[2] == 1 and r[3] == 1 for r in rows["gather_big_list"])
    assert any(r[1] == 1 for r in rows["gather_shift"])
    floor = hostemu.dag_groups(_CAT["gather_floor_flat"][0])
    assert any(r[1] == 0 and r[2] == 0 for r in floor)
    c3 = hostemu.dag_groups(W.c3_text())
    assert c3[0][2] == 1 and c3[0][3] == 3  # conv-transpose taps: exact divisions
    assert all(r[2] == 1 for r in hostemu.dag_groups(W.c4_text()))


def test_dag_c5_variants():
    locs = W.config_locations("c5")[::262144]
    for text in [W.c5_variant_text()] + [W.c5_variant_text(fault=f) for f in W.c5_faults()[:4]]:
        _dag_equal(hostemu.dag(text, locs), oracle.Graph(text).dag(locs))


@pytest.mark.parametrize("name,a,b,interior", tiny_graphs.factored_compare_pairs())
def test_factored_comparison_of_single_term_leaves(name, a, b, interior):
    """Single-term leaves compared factor by factor: support changes in one
    dim, a tap count changed in one dim, counts scaled, another leaf's
    counts changed; every location against the oracle."""
    from paper_2609_19611_amd import binding
    for t in (a, b):
        assert binding.dg_graph_info(binding.dg_graph_parse(t))["max_leaf_terms"] == 1
    n = oracle.Graph(a).output_numel
    want = oracle.compare(oracle.Graph(a), oracle.Graph(b), range(n))
    assert want[n // 2] == interior
    assert np.array_equal(hostemu.compare(a, b, range(n)), want)
    assert np.array_equal(hostemu.compare(b, a, range(n)), want)


def test_split_k_variant_has_single_term_leaves():
    """The canonical forms of factors make every leaf of the split-K NHWC
    variant one term (equal factors share a slot, so its K-split pieces
    merge), at the workload's full size and at a small one."""
    from paper_2609_19611_amd import binding
    for text in (W.c5_variant_text(), W.c5_variant_text(n=2, c=4, hw=6, co=3)):
        assert binding.dg_graph_info(binding.dg_graph_parse(text))["max_leaf_terms"] == 1


@pytest.mark.parametrize("seed", range(12))
def test_frontier_box_dedup_matches_sorted_unique(seed):
    """The frontier dedup by bounding-box bitmap gives exactly the sorted
    set of the candidates (duplicates, one-cell boxes, boxes touching a
    tensor's edges, rank 1 to 5), and declines when its scratch is short."""
    rng = np.random.default_rng(seed)
    rank = int(rng.integers(1, 6))
    shape = [int(rng.integers(1, 9)) for _ in range(rank)]
    lo = [int(rng.integers(0, s)) for s in shape]
    hi = [int(rng.integers(l, s)) + 1 for l, s in zip(lo, shape)]
    stride = np.cumprod([1] + shape[::-1])[:-1][::-1]
    n = int(rng.integers(2, 200))
    coords = np.stack([rng.integers(l, h, size=n) for l, h in zip(lo, hi)], axis=1)
    cand = (coords * stride).sum(axis=1).astype(np.uint32)
    want = np.unique(cand)
    box = int(np.prod([h - l for l, h in zip(lo, hi)]))
    got, ok = hostemu.box_unique(shape, cand, 16 + 2 * ((box + 31) // 32))
    assert ok
    assert got.tolist() == want.tolist()
    # Scratch for one bitmap word only (16 words hold the box bounds of up
    # to 8 dims): declined when the candidates' box spans more.
    vol = np.prod([int(coords[:, d].max() - coords[:, d].min() + 1) for d in range(rank)])
    got, ok = hostemu.box_unique(shape, cand, 16 + 2)
    assert ok == (vol <= 32)
    if ok:
        assert got.tolist() == want.tolist()
