"""GPU parity of the expression DAGs of res(y[l]) (dg_dag_sizes,
dg_dag_fill) against the oracle's DAGs, element by element, through the C
ABI: every location of the small catalogue graphs, samples of the five
workloads (c5's variant and faulty variants too), error paths."""

import os

import numpy as np
import pytest
import torch

import oracle
import tiny_graphs
from paper_2609_19611_amd import workloads as W

pytestmark = pytest.mark.gpu

CAT = tiny_graphs.catalogue()
SEPARABLE = sorted(CAT)
KEYS = ("node_offsets", "edge_offsets", "nodes", "node_edge", "edges", "mults")


@pytest.fixture(scope="module")
def B():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_19611_amd import binding
    return binding


def _host(d):
    out = {}
    for k in KEYS:
        a = d[k].cpu().numpy()
        out[k] = a if a.dtype == np.int64 else a.view(np.uint32).astype(np.uint64)
    return out


def _check(B, text, locs, threads=16):
    got = _host(B.dag_locations(B.dg_graph_parse(text), locs))
    want = oracle.Graph(text).dag(locs, threads=threads)
    for k in KEYS:
        assert np.array_equal(got[k], want[k]), k
    return got


@pytest.mark.parametrize("name", SEPARABLE)
def test_dag_catalogue_all_locations(B, name):
    text = CAT[name][0]
    n = oracle.Graph(text).output_numel
    _check(B, text, list(range(n))[::-1])


DAGCAT = tiny_graphs.dag_catalogue()


@pytest.mark.parametrize("name", sorted(DAGCAT))
def test_dag_extra_catalogue(B, name):
    text = DAGCAT[name]
    n = oracle.Graph(text).output_numel
    _check(B, text, list(range(n))[::-1])


@pytest.mark.parametrize("name,step", [("c1", 1), ("c2", 1), ("c3", 1024), ("c4", 64), ("c5", 256)])
def test_dag_workloads(B, name, step):
    locs = W.config_locations(name)[::step]
    _check(B, W.CONFIGS[name]["text"](), locs)


def test_dag_c5_variants(B):
    locs = W.config_locations("c5")[::4096]
    for text in [W.c5_variant_text()] + [W.c5_variant_text(fault=f) for f in W.c5_faults()]:
        _check(B, text, locs)


def test_dag_c5_boundaries(B):
    """DAGs at the output's padding edges of c5's reference, its split-K
    variant and every fault, against the oracle."""
    N, C, H, Wd = 64, 128, 64, 64
    locs = [((n * C + c) * H + h) * Wd + w for n in (0, N - 1) for c in (0, C - 1)
            for h in (0, 1, H - 2, H - 1) for w in (0, 1, Wd - 2, Wd - 1)]
    texts = [W.c5_reference_text(), W.c5_variant_text()] + [W.c5_variant_text(fault=f) for f in W.c5_faults()]
    for text in texts:
        _check(B, text, locs)


def test_dag_edge_cases(B):
    g = B.dg_graph_parse(W.c2_text())
    d = B.dag_locations(g, torch.empty(0, dtype=torch.int64))
    assert d["node_offsets"].cpu().tolist() == [0] and d["edges"].numel() == 0
    _check(B, W.c2_text(), [65535, 3, 3, 0])
    with pytest.raises(B.DgError) as e:
        B.dag_locations(g, [0, 65536])
    assert e.value.name == "DG_E_RANGE"
    # Output that is a leaf: no nodes, no edges.
    d = B.dag_locations(B.dg_graph_parse("dgir 1\nleaf x 4\noutput x 4\n"), [0, 3])
    assert d["node_offsets"].cpu().tolist() == [0, 0, 0] and d["edge_offsets"].cpu().tolist() == [0, 0, 0]


def test_default_kernel_choice_for_large_dags(B):
    """By default a call over the conv-transpose + softmax DAGs (millions of
    edges per location, 64 of them here) takes the specialised DAG kernels;
    the result is the oracle's."""
    if os.environ.get("DIRIGO_DAG_JIT") or os.environ.get("DIRIGO_JIT") == "0":
        pytest.skip("the default choice only")
    text = W.CONFIGS["c3"]["text"]()
    g = B.dg_graph_parse(text)
    locs = W.config_locations("c3")[::1024]
    got = _host(B.dag_locations(g, locs))
    info = B.dg_graph_info(g)
    assert info["dag_specialized"] == 1
    assert len(locs) * info["dag_edge_bound"] >= 1 << 26
    want = oracle.Graph(text).dag(locs, threads=16)
    for k in KEYS:
        assert np.array_equal(got[k], want[k]), k
