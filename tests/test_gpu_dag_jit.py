"""GPU parity of the specialised expression-DAG kernels (each DAG program
compiled at run time with its ops walked unrolled and only the ways of
taking a group that it uses) against the oracle, element by element,
through the C ABI: every location of one catalogue graph per combination of
ways of taking a group (compiling every catalogue graph would take minutes),
samples of the five workloads, c5's variant and some of its faults.
DIRIGO_DAG_JIT=1 makes every call take them (by default only large calls
do)."""

import ctypes
import os
import re

import numpy as np
import pytest
import torch

import gpu_warm
import hostemu
import oracle
import tiny_graphs
from paper_2609_19611_amd import workloads as W

pytestmark = pytest.mark.gpu

KEYS = ("node_offsets", "edge_offsets", "nodes", "node_edge", "edges", "mults")


def _ways(text):
    """The ways of taking a group compiled into the graph's specialised DAG
    kernels (the masks of its source), for the block size the library
    picks."""
    nodes, edges, frontier, _ = hostemu.dag_bounds(text, 64)
    block = 256 if edges >= 4096 and frontier > 256 else 64
    t = text.encode()
    buf = ctypes.create_string_buffer(1 << 24)
    assert hostemu.lib().dgh_jit_dag_source(t, len(t), block, buf, len(buf)) > 0
    return tuple(re.findall(r"#define (DG_DAG_(?:FAST|NODE|SLOW|BOX|PW) \S+)", buf.value.decode()))


def _one_per_way(graphs):
    seen, out = set(), {}
    for name in sorted(graphs):
        w = _ways(graphs[name])
        if w not in seen:
            seen.add(w)
            out[name] = graphs[name]
    return out


CAT = _one_per_way({**{k: v[0] for k, v in tiny_graphs.catalogue().items()}, **tiny_graphs.dag_catalogue()})
WORK = {name: W.CONFIGS[name]["text"]() for name in ("c1", "c2", "c3", "c4", "c5")}
C5 = ([W.c5_variant_text()] + [W.c5_variant_text(fault=f) for f in W.c5_faults()[:4]]
      + [W.c5_variant_text(fault=f) for f in W.C5_SPARSE_FAULTS])


@pytest.fixture(scope="module")
def B():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_19611_amd import binding
    return binding


@pytest.fixture(scope="module")
def graphs(B):
    """Handles of every graph here, their specialised DAG kernels compiled
    (several at once) and kept loaded for the module."""
    old = os.environ.get("DIRIGO_DAG_JIT")
    os.environ["DIRIGO_DAG_JIT"] = "1"
    texts = list(CAT.values()) + list(WORK.values()) + C5
    handles = gpu_warm.warm_dags(B, texts, threads=16)
    yield dict(zip(texts, handles))
    if old is None:
        del os.environ["DIRIGO_DAG_JIT"]
    else:
        os.environ["DIRIGO_DAG_JIT"] = old


def test_specialised_dag_kernels_loaded(B, graphs):
    for g in graphs.values():
        info = B.dg_graph_info(g)
        assert info["dag_specialized"] == 1
        assert info["dag_block_threads"] in (64, 256) and info["dag_lds_bytes"] > 0 and info["dag_edge_bound"] > 0


def _check(B, g, text, locs):
    d = B.dag_locations(g, locs)
    want = oracle.Graph(text).dag(locs, threads=16)
    for k in KEYS:
        a = d[k].cpu().numpy()
        a = a if a.dtype == np.int64 else a.view(np.uint32).astype(np.uint64)
        assert np.array_equal(a, want[k]), k


@pytest.mark.parametrize("name", sorted(CAT))
def test_specialised_dag_catalogue(B, graphs, name):
    text = CAT[name]
    n = oracle.Graph(text).output_numel
    _check(B, graphs[text], text, list(range(n))[::-1])


@pytest.mark.parametrize("name,step", [("c1", 1), ("c2", 1), ("c3", 1024), ("c4", 64), ("c5", 256)])
def test_specialised_dag_workloads(B, graphs, name, step):
    text = WORK[name]
    _check(B, graphs[text], text, W.config_locations(name)[::step])


def test_specialised_dag_c5_variants(B, graphs):
    locs = W.config_locations("c5")[::4096]
    N, C, H, Wd = 64, 128, 64, 64
    edges = [((n * C + c) * H + h) * Wd + w for n in (0, N - 1) for c in (0, C - 1)
             for h in (0, 1, H - 2, H - 1) for w in (0, 1, Wd - 2, Wd - 1)]
    for text in C5:
        _check(B, graphs[text], text, locs + edges)


def test_specialised_dag_edge_cases(B, graphs):
    """A graph whose output is a leaf (a DAG program with no ops), an empty
    location list, and an out-of-range location, on the specialised DAG
    kernels."""
    g = B.dg_graph_parse("dgir 1\nleaf x 4\noutput x 4\n")
    d = B.dag_locations(g, [0, 3])
    assert d["node_offsets"].cpu().tolist() == [0, 0, 0] and d["edge_offsets"].cpu().tolist() == [0, 0, 0]
    text = WORK["c2"]
    g2 = graphs[text]
    d = B.dag_locations(g2, torch.empty(0, dtype=torch.int64))
    assert d["node_offsets"].cpu().tolist() == [0] and d["edges"].numel() == 0
    with pytest.raises(B.DgError) as e:
        B.dag_locations(g2, [0, 65536])
    assert e.value.name == "DG_E_RANGE"
    _check(B, g2, text, [65535, 3, 3, 0])
