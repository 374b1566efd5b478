"""Seeded random graphs over the whole op vocabulary (fuzz_graphs.py) on the
GPU, through the C ABI, against the oracle at every output location: the
single-pass and two-pass enumerations, expression DAGs and comparisons with
a variant whose counts double, with the precompiled kernels on 160 graphs
and the specialised ones (DAG kernels included) on 16 of them."""

import numpy as np
import pytest
import torch

import fuzz_graphs
import gpu_warm
import oracle
from fuzz_graphs import REFUSALS, squared_variant

pytestmark = pytest.mark.gpu

DAG_KEYS = ("node_offsets", "edge_offsets", "nodes", "node_edge", "edges", "mults")


@pytest.fixture(scope="module")
def B():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_19611_amd import binding
    return binding


def _u32(t):
    return t.cpu().numpy().view(np.uint32)


def check_graph(B, seed, dags):
    text = fuzz_graphs.random_graph(seed)
    og = oracle.Graph(text)
    try:
        g = B.dg_graph_parse(text)
    except B.DgError as e:
        assert e.name == "DG_E_UNSUPPORTED_OP" and any(r in str(e) for r in REFUSALS), (seed, str(e))
        return False
    locs = list(range(og.output_numel))
    ro, io, co = og.enumerate(locs)
    off, ids, cnt = B.enumerate_locations(g, locs)
    assert np.array_equal(off.cpu().numpy(), ro), seed
    assert np.array_equal(_u32(ids), io) and np.array_equal(_u32(cnt), co), seed
    d_locs = torch.as_tensor(locs[::-1], dtype=torch.int64, device="cuda")
    ws = B.workspace(g, len(locs))
    off1 = torch.empty(len(locs) + 1, dtype=torch.int64, device="cuda")
    ids1 = torch.empty(max(1, int(ro[-1])), dtype=torch.int32, device="cuda")
    cnt1 = torch.empty_like(ids1)
    assert B.dg_enumerate(g, d_locs, off1, ids1, cnt1, ws) == int(ro[-1])
    r2 = og.enumerate(locs[::-1])
    assert np.array_equal(off1.cpu().numpy(), r2[0]), seed
    assert np.array_equal(_u32(ids1)[:int(ro[-1])], r2[1]) and np.array_equal(_u32(cnt1)[:int(ro[-1])], r2[2]), seed
    var = squared_variant(text)
    st, _ = B.compare_locations(g, B.dg_graph_parse(var), locs)
    assert np.array_equal(st.cpu().numpy(), oracle.compare(og, oracle.Graph(var), locs)), seed
    if dags:
        d = B.dag_locations(g, locs)
        want = og.dag(locs)
        for k in DAG_KEYS:
            a = d[k].cpu().numpy()
            a = a if a.dtype == np.int64 else a.view(np.uint32).astype(np.uint64)
            assert np.array_equal(a, want[k]), (seed, k)
    return True


@pytest.mark.parametrize("chunk", range(4))
def test_fuzz_precompiled_kernels(B, chunk, monkeypatch):
    monkeypatch.setenv("DIRIGO_JIT", "0")
    done = sum(check_graph(B, seed, dags=True) for seed in range(chunk * 40, (chunk + 1) * 40))
    assert done >= 38


def test_fuzz_specialized_kernels(B, monkeypatch):
    """The same graphs' enumeration, comparison and DAG kernels specialised
    (DIRIGO_DAG_JIT=1: every DAG call takes the specialised DAG kernels)."""
    monkeypatch.setenv("DIRIGO_JIT", "1")
    monkeypatch.setenv("DIRIGO_DAG_JIT", "1")
    texts = []
    for seed in range(1000, 1016):
        try:
            B.dg_graph_parse(fuzz_graphs.random_graph(seed))
            texts.append(fuzz_graphs.random_graph(seed))
        except B.DgError:
            pass
    # (compiled several at once, kept loaded)
    warm = gpu_warm.warm_graphs(B, texts, threads=16) + gpu_warm.warm_dags(B, texts, threads=16)  # noqa: F841
    done = sum(check_graph(B, seed, dags=True) for seed in range(1000, 1016))
    assert done >= 15
