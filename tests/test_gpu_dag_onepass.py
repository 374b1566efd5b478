"""GPU parity of dg_dag, the one-call expression DAGs (each location walked
once, its DAG staged in LDS and placed by decoupled look-backs, when it fits
in LDS; the two passes otherwise), against the oracle's DAGs, element by
element, through the C ABI: every location of the small catalogue graphs,
samples of the workloads (c4 takes the two passes), the specialised
kernels, short buffers, the default choice of path and edge cases.  The
one pass is forced at every size (DIRIGO_DAG_ONEPASS=1) except where the
default is tested."""

import os

import numpy as np
import pytest
import torch

import oracle
import tiny_graphs
from paper_2609_19611_amd import workloads as W

pytestmark = pytest.mark.gpu

KEYS = ("node_offsets", "edge_offsets", "nodes", "node_edge", "edges", "mults")
SLACK = 5  # entries past the totals that must stay untouched


@pytest.fixture(scope="module")
def B():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_19611_amd import binding
    return binding


@pytest.fixture(autouse=True)
def one_pass(monkeypatch):
    """The one pass at every size where its stage fits (by default it runs
    calls of at most 2,048 locations)."""
    monkeypatch.setenv("DIRIGO_DAG_ONEPASS", "1")


def _call(B, text, locs, node_cap, edge_cap):
    """dg_dag into buffers of the given capacities (filled with a sentinel
    first); returns the totals and the device tensors."""
    g = B.dg_graph_parse(text)
    d_locs = torch.as_tensor(locs, dtype=torch.int64).cuda()
    n = len(locs)
    ws = B.workspace(g, n)
    out = {"node_offsets": torch.full((n + 1,), -7, dtype=torch.int64, device="cuda"),
           "edge_offsets": torch.full((n + 1,), -7, dtype=torch.int64, device="cuda")}
    for k, m in (("nodes", node_cap), ("node_edge", node_cap), ("edges", edge_cap), ("mults", edge_cap)):
        out[k] = torch.full((m,), -1, dtype=torch.int32, device="cuda")
    tot = B.dg_dag(g, d_locs, out["node_offsets"], out["edge_offsets"], out["nodes"], out["node_edge"],
                   out["edges"], out["mults"], ws)
    return tot, out


def _host(t):
    a = t.cpu().numpy()
    return a if a.dtype == np.int64 else a.view(np.uint32).astype(np.uint64)


def _check(B, text, locs, threads=16):
    want = oracle.Graph(text).dag(locs, threads=threads)
    nn, ne = len(want["nodes"]), len(want["edges"])
    (gn, ge), out = _call(B, text, locs, nn + SLACK, ne + SLACK)
    assert (gn, ge) == (nn, ne)
    for k in KEYS:
        got = _host(out[k])
        m = len(want[k])
        assert np.array_equal(got[:m], want[k]), k
        assert (got[m:] == 0xFFFFFFFF).all(), k  # nothing written past the totals
    return out


CAT = {**{k: v[0] for k, v in tiny_graphs.catalogue().items()}, **tiny_graphs.dag_catalogue()}


@pytest.mark.parametrize("name", sorted(CAT))
def test_one_call_catalogue_all_locations(B, name):
    text = CAT[name]
    n = oracle.Graph(text).output_numel
    _check(B, text, list(range(n))[::-1])


@pytest.mark.parametrize("name,step", [("c1", 1), ("c2", 1), ("c4", 64), ("c5", 256)])
def test_one_call_workloads(B, name, step):
    locs = W.config_locations(name)[::step]
    _check(B, W.CONFIGS[name]["text"](), locs)


def test_one_call_c5_variants_and_faults(B):
    locs = W.config_locations("c5")[::4096]
    for text in [W.c5_variant_text()] + [W.c5_variant_text(fault=f) for f in W.c5_faults()]:
        _check(B, text, locs)


def test_one_call_specialised(B, monkeypatch):
    """The specialised one-pass kernel (DIRIGO_DAG_JIT=1): c5's reference
    and a catalogue graph with a point tail, against the oracle."""
    monkeypatch.setenv("DIRIGO_DAG_JIT", "1")
    _check(B, W.CONFIGS["c5"]["text"](), W.config_locations("c5")[::512])
    text = CAT["convT3d_bias_mean"]
    _check(B, text, list(range(oracle.Graph(text).output_numel)))
    g = B.dg_graph_parse(W.CONFIGS["c5"]["text"]())
    B.dag_locations(g, [0])
    assert B.dg_graph_info(g)["dag_specialized"] == 1


def test_one_call_short_buffers(B):
    """A total above its capacity: DG_E_BUFFER, the offsets as the oracle's,
    and the DAGs of the locations that fit written in place."""
    text = W.CONFIGS["c5"]["text"]()
    locs = W.config_locations("c5")[::8192]
    want = oracle.Graph(text).dag(locs, threads=16)
    nn, ne = len(want["nodes"]), len(want["edges"])
    last = int(want["edge_offsets"][-2])  # the last location's first edge
    with pytest.raises(B.DgError) as e:
        _call(B, text, locs, nn, ne - 1)
    assert e.value.name == "DG_E_BUFFER"
    g = B.dg_graph_parse(text)
    d_locs = torch.as_tensor(locs, dtype=torch.int64).cuda()
    ws = B.workspace(g, len(locs))
    noff = torch.empty(len(locs) + 1, dtype=torch.int64, device="cuda")
    eoff = torch.empty(len(locs) + 1, dtype=torch.int64, device="cuda")
    nodes = torch.full((nn,), -1, dtype=torch.int32, device="cuda")
    node_edge = torch.full((nn,), -1, dtype=torch.int32, device="cuda")
    edges = torch.full((ne - 1,), -1, dtype=torch.int32, device="cuda")
    mults = torch.full((ne - 1,), -1, dtype=torch.int32, device="cuda")
    with pytest.raises(B.DgError):
        B.dg_dag(g, d_locs, noff, eoff, nodes, node_edge, edges, mults, ws)
    assert np.array_equal(_host(noff), want["node_offsets"])
    assert np.array_equal(_host(eoff), want["edge_offsets"])
    assert np.array_equal(_host(nodes), want["nodes"])
    assert np.array_equal(_host(edges)[:last], want["edges"][:last])
    assert np.array_equal(_host(mults)[:last], want["mults"][:last])
    assert (_host(edges)[last:] == 0xFFFFFFFF).all()


def test_one_call_default_choice(B, monkeypatch):
    """Without DIRIGO_DAG_ONEPASS, a call of at most 2,048 locations takes
    the one pass and a larger one the two passes; both match the oracle."""
    monkeypatch.delenv("DIRIGO_DAG_ONEPASS")
    text = W.CONFIGS["c5"]["text"]()
    _check(B, text, W.config_locations("c5")[::512])      # 2,048 locations
    _check(B, text, W.config_locations("c5")[1::256])     # 4,096 locations


@pytest.mark.parametrize("chunk", range(2))
def test_one_call_fuzz(B, chunk):
    """Seeded random graphs (as the fuzz tests build them): every output
    location's DAG in one call, against the oracle."""
    import fuzz_graphs
    done = 0
    for seed in range(chunk * 20, (chunk + 1) * 20):
        text = fuzz_graphs.random_graph(seed)
        try:
            B.dg_graph_parse(text)
        except B.DgError:
            continue
        _check(B, text, list(range(oracle.Graph(text).output_numel))[::-1])
        done += 1
    assert done >= 15


def test_one_call_edge_cases(B):
    text = W.c2_text()
    (nn, ne), out = _call(B, text, [], 1, 1)
    assert (nn, ne) == (0, 0) and out["node_offsets"].cpu().tolist() == [0]
    _check(B, text, [65535, 3, 3, 0])
    with pytest.raises(B.DgError) as e:
        _call(B, text, [0, 65536], 64, 4096)
    assert e.value.name == "DG_E_RANGE"
    (nn, ne), out = _call(B, "dgir 1\nleaf x 4\noutput x 4\n", [0, 3], 1, 1)
    assert (nn, ne) == (0, 0) and out["edge_offsets"].cpu().tolist() == [0, 0, 0]
