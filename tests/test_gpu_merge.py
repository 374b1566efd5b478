"""GPU comparisons of merged programs (dg_graph_merge, then dg_compare)
against the oracle's comparison of its own merge: the paper's running
example as whole programs at full size (trimmed: every location mismatches,
the kernel's row lacks the rows h >= 32 of M; untrimmed: a sample), and
small pairs at every location, with and without trimming."""

import numpy as np
import pytest
import torch

import oracle
from paper_2609_19611_amd import workloads as W

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def B():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_19611_amd import binding
    return binding


def _gpu_status(B, a, b, locs):
    st, _ = B.compare_locations(a, b, locs)
    return st.cpu().numpy()


def test_paper_programs_full_size(B):
    a, b = W.paper_program_text(False), W.paper_program_text(True)
    ta, tb, k = B.dg_graph_merge(B.dg_graph_parse(a), B.dg_graph_parse(b), True)
    assert k == 1
    n = B.dg_graph_info(ta)["output_numel"]
    st = _gpu_status(B, ta, tb, list(range(n)))
    assert (st == 1).all()
    oa, ob, _ = oracle.merge(oracle.Graph(a), oracle.Graph(b), True)
    sample = list(range(0, n, 2053)) + [11596, n - 1]
    assert np.array_equal(st[sample], oracle.compare(oracle.Graph(oa), oracle.Graph(ob), sample, threads=8))
    ua, ub, k0 = B.dg_graph_merge(B.dg_graph_parse(a), B.dg_graph_parse(b), False)
    assert k0 == 0
    sample = list(range(0, n, 8191)) + [11596]
    oua, oub, _ = oracle.merge(oracle.Graph(a), oracle.Graph(b), False)
    assert np.array_equal(_gpu_status(B, ua, ub, sample),
                          oracle.compare(oracle.Graph(oua), oracle.Graph(oub), sample, threads=8))


@pytest.mark.parametrize("h_limit", [2, 4])
@pytest.mark.parametrize("trim", [True, False])
def test_small_pairs_every_location(B, h_limit, trim):
    a = W.paper_program_text(False, N=2, Cin=2, C=3, H=4, W=2)
    b = W.paper_program_text(True, N=2, Cin=2, C=3, H=4, W=2, h_limit=h_limit)
    ta, tb, _ = B.dg_graph_merge(B.dg_graph_parse(a), B.dg_graph_parse(b), trim)
    oa, ob, _ = oracle.merge(oracle.Graph(a), oracle.Graph(b), trim)
    n = oracle.Graph(oa).output_numel
    want = oracle.compare(oracle.Graph(oa), oracle.Graph(ob), list(range(n)))
    assert np.array_equal(_gpu_status(B, ta, tb, list(range(n))), want)
    assert (want == 0).all() == (h_limit == 4)
