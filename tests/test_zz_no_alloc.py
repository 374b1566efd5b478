"""dg_enumerate_noalloc (no device allocation, library-owned scratch)
against dg_enumerate, through the C ABI: two calls in a row on the same
graph, the second with fewer locations, then a call on another graph; the
error paths (a graph not yet resident on the device, too many locations).
Runs alone in a fresh process as well as after the other tests."""

import numpy as np
import pytest
import torch

from paper_2609_19611_amd import workloads as W

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def B():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_19611_amd import binding
    return binding


def _reference(B, g, d_locs):
    """dg_enumerate with a caller workspace: offsets, ids, counts."""
    n = d_locs.numel()
    ws = B.workspace(g, n)
    off = torch.empty(n + 1, dtype=torch.int64, device="cuda")
    none = torch.empty(0, dtype=torch.int32, device="cuda")
    try:
        total = B.dg_enumerate(g, d_locs, off, none, none, ws)
    except B.DgError as e:
        assert e.name == "DG_E_BUFFER"
        total = int(off[-1])
    ids = torch.empty(max(1, total), dtype=torch.int32, device="cuda")
    cnt = torch.empty_like(ids)
    assert B.dg_enumerate(g, d_locs, off, ids, cnt, ws) == total
    return off, ids[:total], cnt[:total]


def _noalloc(B, g, d_locs, total):
    n = d_locs.numel()
    off = torch.full((n + 1,), -3, dtype=torch.int64, device="cuda")
    ids = torch.full((max(1, total),), -3, dtype=torch.int32, device="cuda")
    cnt = torch.full((max(1, total),), -3, dtype=torch.int32, device="cuda")
    assert B.dg_enumerate_noalloc(g, d_locs, off, ids, cnt) == total
    return off, ids[:total], cnt[:total]


def test_noalloc_equals_enumerate_on_two_calls(B):
    g = B.dg_graph_parse(W.c3_text())
    locs = torch.as_tensor(W.config_locations("c3"), dtype=torch.int64, device="cuda")
    big, small = locs[:20000], locs[30000:33000]
    # The graph becomes resident through the ordinary call.
    want_big = _reference(B, g, big)
    want_small = _reference(B, g, small)
    got_big = _noalloc(B, g, big, int(want_big[0][-1]))
    got_small = _noalloc(B, g, small, int(want_small[0][-1]))
    for got, want in ((got_big, want_big), (got_small, want_small)):
        for x, y in zip(got, want):
            assert torch.equal(x, y)


def test_noalloc_other_graph_and_edges(B):
    g = B.dg_graph_parse(W.c2_text())
    locs = torch.as_tensor(W.config_locations("c2"), dtype=torch.int64, device="cuda")
    want = _reference(B, g, locs)
    got = _noalloc(B, g, locs, int(want[0][-1]))
    for x, y in zip(got, want):
        assert torch.equal(x, y)
    # n = 0
    off = torch.full((1,), 9, dtype=torch.int64, device="cuda")
    assert B.dg_enumerate_noalloc(g, locs[:0], off, want[1], want[2]) == 0 and int(off[0]) == 0
    # a location outside the output
    bad = torch.as_tensor([0, 65536], dtype=torch.int64, device="cuda")
    with pytest.raises(B.DgError) as e:
        B.dg_enumerate_noalloc(g, bad, torch.empty(3, dtype=torch.int64, device="cuda"), want[1], want[2])
    assert e.value.name == "DG_E_RANGE"
    # too many locations for the scratch
    many = torch.zeros(B.NOALLOC_MAX_LOCATIONS + 1, dtype=torch.int64, device="cuda")
    with pytest.raises(B.DgError) as e:
        B.dg_enumerate_noalloc(g, many, torch.empty(many.numel() + 1, dtype=torch.int64, device="cuda"),
                               want[1], want[2])
    assert e.value.name == "DG_E_WORKSPACE"


def test_noalloc_needs_a_resident_graph(B):
    g = B.dg_graph_parse(W.c1_text())
    locs = torch.arange(8, dtype=torch.int64, device="cuda")
    off = torch.empty(9, dtype=torch.int64, device="cuda")
    ids = torch.empty(1152, dtype=torch.int32, device="cuda")
    cnt = torch.empty_like(ids)
    with pytest.raises(B.DgError) as e:
        B.dg_enumerate_noalloc(g, locs, off, ids, cnt)
    assert e.value.name == "DG_E_INVALID_ARG" and ("resident" in str(e.value) or "loaded" in str(e.value))
    want = _reference(B, g, locs)
    assert B.dg_enumerate_noalloc(g, locs, off, ids, cnt) == 1152
    assert torch.equal(off, want[0]) and torch.equal(ids, want[1]) and torch.equal(cnt, want[2])
