"""Seeded random graphs over the whole op vocabulary (fuzz_graphs.py)
against the oracle, on the CPU: the library's compiler and block code (host
emulation, one thread per block) at every output location of each graph,
for rows, expression DAGs and comparisons with a variant whose counts
double; the static bounds hold.  A graph the library refuses must be one of
its documented refusals, and those stay rare."""

import numpy as np
import pytest

import fuzz_graphs
import hostemu
import oracle
from paper_2609_19611_amd import binding as B

from fuzz_graphs import REFUSALS, squared_variant

DAG_KEYS = ("node_offsets", "edge_offsets", "nodes", "node_edge", "edges", "mults")
CHUNK = 100


@pytest.mark.parametrize("chunk", range(8))
def test_fuzz_against_oracle(chunk):
    refused = 0
    for seed in range(chunk * CHUNK, (chunk + 1) * CHUNK):
        text = fuzz_graphs.random_graph(seed)
        og = oracle.Graph(text)
        locs = list(range(og.output_numel))
        try:
            got = hostemu.enumerate(text, locs)
        except hostemu.HostEmuError as e:
            assert e.code == -4 and any(r in str(e) for r in REFUSALS), (seed, str(e))
            refused += 1
            continue
        want = og.enumerate(locs, wide=False)
        for x, y in zip(got, want):
            assert np.array_equal(x, y), f"rows differ, seed {seed}"
        info = B.dg_graph_info(B.dg_graph_parse(text))
        wo, _, wc = og.enumerate(locs, wide=True)
        assert info["max_row_size"] >= int(np.diff(wo).max(initial=0)), seed
        assert info["count_bound"] >= int(wc.max(initial=0)), seed
        gd, wd = hostemu.dag(text, locs), og.dag(locs)
        for k in DAG_KEYS:
            assert np.array_equal(gd[k], wd[k]), f"DAG {k} differs, seed {seed}"
        var = squared_variant(text)
        st = hostemu.compare(text, var, locs)
        assert np.array_equal(st, oracle.compare(og, oracle.Graph(var), locs)), f"compare differs, seed {seed}"
    assert refused <= 3, refused
