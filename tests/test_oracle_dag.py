"""Pins of the oracle's expression DAG of res(y[l]) (Sec. 3.4,
"Back-projection"), independent of its read loops:

* Value: every DAG node, evaluated bottom-up from its ordered element
  references with the op's own arithmetic (a conv node is the sum of the
  products of its consecutive (x, W) references plus its bias reference, a
  norm node standardises its element by the statistics references, ...),
  equals the element PyTorch computes for that tensor in float64 (random
  leaves).  A wrong pairing, a wrong order of operands, a missing or an extra
  reference changes the value.
* Path counts: summing products of multiplicities over the DAG's paths from
  y[l] to each leaf element gives the enumeration's row (pinned elsewhere by
  autograd of the linearised graph).
* Shape: nodes are the distinct non-leaf cone elements, ops in reverse SSA
  order and elements ascending; every node but y[l] is referenced by another.
"""

from __future__ import annotations

import math

import numpy as np
import pytest
import torch

import oracle
import tiny_graphs
import torch_eval
from paper_2609_19611_amd import workloads as W

CAT = tiny_graphs.catalogue()
EPS = 1e-5  # PyTorch's default eps of the normalisations


def _program(text):
    leaves, ops, out = torch_eval.parse(text)
    return leaves, ops, out


def _tensor_table(g: oracle.Graph):
    """[(gid base, numel, tensor index)] sorted by base, for id lookups."""
    tab = sorted((g.gid(t), g.tensors[t].numel, t) for t in range(len(g.tensors)))
    return tab


def _locate(tab, gid):
    lo, hi = 0, len(tab)
    while hi - lo > 1:
        mid = (lo + hi) // 2
        if tab[mid][0] <= gid:
            lo = mid
        else:
            hi = mid
    base, n, t = tab[lo]
    assert base <= gid < base + n, gid
    return t, gid - base


def _node_value(kind, attrs, vals, mults, n_in):
    """One node's value from its ordered references (values and
    multiplicities), by the op's arithmetic."""
    v = vals
    if kind in torch_eval._UNARY:
        return torch_eval._UNARY[kind](torch.tensor(v[0], dtype=torch.float64)).item()
    if kind in torch_eval._BINARY:
        return torch_eval._BINARY[kind](torch.tensor(v[0], dtype=torch.float64),
                                        torch.tensor(v[1], dtype=torch.float64)).item()
    if kind in ("matmul", "linear", "conv", "conv_transpose"):
        bias = (kind != "matmul") and n_in == 3
        body = v[:-1] if bias else v
        assert len(body) % 2 == 0
        acc = sum(body[2 * i] * body[2 * i + 1] for i in range(len(body) // 2))
        return acc + (v[-1] if bias else 0.0)
    if kind == "max_pool":
        return max(v)
    if kind == "avg_pool":
        return sum(v) / len(v)
    if kind == "sum":
        return sum(v)
    if kind == "mean":
        return sum(v) / len(v)
    if kind in ("amax", "max"):
        return max(v)
    if kind in ("amin", "min"):
        return min(v)
    if kind == "prod":
        return math.prod(v)
    if kind in ("softmax", "log_softmax"):
        sl, xl = v[:-1], v[-1]
        m = max(sl)
        lse = m + math.log(sum(math.exp(a - m) for a in sl))
        return math.exp(xl - lse) if kind == "softmax" else xl - lse
    if kind in ("group_norm", "batch_norm", "layer_norm"):
        aff = n_in == 3
        stats = v[:-3] if aff else v[:-1]
        xl = v[-3] if aff else v[-1]
        S = len(stats)
        assert all(m == S + 2 for m in mults[:S])
        mu = sum(stats) / S
        var = sum((a - mu) ** 2 for a in stats) / S
        y = (xl - mu) / math.sqrt(var + EPS)
        return y * v[-2] + v[-1] if aff else y
    if kind == "channel_affine":
        return v[0] * v[1] + v[2]
    if kind in ("slice", "permute", "reshape", "expand"):
        return v[0]
    if kind == "affine_gather":
        m = [int(x) for x in attrs.get("mult", ["1"] * n_in)]
        assert len(v) % n_in == 0
        acc = 0.0
        for p in range(len(v) // n_in):
            term = 1.0
            for j in range(n_in):
                assert mults[p * n_in + j] == m[j]
                term *= v[p * n_in + j] ** m[j]
            acc += term
        return acc
    raise NotImplementedError(kind)


def _check_dag(text, locs, seed=0):
    g = oracle.Graph(text)
    d = g.dag(locs)
    leaves, ops, out = _program(text)
    gen = torch.Generator().manual_seed(seed)
    leaf_vals = {n: torch.randn(s, dtype=torch.float64, generator=gen) for n, s in leaves}
    env = torch_eval.evaluate_all(text, leaf_vals)
    names = [t.name for t in g.tensors]
    op_of = {name: (kind, attrs, len(operands)) for name, kind, operands, attrs in ops}
    tab = _tensor_table(g)
    op_rank = {name: i for i, (name, _, _, _) in enumerate(ops)}
    rows = g.enumerate(locs, wide=True)
    for i, loc in enumerate(locs):
        n0, n1 = d["node_offsets"][i], d["node_offsets"][i + 1]
        e0, e1 = d["edge_offsets"][i], d["edge_offsets"][i + 1]
        nodes = [int(x) for x in d["nodes"][n0:n1]]
        starts = [int(x) for x in d["node_edge"][n0:n1]] + [int(e1 - e0)]
        edges = [int(x) for x in d["edges"][e0:e1]]
        mults = [int(x) for x in d["mults"][e0:e1]]
        assert len(set(nodes)) == len(nodes)
        # Order: ops in reverse SSA order, elements ascending.
        keys = [(-op_rank[names[_locate(tab, nd)[0]]], _locate(tab, nd)[1]) for nd in nodes]
        assert keys == sorted(keys)
        if nodes:
            assert _locate(tab, nodes[0]) == (g.output, loc)
        # Every referenced non-leaf element is a node; every node but the
        # root is referenced.
        node_set = set(nodes)
        referenced = set()
        for e in edges:
            t, _ = _locate(tab, e)
            if g.tensors[t].leaf_index < 0:
                assert e in node_set
                referenced.add(e)
        assert referenced == node_set - {nodes[0]} if nodes else not referenced
        # Values, bottom-up (reverse of the node order).
        value = {}

        def val(gid):
            if gid in value:
                return value[gid]
            t, idx = _locate(tab, gid)
            assert g.tensors[t].leaf_index >= 0
            return leaf_vals[names[t]].reshape(-1)[idx].item()

        for k in range(len(nodes) - 1, -1, -1):
            t, idx = _locate(tab, nodes[k])
            kind, attrs, n_in = op_of[names[t]]
            es = edges[starts[k]:starts[k + 1]]
            ms = mults[starts[k]:starts[k + 1]]
            if kind in ("conv", "conv_transpose"):
                # Canonical order: input channel, then taps row-major, so the
                # weight references ascend.
                wref = es[1:len(es) - (n_in == 3):2]
                assert all(a < b for a, b in zip(wref, wref[1:])), (names[t], idx)
            v = _node_value(kind, attrs, [val(e) for e in es], ms, n_in)
            want = env[names[t]].reshape(-1)[idx].item()
            assert v == pytest.approx(want, rel=1e-9, abs=1e-9), (names[t], idx, kind)
            value[nodes[k]] = v
        # Path counts over the DAG equal the row.
        paths = {nodes[0]: 1} if nodes else {}
        leaf_count = {}
        for k in range(len(nodes)):
            c = paths.get(nodes[k], 0)
            for e, m in zip(edges[starts[k]:starts[k + 1]], mults[starts[k]:starts[k + 1]]):
                t, _ = _locate(tab, e)
                if g.tensors[t].leaf_index >= 0:
                    leaf_count[e] = leaf_count.get(e, 0) + c * m
                else:
                    paths[e] = paths.get(e, 0) + c * m
        off, ids, cnt = rows
        want_row = dict(zip(ids[off[i]:off[i + 1]].tolist(), cnt[off[i]:off[i + 1]].tolist()))
        if nodes:
            assert leaf_count == want_row


@pytest.mark.parametrize("name", sorted(CAT))
def test_dag_values_and_paths(name):
    text = CAT[name][0]
    g = oracle.Graph(text)
    n = g.output_numel
    locs = list(range(n)) if n <= 64 else sorted(set(np.linspace(0, n - 1, 48).astype(int).tolist()))
    _check_dag(text, locs)


def test_dag_workloads_small():
    for name in ("c1", "c2"):
        locs = W.config_locations(name)[:16]
        _check_dag(W.CONFIGS[name]["text"](), locs)


def test_dag_c1_closed_form():
    """y = sum_j relu(A @ B)[i, j] over [8,16] @ [16,8]: y[i] reads the 8
    relu elements of row i; each reads its matmul element; each matmul
    element (i, j) reads A[i, k], B[k, j] for k = 0..15 in turn."""
    g = oracle.Graph(W.c1_text())
    gid = {t.name: g.gid(k) for k, t in enumerate(g.tensors)}
    i = 5
    d = g.dag([i])
    want_nodes = [gid["y"] + i] + [gid["R"] + 8 * i + j for j in range(8)] + [gid["C"] + 8 * i + j for j in range(8)]
    assert d["nodes"].tolist() == want_nodes
    edges = d["edges"].tolist()
    assert edges[:8] == [gid["R"] + 8 * i + j for j in range(8)]
    assert edges[8:16] == [gid["C"] + 8 * i + j for j in range(8)]
    for j in range(8):
        blk = edges[16 + 32 * j:16 + 32 * (j + 1)]
        assert blk == [x for k in range(16) for x in (gid["A"] + 16 * i + k, gid["B"] + 8 * k + j)]
    assert set(d["mults"].tolist()) == {1}


def test_dag_output_leaf_and_range():
    g = oracle.Graph("dgir 1\nleaf x 4\noutput x 4\n")
    d = g.dag([0, 3])
    assert d["node_offsets"].tolist() == [0, 0, 0] and d["edges"].size == 0
    with pytest.raises(oracle.OracleError):
        oracle.Graph(W.c1_text()).dag([8])
