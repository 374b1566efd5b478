"""Compiles graphs' specialised kernels ahead of the GPU tests, many at
once: each graph (or pair) compiles on first use, and doing that for dozens
of graphs one after another would dominate the tests' run time.  The
returned handles keep the loaded kernels alive for the caller's scope."""

import concurrent.futures as cf
import sys
import time


def warm_graphs(B, texts, threads=8):
    """Parses each text and runs one location through it (which compiles
    and loads its specialised kernels); returns the graph handles."""
    def one(text):
        g = B.dg_graph_parse(text)
        B.enumerate_locations(g, [0])
        return g
    t0 = time.time()
    with cf.ThreadPoolExecutor(threads) as ex:
        out = list(ex.map(one, texts))
    print(f"[warm] {len(texts)} graphs in {time.time() - t0:.1f} s", file=sys.stderr, flush=True)
    return out


def warm_pairs(B, pairs, threads=8):
    """The same for comparisons: (graph a, graph b) handles, one location each."""
    def one(p):
        B.compare_locations(p[0], p[1], [0])
        return p
    t0 = time.time()
    with cf.ThreadPoolExecutor(threads) as ex:
        out = list(ex.map(one, pairs))
    print(f"[warm] {len(pairs)} pairs in {time.time() - t0:.1f} s", file=sys.stderr, flush=True)
    return out


def warm_dags(B, texts, threads=8):
    """The same for expression DAGs: parses each text and takes one
    location's DAG (which compiles and loads its DAG kernels, specialised
    when DIRIGO_DAG_JIT=1); returns the graph handles."""
    def one(text):
        g = B.dg_graph_parse(text)
        B.dag_locations(g, [0])
        return g
    t0 = time.time()
    with cf.ThreadPoolExecutor(threads) as ex:
        out = list(ex.map(one, texts))
    print(f"[warm] {len(texts)} DAG programs in {time.time() - t0:.1f} s", file=sys.stderr, flush=True)
    return out
