"""GPU parity of the location order's device part (dg_order_permute)
against the oracle's keyed permutation, element by element through the C
ABI: whole permutations, ranges with ragged tails over several tiles,
excluded values, edge cases; and the full order of the c5 variant's
33,554,432 output locations as a permutation led by the prefix."""

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


def _permute(B, n, seed, first, count, exclude=None):
    dev = torch.device("cuda", 0)
    ex = list(exclude or [])
    out = torch.full((max(1, count),), -1, dtype=torch.int64, device=dev)
    ws = torch.empty(max(1, B.dg_order_workspace_size(len(ex))), dtype=torch.uint8, device=dev)
    w = B.dg_order_permute(n, seed, ex, first, count, out, ws)
    return out[:w].cpu().numpy()


@pytest.mark.parametrize("n", [1, 2, 3, 5, 17, 1000, 2048, 2049, 4097, 65537, 1048576])
def test_whole_permutation(B, n):
    assert np.array_equal(_permute(B, n, 12345, 0, n), oracle.permutation(n, 12345))


@pytest.mark.parametrize("first,count", [(0, 1), (5, 2047), (2047, 2), (1000, 6000), (99_000, 1000), (0, 0)])
def test_ranges(B, first, count):
    n = 100_000
    assert np.array_equal(_permute(B, n, 7, first, count), oracle.permutation(n, 7, first, count))


def test_excluded_values(B):
    n = 20_000
    rng = np.random.default_rng(3)
    ex = rng.integers(0, n, 300).tolist()  # unsorted, with repeats
    want = oracle.permutation(n, 11)
    want = want[~np.isin(want, ex)]
    assert np.array_equal(_permute(B, n, 11, 0, n, ex), want)
    # A range: the kept values of that range of positions, in order.
    part = oracle.permutation(n, 11, 4000, 5000)
    assert np.array_equal(_permute(B, n, 11, 4000, 5000, ex), part[~np.isin(part, ex)])
    # Every value excluded: nothing written.
    assert len(_permute(B, 50, 1, 0, 50, list(range(50)))) == 0


def test_large_n_samples(B):
    # n near 2^40 (h = 20): a range of positions against the oracle.
    n = (1 << 40) - 12345
    assert np.array_equal(_permute(B, n, 5, n - 5000, 5000), oracle.permutation(n, 5, n - 5000, 5000))


@pytest.mark.parametrize("name,threads,warp", [("c5v-small", 16, 4), ("c4", 256, 32), ("c2", 64, 32)])
def test_order_locations_small(B, name, threads, warp):
    text = W.c5_variant_text(n=1, c=4, hw=5, co=3) if name == "c5v-small" else W.CONFIGS[name]["text"]()
    got = B.order_locations(B.dg_graph_parse(text), 9, threads, warp).cpu().numpy()
    want = oracle.location_order(oracle.Graph(text), 9, threads, warp)
    assert np.array_equal(got, want)


def test_order_locations_c5_variant_full(B):
    g = B.dg_graph_parse(W.c5_variant_text())
    n = B.dg_graph_info(g)["output_numel"]
    order = B.order_locations(g, 5)
    prefix = B.dg_order_prefix(g)
    assert order.numel() == n == 33_554_432
    assert order[: len(prefix)].cpu().tolist() == prefix
    s, _ = torch.sort(order)
    assert torch.equal(s, torch.arange(n, dtype=torch.int64, device=order.device))
    # Sampled permutation positions against the oracle: the rest of the
    # order is the permutation with the prefix's values left out.
    perm = oracle.permutation(n, 5, 0, 200_000)
    perm = perm[~np.isin(perm, prefix)]
    k = len(prefix)
    assert np.array_equal(order[k: k + len(perm)].cpu().numpy(), perm)


@pytest.mark.parametrize("kind", W.C5_SPARSE_FAULTS)
def test_sparse_fault_found_first_by_the_order(B, kind):
    """A sparse fault of the c5 split-K variant (split 0 reads a shifted row
    at the last output row only, or a shifted column at the last output
    column only): the GPU comparison over all 33,554,432 output locations
    mismatches exactly at those locations (for the column fault, not at the
    first row: split 0 reads only kernel row 0, which lies in the padding
    there), the oracle agrees there and on a sample of the rest (their
    neighbours included), and the location order reaches a mismatch within
    its prefix, no later than the plain permutation or sequential order."""
    dev = torch.device("cuda", 0)
    ref_t, var_t = W.c5_reference_text(), W.c5_variant_text(fault=kind)
    ref, var = B.dg_graph_parse(ref_t), B.dg_graph_parse(var_t)
    N, C, H, Wd = 64, 128, 64, 64
    n = N * C * H * Wd
    status = torch.empty(n, dtype=torch.uint8, device=dev)
    mism = torch.empty(n, dtype=torch.int64, device=dev)
    ws = torch.empty(max(B.dg_workspace_size(ref, n), B.dg_workspace_size(var, n)), dtype=torch.uint8, device=dev)
    k = B.dg_compare_range(ref, var, 0, n, status, mism, ws)
    st = status.cpu().numpy()
    h = (np.arange(n) // Wd) % H
    w = np.arange(n) % Wd
    want = (h == H - 1) if kind == "last-row" else (w == Wd - 1) & (h >= 1)
    assert np.array_equal(st != 0, want) and k == int(want.sum())
    rng = np.random.default_rng(7)
    hit = np.nonzero(want)[0]
    near = np.nonzero(((h == H - 2) | (h == 0) | (w == Wd - 2) | (w == Wd - 1)) & ~want)[0]
    sample = np.unique(np.concatenate([rng.choice(hit, min(len(hit), 4096), replace=False),
                                       rng.choice(near, 2048, replace=False),
                                       rng.integers(0, n, 4096)]))
    o = oracle.compare(oracle.Graph(ref_t), oracle.Graph(var_t), sample.tolist(), threads=16)
    assert np.array_equal(o, st[sample])

    def first(order):
        pos = np.nonzero(want[order])[0]
        return int(pos[0])
    heur = B.order_locations(var, 5).cpu().numpy()
    perm = _permute(B, n, 5, 0, n)  # the plain permutation (its parity is tested above)
    r_h, r_p, r_s = first(heur), first(perm), first(np.arange(n))
    assert r_h < len(B.dg_order_prefix(var)) and r_h <= r_p and r_h <= r_s, (r_h, r_p, r_s)
