"""GPU parity: the HIP library against the CPU oracle, bit for bit.

Every call goes through the C ABI (paper_2609_19611_amd.binding).  Small
graphs are compared at every output location; the five workloads run at
their full sizes in the same launch configuration the benchmark times, with
sampled rows checked against the oracle and closed-form properties checked
at every location.
"""

import numpy as np
import pytest
import torch

import gpu_warm
import oracle
import tiny_graphs
from paper_2609_19611_amd import workloads as W

pytestmark = pytest.mark.gpu

CAT = tiny_graphs.catalogue()
SEPARABLE = sorted(CAT)


@pytest.fixture(scope="module")
def B():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_19611_amd import binding
    # Compile the specialised kernels of every catalogue graph and of the
    # comparison pairs below ahead, several at once (the handles keep them
    # loaded for the module).
    global _WARM
    ref = binding.dg_graph_parse(W.c5_reference_text())
    small = binding.dg_graph_parse(W.c5_reference_text(n=2, c=4, hw=6, co=3))
    pairs = [(ref, binding.dg_graph_parse(W.c5_variant_text(fault=f))) for f in W.c5_faults()]
    pairs += [(small, binding.dg_graph_parse(W.c5_variant_text(fault=f, n=2, c=4, hw=6, co=3))) for f in W.c5_faults()]
    _WARM = (gpu_warm.warm_graphs(binding, [CAT[n][0] for n in SEPARABLE]), gpu_warm.warm_pairs(binding, pairs))
    return binding


def rows_to_host(off, ids, cnt, positions):
    """Rows at the given positions: (lengths, ids, counts) as numpy, taken
    slice by slice on the device."""
    off_h = off.cpu().numpy()
    out = []
    for p in positions:
        a, b = int(off_h[p]), int(off_h[p + 1])
        out.append((ids[a:b].cpu().numpy().view(np.uint32), cnt[a:b].cpu().numpy().view(np.uint32)))
    return off_h, out


def oracle_rows(text, locs, threads=8):
    off, ids, cnt = oracle.Graph(text).enumerate(locs, threads=threads)
    return [(ids[off[i]:off[i + 1]], cnt[off[i]:off[i + 1]]) for i in range(len(locs))]


def check_rows_sorted(off, ids):
    """Within every row ids strictly increase (checked on the device)."""
    if ids.numel() < 2:
        return
    chunk = 1 << 28
    starts = torch.zeros(ids.numel(), dtype=torch.bool, device=ids.device)
    inner = off[1:-1]
    starts[inner[inner < ids.numel()]] = True
    for a in range(1, ids.numel(), chunk):
        b = min(ids.numel(), a + chunk)
        cur = ids[a:b].to(torch.int64) & 0xFFFFFFFF
        prev = ids[a - 1:b - 1].to(torch.int64) & 0xFFFFFFFF
        assert bool(((cur > prev) | starts[a:b]).all())


@pytest.mark.parametrize("name", SEPARABLE)
@pytest.mark.parametrize("kernels", ["specialized", "interpreted"])
def test_catalogue_all_locations(B, name, kernels, monkeypatch):
    monkeypatch.setenv("DIRIGO_JIT", "1" if kernels == "specialized" else "0")
    text = CAT[name][0]
    g = B.dg_graph_parse(text)
    og = oracle.Graph(text)
    locs = list(range(og.output_numel))
    off, ids, cnt = B.enumerate_locations(g, locs)
    ro, io, co = og.enumerate(locs)
    assert np.array_equal(off.cpu().numpy(), ro)
    assert np.array_equal(ids.cpu().numpy().view(np.uint32), io)
    assert np.array_equal(cnt.cpu().numpy().view(np.uint32), co)


def test_specialized_kernels_load(B, monkeypatch):
    """With specialisation on (the default), a graph's first device call
    compiles and loads its own kernels; with DIRIGO_JIT=0 it never does."""
    monkeypatch.delenv("DIRIGO_JIT", raising=False)
    g = B.dg_graph_parse(W.c2_text())
    assert B.dg_graph_info(g)["specialized"] == -1
    B.enumerate_locations(g, [0, 1, 2])
    assert B.dg_graph_info(g)["specialized"] == 1
    monkeypatch.setenv("DIRIGO_JIT", "0")
    assert B.dg_graph_info(B.dg_graph_parse(W.c1_text()))["specialized"] == 0


def test_c1_all(B):
    text = W.c1_text()
    off, ids, cnt = B.enumerate_locations(B.dg_graph_parse(text), W.config_locations("c1"))
    ro, io, co = oracle.Graph(text).enumerate(range(8))
    assert np.array_equal(off.cpu().numpy(), ro)
    assert np.array_equal(ids.cpu().numpy().view(np.uint32), io)
    assert np.array_equal(cnt.cpu().numpy().view(np.uint32), co)


def test_c2_all_4096(B):
    text = W.c2_text()
    locs = W.config_locations("c2")
    off, ids, cnt = B.enumerate_locations(B.dg_graph_parse(text), locs)
    ro, io, co = oracle.Graph(text).enumerate(locs, threads=8)
    assert np.array_equal(off.cpu().numpy(), ro)
    assert np.array_equal(ids.cpu().numpy().view(np.uint32), io)
    assert np.array_equal(cnt.cpu().numpy().view(np.uint32), co)


def test_c3_full(B):
    text = W.c3_text()
    locs = W.config_locations("c3")
    off, ids, cnt = B.enumerate_locations(B.dg_graph_parse(text), locs)
    la = np.asarray(locs)
    d, h = (la // 4096) % 32, (la // 64) % 64
    td = np.where((d % 2 == 1) & (d <= 29), 2, 1)
    th = np.where((h % 2 == 1) & (h <= 61), 2, 1)
    off_h = off.cpu().numpy()
    assert np.array_equal(np.diff(off_h), 7168 * td * th + 64)
    check_rows_sorted(off, ids)
    rng = np.random.default_rng(3)
    pos = sorted(set(rng.choice(len(locs), 24, replace=False).tolist()) | {0, len(locs) - 1})
    _, got = rows_to_host(off, ids, cnt, pos)
    want = oracle_rows(text, [locs[p] for p in pos])
    for (gi, gc), (wi, wc) in zip(got, want):
        assert np.array_equal(gi, wi) and np.array_equal(gc, wc)


def test_c4_full(B):
    text = W.c4_text()
    locs = W.config_locations("c4")
    off, ids, cnt = B.enumerate_locations(B.dg_graph_parse(text), locs)
    off_h = off.cpu().numpy()
    assert np.all(np.diff(off_h) == 66626)
    assert off_h[-1] == 4366401536
    rng = np.random.default_rng(4)
    pos = sorted(set(rng.choice(len(locs), 6, replace=False).tolist()) | {0, len(locs) - 1})
    _, got = rows_to_host(off, ids, cnt, pos)
    want = oracle_rows(text, [locs[p] for p in pos])
    for (gi, gc), (wi, wc) in zip(got, want):
        assert np.array_equal(gi, wi) and np.array_equal(gc, wc)
    # Counts take only the closed-form values.
    vals = torch.unique(cnt[: 66626 * 64])
    assert set(vals.cpu().tolist()) == {1, 66, 67, 4225, 4226}


def test_c5_faults_at_boundaries(B):
    """Every fault of the split-K variant against the oracle at the output's
    padding edges (first and last two rows and columns, corner images and
    channels) and at 1,024 more locations drawn over the whole output."""
    ref_text = W.c5_reference_text()
    ref = B.dg_graph_parse(ref_text)
    N, C, H, Wd = 64, 128, 64, 64
    edge = [((n * C + c) * H + h) * Wd + w for n in (0, N - 1) for c in (0, C - 1)
            for h in (0, 1, H - 2, H - 1) for w in (0, 1, Wd - 2, Wd - 1)]
    rng = np.random.default_rng(55)
    locs = edge + sorted(rng.choice(N * C * H * Wd, 1024, replace=False).tolist())
    og_ref = oracle.Graph(ref_text)
    for f in W.c5_faults():
        vt = W.c5_variant_text(fault=f)
        st, mism = B.compare_locations(ref, B.dg_graph_parse(vt), locs)
        want = oracle.compare(og_ref, oracle.Graph(vt), locs, threads=8)
        assert np.array_equal(st.cpu().numpy(), want), f
        assert np.array_equal(mism.cpu().numpy(), np.nonzero(want)[0]), f


def test_paper_example(B):
    a = B.dg_graph_parse(W.paper_kernel_text())
    b = B.dg_graph_parse(W.paper_reference_text())
    status, mism = B.compare_locations(a, b, [11596, 0])
    assert status.cpu().tolist() == [1, 1] and mism.cpu().tolist() == [0, 1]
    off_a, _, _ = B.enumerate_locations(a, [11596])
    off_b, _, _ = B.enumerate_locations(b, [11596])
    assert int(off_a[1]) == 513 and int(off_b[1]) == 1025


@pytest.mark.parametrize("kernels", ["specialized", "interpreted"])
def test_compare_small_graphs_against_oracle(B, kernels, monkeypatch):
    monkeypatch.setenv("DIRIGO_JIT", "1" if kernels == "specialized" else "0")
    ref = W.c5_reference_text(n=2, c=4, hw=6, co=3)
    locs = list(range(2 * 3 * 6 * 6))
    g_ref, o_ref = B.dg_graph_parse(ref), oracle.Graph(ref)
    for f in W.c5_faults():
        vt = W.c5_variant_text(fault=f, n=2, c=4, hw=6, co=3)
        st, _ = B.compare_locations(g_ref, B.dg_graph_parse(vt), locs)
        assert np.array_equal(st.cpu().numpy(), oracle.compare(o_ref, oracle.Graph(vt), locs)), f
    a = CAT["self_product"][0]
    b = tiny_graphs._g([("x", [3, 2]), ("w", [2])], [("a", "add", ["x", "x"], {}), ("y", "mul", ["a", "w"], {})],
                       "y", [3, 2])
    st, _ = B.compare_locations(B.dg_graph_parse(a), B.dg_graph_parse(b), range(6))
    assert st.cpu().tolist() == [2] * 6


@pytest.mark.parametrize("kernels", ["specialized", "interpreted"])
def test_compare_pairs_viewed_with_different_merged_dims(B, kernels, monkeypatch):
    """Pairs where one graph reads a leaf through merged dims (a reshape)
    and the other does not: compared over the joined view, both orders,
    against the oracle."""
    monkeypatch.setenv("DIRIGO_JIT", "1" if kernels == "specialized" else "0")
    for name, a, b in tiny_graphs.merged_view_pairs():
        n = oracle.Graph(a).output_numel
        want = oracle.compare(oracle.Graph(a), oracle.Graph(b), range(n))
        for x, y in ((a, b), (b, a)):
            st, mism = B.compare_locations(B.dg_graph_parse(x), B.dg_graph_parse(y), list(range(n)))
            assert np.array_equal(st.cpu().numpy(), want), name
            assert np.array_equal(mism.cpu().numpy(), np.nonzero(want)[0]), name


@pytest.mark.parametrize("kernels", ["specialized", "interpreted"])
def test_factored_comparison_of_single_term_leaves(B, kernels, monkeypatch):
    monkeypatch.setenv("DIRIGO_JIT", "1" if kernels == "specialized" else "0")
    for name, a, b, _ in tiny_graphs.factored_compare_pairs():
        n = oracle.Graph(a).output_numel
        want = oracle.compare(oracle.Graph(a), oracle.Graph(b), range(n))
        for x, y in ((a, b), (b, a)):
            st, mism = B.compare_locations(B.dg_graph_parse(x), B.dg_graph_parse(y), list(range(n)))
            assert np.array_equal(st.cpu().numpy(), want), name
            assert np.array_equal(mism.cpu().numpy(), np.nonzero(want)[0]), name


def test_edge_cases(B):
    g = B.dg_graph_parse(W.c2_text())
    off, ids, cnt = B.enumerate_locations(g, torch.empty(0, dtype=torch.int64))
    assert off.cpu().tolist() == [0] and ids.numel() == 0
    locs = [65535, 3, 3, 40000, 0, 3]
    off, ids, cnt = B.enumerate_locations(g, locs)
    ro, io, co = oracle.Graph(W.c2_text()).enumerate(locs)
    assert np.array_equal(off.cpu().numpy(), ro)
    assert np.array_equal(ids.cpu().numpy().view(np.uint32), io)
    with pytest.raises(B.DgError) as e:
        B.enumerate_locations(g, [0, 65536])
    assert e.value.name == "DG_E_RANGE"
    with pytest.raises(B.DgError) as e:
        B.enumerate_locations(g, [-1])
    assert e.value.name == "DG_E_RANGE"
    # Path counts past 32 bits (the 64-bit call handles them).
    with pytest.raises(B.DgError) as e:
        B.enumerate_locations(B.dg_graph_parse(tiny_graphs.nested_layer_norms(2048)), [0])
    assert e.value.name == "DG_E_OVERFLOW"
    # More LDS than one block can have.
    with pytest.raises(B.DgError) as e:
        B.enumerate_locations(B.dg_graph_parse(tiny_graphs.nested_layer_norms(4096)), [0])
    assert e.value.name == "DG_E_CAPACITY"
    with pytest.raises(B.DgError) as e:
        B.compare_locations(g, B.dg_graph_parse(W.c1_text()), [0])
    assert e.value.name == "DG_E_SIGNATURE"
    # Comparisons: no locations; an output that is a leaf against an op of
    # it (same footprint) and against x + x (same footprint, counts 2).
    st, mm = B.compare_locations(g, g, torch.empty(0, dtype=torch.int64))
    assert st.numel() == 0 and mm.numel() == 0
    leaf = B.dg_graph_parse("dgir 1\nleaf x 4\noutput x 4\n")
    relu = B.dg_graph_parse("dgir 1\nleaf x 4\nop y relu x\noutput y 4\n")
    twice = B.dg_graph_parse("dgir 1\nleaf x 4\nop y add x x\noutput y 4\n")
    st, mm = B.compare_locations(leaf, relu, [0, 1, 2, 3])
    assert st.cpu().tolist() == [0] * 4 and mm.numel() == 0
    st, mm = B.compare_locations(relu, twice, [3, 0])
    assert st.cpu().tolist() == [2, 2] and mm.cpu().tolist() == [0, 1]


@pytest.mark.parametrize("shape", [[1, 6, 12], [2, 6, 12]])
@pytest.mark.parametrize("kernels", ["specialized", "interpreted"])
def test_compare_counts_near_2_32(B, shape, kernels, monkeypatch):
    """32-bit comparison arithmetic under static bounds just below 2^32
    (counts up to 2,101,864,255), at every location, against the oracle,
    with the specialised and the precompiled comparison kernels."""
    monkeypatch.setenv("DIRIGO_JIT", "1" if kernels == "specialized" else "0")
    a = tiny_graphs.large_count_norms(shape)
    ga = B.dg_graph_parse(a)
    n = B.dg_graph_info(ga)["output_numel"]
    assert B.dg_graph_info(ga)["count_bound"] < 2 ** 32
    for v in ("permuted", "mid_1d"):
        b = tiny_graphs.large_count_norms(shape, v)
        st, _ = B.compare_locations(ga, B.dg_graph_parse(b), list(range(n)))
        want = oracle.compare(oracle.Graph(a), oracle.Graph(b), range(n))
        assert np.array_equal(st.cpu().numpy(), want)


def test_repeatable(B):
    g = B.dg_graph_parse(W.c3_text())
    locs = W.config_locations("c3")[:2048]
    a = B.enumerate_locations(g, locs)
    b = B.enumerate_locations(g, locs)
    for x, y in zip(a, b):
        assert torch.equal(x, y)


def _fused(B, g, locs):
    d_locs = torch.as_tensor(locs, dtype=torch.int64, device="cuda")
    n = d_locs.numel()
    ws = B.workspace(g, n)
    off = torch.empty(n + 1, dtype=torch.int64, device="cuda")
    total = B.dg_enumerate_sizes(g, d_locs, off, ws)
    ids = torch.empty(max(total, 1), dtype=torch.int32, device="cuda")
    cnt = torch.empty(max(total, 1), dtype=torch.int32, device="cuda")
    off2 = torch.full((n + 1,), -7, dtype=torch.int64, device="cuda")
    t2 = B.dg_enumerate(g, d_locs, off2, ids, cnt, ws)
    assert t2 == total and torch.equal(off, off2)
    return off2, ids[:total], cnt[:total]


@pytest.mark.parametrize("name", ["c1", "c2", "c3"])
def test_single_pass_equals_two_pass(B, name):
    text = W.CONFIGS[name]["text"]()
    g = B.dg_graph_parse(text)
    locs = W.config_locations(name)
    a = B.enumerate_locations(g, locs)
    b = _fused(B, g, locs)
    for x, y in zip(a, b):
        assert torch.equal(x, y)


def test_single_pass_c4_against_oracle(B):
    text = W.c4_text()
    g = B.dg_graph_parse(text)
    locs = W.config_locations("c4")
    off, ids, cnt = _fused(B, g, locs)
    assert int(off[-1]) == 4366401536
    assert bool((off[1:] - off[:-1] == 66626).all())
    pos = [0, 1, 31337, len(locs) - 1]
    _, got = rows_to_host(off, ids, cnt, pos)
    want = oracle_rows(text, [locs[p] for p in pos])
    for (gi, gc), (wi, wc) in zip(got, want):
        assert np.array_equal(gi, wi) and np.array_equal(gc, wc)


@pytest.mark.parametrize("name", ["c5_small_var", "conv3d_groups", "gather_floor_flat", "diamond"])
@pytest.mark.parametrize("kernels", ["specialized", "interpreted"])
def test_single_pass_catalogue(B, name, kernels, monkeypatch):
    monkeypatch.setenv("DIRIGO_JIT", "1" if kernels == "specialized" else "0")
    text = CAT[name][0]
    og = oracle.Graph(text)
    locs = list(range(og.output_numel))[::-1]  # descending order, still one row per location
    off, ids, cnt = _fused(B, B.dg_graph_parse(text), locs)
    ro, io, co = og.enumerate(locs)
    assert np.array_equal(off.cpu().numpy(), ro)
    assert np.array_equal(ids.cpu().numpy().view(np.uint32), io)
    assert np.array_equal(cnt.cpu().numpy().view(np.uint32), co)


def test_single_pass_small_buffer(B):
    text = W.c2_text()
    g = B.dg_graph_parse(text)
    locs = W.config_locations("c2")[:300]
    d_locs = torch.as_tensor(locs, dtype=torch.int64, device="cuda")
    ws = B.workspace(g, len(locs))
    off = torch.empty(len(locs) + 1, dtype=torch.int64, device="cuda")
    ro, io, co = oracle.Graph(text).enumerate(locs)
    cap = int(ro[150])  # room for exactly the first 150 rows
    guard = 4096
    ids = torch.full((cap + guard,), -1, dtype=torch.int32, device="cuda")
    cnt = torch.full((cap + guard,), -1, dtype=torch.int32, device="cuda")
    with pytest.raises(B.DgError) as e:
        B.dg_enumerate(g, d_locs, off, ids[:cap], cnt[:cap], ws)
    assert e.value.name == "DG_E_BUFFER"
    assert np.array_equal(off.cpu().numpy(), ro)
    assert np.array_equal(ids[:cap].cpu().numpy().view(np.uint32), io[:cap])
    assert bool((ids[cap:] == -1).all()) and bool((cnt[cap:] == -1).all())
    # n = 0
    off0 = torch.full((1,), 5, dtype=torch.int64, device="cuda")
    assert B.dg_enumerate(g, d_locs[:0], off0, ids, cnt, ws) == 0 and int(off0[0]) == 0


@pytest.mark.parametrize("K", [4096, 6144])
@pytest.mark.parametrize("kernels", ["specialized", "interpreted"])
def test_large_lds_graphs(B, K, kernels, monkeypatch):
    """Graphs whose location needs more than 64 KB of LDS (a long
    contraction): both kernel kinds launch with the larger allocation."""
    monkeypatch.setenv("DIRIGO_JIT", "1" if kernels == "specialized" else "0")
    text = tiny_graphs._g([("x", [2, K]), ("W", [K, 3])], [("y", "matmul", ["x", "W"], {})], "y", [2, 3])
    g = B.dg_graph_parse(text)
    assert B.dg_graph_info(g)["lds_bytes"] > 65536
    locs = list(range(6))
    off, ids, cnt = B.enumerate_locations(g, locs)
    ro, io, co = oracle.Graph(text).enumerate(locs)
    assert np.array_equal(off.cpu().numpy(), ro)
    assert np.array_equal(ids.cpu().numpy().view(np.uint32), io)
    assert np.array_equal(cnt.cpu().numpy().view(np.uint32), co)
    off2, ids2, cnt2 = _fused(B, g, locs)
    assert torch.equal(off, off2) and torch.equal(ids, ids2) and torch.equal(cnt, cnt2)


def test_lds_beyond_the_device_is_rejected(B):
    text = tiny_graphs._g([("x", [2, 8192]), ("W", [8192, 3])], [("y", "matmul", ["x", "W"], {})], "y", [2, 3])
    g = B.dg_graph_parse(text)
    assert B.dg_graph_info(g)["lds_bytes"] > 160 * 1024
    with pytest.raises(B.DgError) as e:
        B.enumerate_locations(g, [0])
    assert e.value.name == "DG_E_CAPACITY"


def test_range_enumeration_equals_list(B):
    text = W.c2_text()
    g = B.dg_graph_parse(text)
    first, n = 1000, 3000
    a = B.enumerate_locations(g, list(range(first, first + n)))
    ws = B.workspace(g, n)
    off = torch.empty(n + 1, dtype=torch.int64, device="cuda")
    ids = torch.empty(int(a[0][-1]), dtype=torch.int32, device="cuda")
    cnt = torch.empty_like(ids)
    total = B.dg_enumerate_range(g, first, n, off, ids, cnt, ws)
    assert total == int(a[0][-1])
    assert torch.equal(off, a[0]) and torch.equal(ids, a[1]) and torch.equal(cnt, a[2])
    # the whole output of the GEMM + GroupNorm graph, by range
    g4 = B.dg_graph_parse(W.c4_text())
    n4 = 128 * 512
    ws4 = B.workspace(g4, n4)
    off4 = torch.empty(n4 + 1, dtype=torch.int64, device="cuda")
    ids4 = torch.empty(4366401536, dtype=torch.int32, device="cuda")
    cnt4 = torch.empty_like(ids4)
    assert B.dg_enumerate_range(g4, 0, n4, off4, ids4, cnt4, ws4) == 4366401536
    assert bool((off4[1:] - off4[:-1] == 66626).all())
    pos = [0, 777, n4 - 1]
    _, got = rows_to_host(off4, ids4, cnt4, pos)
    want = oracle_rows(W.c4_text(), pos)
    for (gi, gc), (wi, wc) in zip(got, want):
        assert np.array_equal(gi, wi) and np.array_equal(gc, wc)
    del ids4, cnt4


def test_range_compare_and_mismatch_limit(B):
    ref_text = W.c5_reference_text(n=2, c=4, hw=6, co=3)
    ref = B.dg_graph_parse(ref_text)
    numel = 2 * 3 * 6 * 6
    ws = B.workspace(ref, numel)
    status = torch.empty(numel, dtype=torch.uint8, device="cuda")
    mism = torch.empty(numel, dtype=torch.int64, device="cuda")
    og_ref = oracle.Graph(ref_text)
    for f in W.c5_faults()[:8]:
        vt = W.c5_variant_text(fault=f, n=2, c=4, hw=6, co=3)
        var = B.dg_graph_parse(vt)
        want = oracle.compare(og_ref, oracle.Graph(vt), list(range(numel)))
        k = B.dg_compare_range(ref, var, 0, numel, status, mism, ws)
        st = status.cpu().numpy()
        assert np.array_equal(st, want), f
        assert np.array_equal(mism[:k].cpu().numpy(), np.nonzero(want)[0])
        # a sub-range reports positions relative to its first location
        k = B.dg_compare_range(ref, var, 50, 100, status, mism, ws)
        assert np.array_equal(status[:100].cpu().numpy(), want[50:150])
        assert np.array_equal(mism[:k].cpu().numpy(), np.nonzero(want[50:150])[0])
        # with a budget: every reported status is right, skipped ones are 3
        nbad = int((want != 0).sum())
        for limit in (1, 5):
            k = B.dg_compare_range(ref, var, 0, numel, status, mism, ws, max_mismatch=limit)
            st = status.cpu().numpy()
            done = st != 3
            assert np.array_equal(st[done], want[done]), (f, limit)
            assert int(((st == 1) | (st == 2)).sum()) >= min(limit, nbad)
            assert np.array_equal(mism[:k].cpu().numpy(), np.nonzero((st == 1) | (st == 2))[0])
            if nbad == 0:
                assert not (st == 3).any()


def test_full_output_verification_of_the_split_k_variant(B):
    """Every one of the 33,554,432 output locations of the conv2d pair: the
    clean split-K NHWC variant is footprint-equivalent to the reference."""
    ref = B.dg_graph_parse(W.c5_reference_text())
    var = B.dg_graph_parse(W.c5_variant_text())
    numel = 64 * 128 * 64 * 64
    ws = B.workspace(ref, numel)
    status = torch.empty(numel, dtype=torch.uint8, device="cuda")
    mism = torch.empty(numel, dtype=torch.int64, device="cuda")
    assert B.dg_compare_range(ref, var, 0, numel, status, mism, ws) == 0
    assert int(status.max()) == 0
    # a faulty variant stops early under a budget of one mismatch
    bad = B.dg_graph_parse(W.c5_variant_text(fault=W.c5_faults()[0]))
    k = B.dg_compare_range(ref, bad, 0, numel, status, mism, ws, max_mismatch=1)
    assert k >= 1
    first = int(mism[0])
    want = oracle.compare(oracle.Graph(W.c5_reference_text()), oracle.Graph(W.c5_variant_text(fault=W.c5_faults()[0])),
                          [first])
    assert want[0] == int(status[first]) != 0


def test_streamed_enumeration_matches_one_pass(B):
    """A whole output streamed through two small buffer halves (chunks cut
    where the rows stop fitting) gives the one-pass CSR, chunk by chunk."""
    text = W.c2_text()
    g = B.dg_graph_parse(text)
    numel = 16 * 16 * 16 * 16
    ws = B.workspace(g, numel)
    off = torch.empty(numel + 1, dtype=torch.int64, device="cuda")
    ids = torch.empty(numel * 80, dtype=torch.int32, device="cuda")
    cnt = torch.empty_like(ids)
    total = B.dg_enumerate_range(g, 0, numel, off, ids, cnt, ws)
    want_off = off.cpu().numpy()
    want_ids = ids[:total].cpu().numpy()
    want_cnt = cnt[:total].cpu().numpy()
    buf = torch.empty(2 * (1 << 20), dtype=torch.uint8, device="cuda")
    chunks = []

    def consume(first, o, i, c, stream):
        # (.cpu() on the current stream, which is the chunk's)
        chunks.append((first, o.cpu().numpy().copy(), i.cpu().numpy().copy(), c.cpu().numpy().copy()))

    B.dg_enumerate_stream(g, 0, numel, buf, 8192, consume)
    assert len(chunks) > 8
    pos = 0
    for first, o, i, c in chunks:
        assert first == pos
        m = len(o) - 1
        base = want_off[pos]
        assert np.array_equal(o, want_off[pos:pos + m + 1] - base)
        assert np.array_equal(i, want_ids[base:base + o[-1]]) and np.array_equal(c, want_cnt[base:base + o[-1]])
        pos += m
    assert pos == numel
    # a consumer can stop the stream
    seen = []
    with pytest.raises(B.DgError) as e:
        B.dg_enumerate_stream(g, 0, numel, buf, 4096, lambda *a: seen.append(1) or len(seen) == 2)
    assert e.value.name == "DG_E_STOPPED" and len(seen) == 2
    # halves of 64 entries: the first row (56 entries, a corner) fits, the
    # second (65) does not
    got = []
    def up(x):
        return (x + 255) & ~255

    used = up(8 * 9) + up(B.dg_workspace_size(g, 8))
    half = up(8 * 5) + up(B.dg_workspace_size(g, 4)) + 64 * 8  # room for 64 entries
    small = torch.empty(used + 2 * half, dtype=torch.uint8, device="cuda")
    with pytest.raises(B.DgError) as e:
        B.dg_enumerate_stream(g, 0, 8, small, 4, lambda first, o, i, c, s: got.append((first, int(o[-1]))))
    assert e.value.name == "DG_E_BUFFER"
    assert got == [(0, int(want_off[1]))]


def _wide(B, g, locs):
    """dg_enumerate_wide in two calls: the first, with no room for rows,
    gives the offsets (DG_E_BUFFER unless every row is empty)."""
    d_locs = torch.as_tensor(locs, dtype=torch.int64, device="cuda")
    n = d_locs.numel()
    ws = B.workspace(g, n)
    off = torch.full((n + 1,), -7, dtype=torch.int64, device="cuda")
    none = torch.empty(0, dtype=torch.int64, device="cuda")
    try:
        total = B.dg_enumerate_wide(g, d_locs, off, none, none, ws)
    except B.DgError as e:
        assert e.name == "DG_E_BUFFER"
        total = int(off[-1])
    ids = torch.full((max(total, 1),), -1, dtype=torch.int64, device="cuda")
    cnt = torch.full((max(total, 1),), -1, dtype=torch.int64, device="cuda")
    off2 = torch.full((n + 1,), -7, dtype=torch.int64, device="cuda")
    assert B.dg_enumerate_wide(g, d_locs, off2, ids, cnt, ws) == total
    assert torch.equal(off, off2)
    return off2, ids[:total], cnt[:total]


def _u64(t):
    return t.cpu().numpy().view(np.uint64)


@pytest.mark.parametrize("name", ["c5_small_var", "conv3d_groups", "gather_floor_flat", "diamond", "paper_kernel_small"])
@pytest.mark.parametrize("kernels", ["specialized", "interpreted"])
def test_wide_catalogue(B, name, kernels, monkeypatch):
    monkeypatch.setenv("DIRIGO_JIT", "1" if kernels == "specialized" else "0")
    text = CAT[name][0]
    og = oracle.Graph(text)
    locs = list(range(og.output_numel))[::-1]
    off, ids, cnt = _wide(B, B.dg_graph_parse(text), locs)
    ro, io, co = og.enumerate(locs, wide=True)
    assert np.array_equal(off.cpu().numpy(), ro)
    assert np.array_equal(_u64(ids), io) and np.array_equal(_u64(cnt), co)


@pytest.mark.parametrize("name,step", [("c1", 1), ("c2", 1), ("c3", 5), ("c4", 97)])
def test_wide_equals_narrow_on_workloads(B, name, step):
    g = B.dg_graph_parse(W.CONFIGS[name]["text"]())
    locs = W.config_locations(name)[::step]
    a = _fused(B, g, locs)
    b = _wide(B, g, locs)
    assert torch.equal(a[0], b[0])
    for x, y in zip(a[1:], b[1:]):
        assert torch.equal(x.to(torch.int64) & 0xFFFFFFFF, y)


@pytest.mark.parametrize("kernels", ["specialized", "interpreted"])
def test_wide_counts_past_32_bits(B, kernels, monkeypatch):
    """Three nested layer norms over 2048 elements: counts near 3.6e16.
    The 32-bit call reports DG_E_OVERFLOW; the 64-bit one matches the
    closed form and the oracle."""
    monkeypatch.setenv("DIRIGO_JIT", "1" if kernels == "specialized" else "0")
    n = 2048
    text = tiny_graphs.nested_layer_norms(n)
    g = B.dg_graph_parse(text)
    locs = [0, 1, 1000, n - 1]
    d_locs = torch.as_tensor(locs, dtype=torch.int64, device="cuda")
    ws = B.workspace(g, len(locs))
    off = torch.empty(len(locs) + 1, dtype=torch.int64, device="cuda")
    ids = torch.empty(len(locs) * n, dtype=torch.int32, device="cuda")
    cnt = torch.empty(len(locs) * n, dtype=torch.int32, device="cuda")
    with pytest.raises(B.DgError) as e:
        B.dg_enumerate(g, d_locs, off, ids, cnt, ws)
    assert e.value.name == "DG_E_OVERFLOW"
    off, ids, cnt = _wide(B, g, locs)
    assert off.cpu().tolist() == [i * n for i in range(len(locs) + 1)]
    ids_h, cnt_h = _u64(ids), _u64(cnt)
    for i, l in enumerate(locs):
        assert ids_h[i * n:(i + 1) * n].tolist() == list(range(n))
        assert cnt_h[i * n:(i + 1) * n].tolist() == tiny_graphs.nested_layer_norm_counts(n, l)
    ro, io, co = oracle.Graph(text).enumerate(locs, threads=4, wide=True)
    assert np.array_equal(ids_h, io) and np.array_equal(cnt_h, co)


def test_wide_ids_past_2_32(B):
    """Leaves holding more than 2^32 elements: ids past 2^32, 32-bit calls
    refuse the graph before any device work."""
    # Row sums of a 2^20 x 4096 leaf declared after a 4096-element one: the
    # last rows' ids cross 2^32.
    R, K = 1 << 20, 4096
    text = f"dgir 1\nleaf p {K}\nleaf a {R},{K}\nop y sum a ; dims=1 keepdim=0\noutput y {R}\n"
    g = B.dg_graph_parse(text)
    assert B.dg_graph_info(g)["leaf_total"] == K + 2 ** 32
    locs = [0, 12345, R - 2, R - 1]
    d_locs = torch.as_tensor(locs, dtype=torch.int64, device="cuda")
    ws = B.workspace(g, len(locs))
    off = torch.empty(len(locs) + 1, dtype=torch.int64, device="cuda")
    buf = torch.empty(len(locs) * K, dtype=torch.int32, device="cuda")
    with pytest.raises(B.DgError) as e:
        B.dg_enumerate(g, d_locs, off, buf, buf, ws)
    assert e.value.name == "DG_E_OVERFLOW"
    off, ids, cnt = _wide(B, g, locs)
    ids_h = _u64(ids)
    for i, l in enumerate(locs):
        want = K + l * K + np.arange(K, dtype=np.uint64)
        assert np.array_equal(ids_h[i * K:(i + 1) * K], want)
    assert bool((cnt == 1).all())
    assert int(ids_h.max()) > 2 ** 32
    ro, io, co = oracle.Graph(text).enumerate(locs, threads=4, wide=True)
    assert np.array_equal(off.cpu().numpy(), ro) and np.array_equal(ids_h, io) and np.array_equal(_u64(cnt), co)
