"""Whole-workload parity against the oracle, element by element, through the
C ABI, in the launch configuration the benchmark times (specialised kernels,
single pass):

- every row of the two output-bound workloads: all 65,536 locations of the
  GEMM + GroupNorm graph (4,366,401,536 entries) and all 65,536 sampled
  locations of the conv-transpose + softmax graph (about 1.03e9 entries);
- the conv2d pair check: the clean split-K variant and every one of its 16
  faults, statuses at 32,768 random positions plus every position at the
  output's padding edge, and all 1,048,576 positions for two faults;
- the streamed and range calls over the whole output of the conv2d + pool
  graph, against the oracle (not against the library's other calls).

The long comparisons are split into slices, one test each.  The oracle runs
one chunk ahead of the comparison on up to 16 host threads; each chunk's GPU
rows are copied to the host and compared with numpy.
"""

import concurrent.futures as cf
import os

import numpy as np
import pytest
import torch

import gpu_warm
import oracle
from paper_2609_19611_amd import workloads as W

pytestmark = pytest.mark.gpu

THREADS = max(1, min(16, os.cpu_count() or 1))


@pytest.fixture(scope="module")
def B():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_19611_amd import binding
    return binding


def _u32(t):
    return t.cpu().numpy().view(np.uint32)


def single_pass(B, g, locs, total):
    """dg_enumerate over a location list into buffers of exactly `total`
    entries (the benchmarked call)."""
    d_locs = torch.as_tensor(np.asarray(locs, dtype=np.int64), device="cuda")
    n = d_locs.numel()
    ws = B.workspace(g, n)
    off = torch.full((n + 1,), -1, dtype=torch.int64, device="cuda")
    ids = torch.empty(max(1, total), dtype=torch.int32, device="cuda")
    cnt = torch.empty(max(1, total), dtype=torch.int32, device="cuda")
    assert B.dg_enumerate(g, d_locs, off, ids, cnt, ws) == total
    return off, ids, cnt


def first_bad_row(got_off, got_ids, got_cnt, ro, io, co):
    """Index (within a chunk) of the first row that differs."""
    for i in range(len(ro) - 1):
        a, b = got_off[i], got_off[i + 1]
        if b - a != ro[i + 1] - ro[i]:
            return i
        if not (np.array_equal(got_ids[a:b], io[ro[i]:ro[i + 1]]) and
                np.array_equal(got_cnt[a:b], co[ro[i]:ro[i + 1]])):
            return i
    return None


def check_every_row(text, locs, off, ids, cnt, chunk):
    """Every row of (off, ids, cnt) against the oracle's rows of the same
    locations, `chunk` locations at a time.  Returns the number of entries
    compared."""
    og = oracle.Graph(text)
    off_h = off.cpu().numpy()
    n = len(locs)
    assert off_h[0] == 0
    bounds = list(range(0, n, chunk)) + [n]
    compared = 0
    with cf.ThreadPoolExecutor(1) as ex:
        fut = ex.submit(og.enumerate, locs[bounds[0]:bounds[1]], THREADS)
        for k in range(len(bounds) - 1):
            a, b = bounds[k], bounds[k + 1]
            ro, io, co = fut.result()
            if k + 2 < len(bounds):
                fut = ex.submit(og.enumerate, locs[b:bounds[k + 2]], THREADS)
            lo, hi = int(off_h[a]), int(off_h[b])
            got_off = off_h[a:b + 1] - lo
            gi, gc = _u32(ids[lo:hi]), _u32(cnt[lo:hi])
            if not (np.array_equal(got_off, ro) and np.array_equal(gi, io) and np.array_equal(gc, co)):
                i = first_bad_row(got_off, gi, gc, ro, io, co)
                pytest.fail(f"row {a + i} (location {locs[a + i]}) differs from the oracle" if i is not None
                            else f"chunk [{a}, {b}) differs from the oracle")
            compared += hi - lo
    return compared


# The long comparisons run as slices (one test each), so that every test
# finishes, and reports, within a minute or two.
C4_SLICES = 4
C3_SLICES = 16


@pytest.fixture(scope="module")
def c4_rows(B):
    """All 65,536 rows of the GEMM + bias -> GroupNorm -> hardtanh ->
    residual graph (66,626 entries each) by the single-pass call."""
    text = W.c4_text()
    locs = W.config_locations("c4")
    off, ids, cnt = single_pass(B, B.dg_graph_parse(text), locs, 4366401536)
    yield text, locs, off, ids, cnt
    del off, ids, cnt
    torch.cuda.empty_cache()


@pytest.mark.parametrize("part", range(C4_SLICES))
def test_c4_every_row_against_oracle(c4_rows, part):
    text, locs, off, ids, cnt = c4_rows
    n = len(locs)
    a, b = part * n // C4_SLICES, (part + 1) * n // C4_SLICES
    sub = off[a:b + 1]
    assert check_every_row(text, locs[a:b], sub - sub[0], ids[int(sub[0]):int(sub[-1])],
                           cnt[int(sub[0]):int(sub[-1])], chunk=1024) == 66626 * (b - a)


@pytest.fixture(scope="module")
def c3_rows(B):
    """All 65,536 sampled rows of the conv_transpose3d -> mean -> softmax
    graph (rows of 7,232 to 28,736 entries) by the single-pass call."""
    text = W.c3_text()
    locs = W.config_locations("c3")
    g = B.dg_graph_parse(text)
    d_locs = torch.as_tensor(np.asarray(locs, dtype=np.int64), device="cuda")
    ws = B.workspace(g, len(locs))
    off = torch.empty(len(locs) + 1, dtype=torch.int64, device="cuda")
    total = B.dg_enumerate_sizes(g, d_locs, off, ws)
    del d_locs, ws
    off, ids, cnt = single_pass(B, g, locs, total)
    yield text, locs, off, ids, cnt
    del off, ids, cnt
    torch.cuda.empty_cache()


@pytest.mark.parametrize("part", range(C3_SLICES))
def test_c3_every_row_against_oracle(c3_rows, part):
    text, locs, off, ids, cnt = c3_rows
    n = len(locs)
    a, b = part * n // C3_SLICES, (part + 1) * n // C3_SLICES
    sub = off[a:b + 1]
    lo, hi = int(sub[0]), int(sub[-1])
    assert check_every_row(text, locs[a:b], sub - lo, ids[lo:hi], cnt[lo:hi], chunk=1024) == hi - lo


def padding_edge_positions(locs, H=64, Wd=64):
    """Positions into `locs` whose location lies on the first or last row or
    column of its image (where the conv's padding drops taps)."""
    la = np.asarray(locs, dtype=np.int64)
    h, w = (la // Wd) % H, la % Wd
    return np.nonzero((h == 0) | (h == H - 1) | (w == 0) | (w == Wd - 1))[0]


@pytest.fixture(scope="module")
def c5_setup(B):
    ref_text = W.c5_reference_text()
    locs = np.asarray(W.config_locations("c5"), dtype=np.int64)
    rng = np.random.default_rng(505)
    sample = np.union1d(rng.choice(len(locs), 32768, replace=False), padding_edge_positions(locs))
    assert len(sample) > 32768 + 40000
    ref = B.dg_graph_parse(ref_text)
    variants = [B.dg_graph_parse(W.c5_variant_text(fault=f)) for f in C5_VARIANTS]
    gpu_warm.warm_pairs(B, [(ref, v) for v in variants])  # compile the 17 pair kernels several at once
    return ref, oracle.Graph(ref_text), locs, torch.as_tensor(locs, device="cuda"), sample, variants


C5_VARIANTS = [None] + W.c5_faults()
C5_FULL = {2, 3}  # fault indices compared at all positions: a stride fault and an offset fault


@pytest.mark.parametrize("k", range(len(C5_VARIANTS)))
def test_c5_statuses_against_oracle(B, c5_setup, k):
    """The pair check at its 1,048,576 locations, for the clean variant and
    each fault: statuses against the oracle at 32,768 random positions plus
    every padding-edge position (all positions for two faults); the mismatch
    list equals the nonzero statuses."""
    ref, og_ref, locs, d_locs, sample, variants = c5_setup
    f = C5_VARIANTS[k]
    vt = W.c5_variant_text(fault=f)
    st, mism = B.compare_locations(ref, variants[k], d_locs)
    st = st.cpu().numpy()
    assert np.array_equal(mism.cpu().numpy(), np.nonzero(st)[0]), f
    pos = np.arange(len(locs)) if (k - 1) in C5_FULL else sample
    want = oracle.compare(og_ref, oracle.Graph(vt), locs[pos], threads=THREADS)
    bad = np.nonzero(st[pos] != want)[0]
    assert len(bad) == 0, (f, int(pos[bad[0]]), int(locs[pos[bad[0]]]), int(st[pos[bad[0]]]), int(want[bad[0]]))
    if f is None:
        assert not st.any()
    else:
        assert st.any(), f


def test_split_k_fault_with_budget_against_oracle(B):
    """The whole 33,554,432-location output of one fault with a budget of
    one mismatch: every reported mismatch and a sample of the locations
    compared equal agree with the oracle."""
    ref_text = W.c5_reference_text()
    f = W.c5_faults()[0]
    vt = W.c5_variant_text(fault=f)
    ref, bad = B.dg_graph_parse(ref_text), B.dg_graph_parse(vt)
    numel = 64 * 128 * 64 * 64
    ws = B.workspace(ref, numel)
    status = torch.empty(numel, dtype=torch.uint8, device="cuda")
    mism = torch.empty(numel, dtype=torch.int64, device="cuda")
    k = B.dg_compare_range(ref, bad, 0, numel, status, mism, ws, max_mismatch=1)
    assert k >= 1
    reported = mism[:k].cpu().numpy()
    st = status.cpu().numpy()
    assert np.array_equal(reported, np.nonzero((st == 1) | (st == 2))[0])
    rng = np.random.default_rng(7)
    checked = reported if k <= 8192 else np.sort(rng.choice(reported, 8192, replace=False))
    equal = np.nonzero(st == 0)[0]
    if len(equal) > 8192:
        equal = np.sort(rng.choice(equal, 8192, replace=False))
    og_ref, og_bad = oracle.Graph(ref_text), oracle.Graph(vt)
    for pos in (checked, equal):
        if len(pos):
            want = oracle.compare(og_ref, og_bad, pos, threads=THREADS)
            assert np.array_equal(st[pos], want)


def test_stream_whole_output_against_oracle(B):
    """dg_enumerate_stream over every one of the 65,536 output locations of
    the conv2d -> bias -> gelu -> maxpool graph, through two halves of a
    small buffer: every chunk's rows equal the oracle's."""
    text = W.c2_text()
    g = B.dg_graph_parse(text)
    numel = 16 * 16 * 16 * 16
    ro, io, co = oracle.Graph(text).enumerate(np.arange(numel), threads=THREADS)
    buf = torch.empty(3 * (1 << 20), dtype=torch.uint8, device="cuda")
    chunks = []

    def consume(first, o, i, c, stream):
        chunks.append((first, o.cpu().numpy().copy(), _u32(i).copy(), _u32(c).copy()))

    B.dg_enumerate_stream(g, 0, numel, buf, 8192, consume)
    assert len(chunks) > 4
    pos = 0
    for first, o, i, c in chunks:
        assert first == pos
        m = len(o) - 1
        base = int(ro[pos])
        assert np.array_equal(o, ro[pos:pos + m + 1] - base)
        assert np.array_equal(i, io[base:base + int(o[-1])]) and np.array_equal(c, co[base:base + int(o[-1])])
        pos += m
    assert pos == numel


def test_range_whole_output_against_oracle(B):
    """dg_enumerate_range over the whole output of the conv2d + pool graph
    in two ranges, against the oracle."""
    text = W.c2_text()
    g = B.dg_graph_parse(text)
    numel = 16 * 16 * 16 * 16
    ro, io, co = oracle.Graph(text).enumerate(np.arange(numel), threads=THREADS)
    for first, n in ((0, 40000), (40000, numel - 40000)):
        ws = B.workspace(g, n)
        off = torch.empty(n + 1, dtype=torch.int64, device="cuda")
        total = int(ro[first + n] - ro[first])
        ids = torch.empty(total, dtype=torch.int32, device="cuda")
        cnt = torch.empty_like(ids)
        assert B.dg_enumerate_range(g, first, n, off, ids, cnt, ws) == total
        assert np.array_equal(off.cpu().numpy(), ro[first:first + n + 1] - ro[first])
        a, b = int(ro[first]), int(ro[first + n])
        assert np.array_equal(_u32(ids), io[a:b]) and np.array_equal(_u32(cnt), co[a:b])


def test_paper_example_rows_against_oracle(B):
    """The worked example's two programs at l = 11,596 and at the first and
    last output locations: rows element by element and statuses."""
    locs = [11596, 0, 128 * 16 * 64 - 1]
    for text in (W.paper_kernel_text(), W.paper_reference_text()):
        off, ids, cnt = B.enumerate_locations(B.dg_graph_parse(text), locs)
        ro, io, co = oracle.Graph(text).enumerate(locs)
        assert np.array_equal(off.cpu().numpy(), ro)
        assert np.array_equal(_u32(ids), io) and np.array_equal(_u32(cnt), co)
