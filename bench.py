"""Benchmark of batched backward dataflow enumeration on one MI355X.

One step is one pass of the enumeration hot path over the workload's
location list, with the locations already resident in device memory:
the sizes kernel (per-location plan + row sizes), the device-wide scan of
the offsets, and the fill kernel writing the CSR rows.  The default workload
is the GEMM -> GroupNorm -> Hardtanh -> residual graph with all 65,536
output locations enumerated (4,366,401,536 entries, 34.9 GB of rows per
step); --workload selects another configuration (c5 times the two-graph
comparator over the clean split-K variant and the 16 fault variants).

Prints one JSON line.  Values are synthetic and irrelevant: footprints are
data independent, so only shapes are used.
"""

from __future__ import annotations

import argparse
import json
import os
import subprocess
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

ALU_PEAK_TOPS = 256 * 4 * 16 * 2.4e9 / 1e12  # int32 VALU operations, no packing
# A comparison's per-entry work: the entry's id (one add of two table
# parts), its count (one product) and its share of the equality test.
COMPARE_OPS_PER_ENTRY = 3
HBM_PEAK_GBS = 8000.0  # MI355X HBM3E, published


def parse_args():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=10)
    p.add_argument("--warmup", type=int, default=3)
    p.add_argument("--workload", default="c4", choices=["c1", "c2", "c3", "c4", "c5"])
    p.add_argument("--cpu-seconds", type=float, default=15.0, help="target length of the oracle sample")
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--no-secondary", action="store_true",
                   help="skip the c3 enumeration and c5 comparison figures added to the default c4 line")
    p.add_argument("--two-pass", action="store_true",
                   help="time dg_enumerate_sizes + dg_enumerate_fill instead of the single-pass dg_enumerate")
    p.add_argument("--wide", action="store_true",
                   help="time dg_enumerate_wide (64-bit ids and counts) instead of dg_enumerate")
    p.add_argument("--merge", action="store_true",
                   help="time the comparison of the paper's two whole programs (shared convolution, reference "
                        "ops vs fused kernel) at every output location, after MERGE with and without trimming "
                        "the common prefix")
    p.add_argument("--order", action="store_true",
                   help="time the location order (keyed permutation of every output location of the c5 split-K "
                        "variant, corner and boundary prefix left out) and count the locations checked before "
                        "each fault's first mismatch under three orders")
    p.add_argument("--dag", action="store_true",
                   help="time expression-DAG emission (dg_dag_sizes + dg_dag_fill) instead of the rows; c3 takes "
                        "every 8th of its locations, c5 the reference graph")
    p.add_argument("--full-output", action="store_true",
                   help="every output location: c5 compares all 33,554,432 (dg_compare_range; the faulty variants "
                        "stop at their first mismatch); c1-c4 stream the whole output's rows through a bounded "
                        "buffer (dg_enumerate_stream) into a checksum consumer")
    p.add_argument("--stream-gib", type=float, default=16.0, help="buffer of the streamed full output (two halves)")
    p.add_argument("--copy-gib", type=float, default=0.0,
                   help="instead of the workload, time a plain device copy of this many GiB (HBM calibration)")
    p.add_argument("--write-sweep", action="store_true",
                   help="instead of the workload, time torch's fill (int32) over buffers of 0.5 to 32 GiB: the "
                        "plain write rate against the size written")
    return p.parse_args()


def write_rates(gib, steps, warmup):
    """Device-to-device copy and a write-only fill of a known size (torch's
    kernels): the HBM bandwidth this machine reaches, beside the spec peak."""
    import torch
    n = int(gib * (1 << 30)) // 4
    src = torch.ones(n, dtype=torch.int32, device="cuda")
    dst = torch.empty_like(src)

    def timed(fn):
        for _ in range(warmup):
            fn()
        ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(steps)]
        torch.cuda.synchronize()
        for a, b in ev:
            a.record()
            fn()
            b.record()
        torch.cuda.synchronize()
        return float(np.median([a.elapsed_time(b) for a, b in ev]))

    ms_copy = timed(lambda: dst.copy_(src))
    ms_fill = timed(lambda: dst.fill_(7))
    return {"bytes": n * 4, "copy_ms": ms_copy, "copy_GBps_read_plus_write": 2 * n * 4 / (ms_copy * 1e-3) / 1e9,
            "fill_ms": ms_fill, "fill_GBps_write": n * 4 / (ms_fill * 1e-3) / 1e9}


def copy_calibration(gib, steps, warmup):
    """The copy and fill of write_rates as a line of their own; their
    dispatches are the reference for scaling the FETCH_SIZE / WRITE_SIZE
    counters."""
    print(json.dumps(write_rates(gib, steps, warmup)), flush=True)


def write_sweep(steps, warmup):
    """Plain write rate against buffer size: torch's int32 fill over one
    buffer of each size (median of `steps` fills), one JSON line."""
    import torch
    stream = torch.cuda.current_stream()
    rows = []
    for gib in (0.5, 1, 2, 4, 8, 16, 32):
        n = int(gib * (1 << 30)) // 4
        buf = torch.empty(n, dtype=torch.int32, device="cuda")
        ms = _median_ms(lambda: buf.fill_(7), steps, warmup, stream)
        rows.append({"gib": gib, "bytes": n * 4, "ms": ms, "GBps": n * 4 / (ms * 1e-3) / 1e9})
        print(f"fill {gib} GiB: {ms:.3f} ms, {rows[-1]['GBps']:.1f} GB/s", file=sys.stderr, flush=True)
        del buf
        torch.cuda.empty_cache()
    print(json.dumps({"write_sweep": rows, "statistic": f"median of {steps} fills", "git": git_sha()}), flush=True)


KERNEL_SOURCES = ["program.h", "core.h", "kernels_dev.h", "jit_source.cpp", "jit.cpp", "compile.cpp", "graph.cpp"]
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "dg_enumerate_hbm_traffic.txt")
DAG_SOURCES = ["program.h", "core.h", "kernels_dev.h", "dag_program.h", "dag_core.h", "dag_dev.h", "dag.cpp",
               "kernels.hip", "jit_source.cpp", "jit.cpp", "graph.cpp"]
DAG_TRAFFIC_FILE = os.path.join(ROOT, "profiles", "dg_dag_fill_hbm_traffic.txt")


def measured_traffic(workload, path=TRAFFIC_FILE, sources=KERNEL_SOURCES):
    """HBM bytes per launch of the dominant kernel from a committed rocprofv3
    counter summary (FETCH_SIZE and WRITE_SIZE scaled by a copy of known
    size), or None when the kernel sources have changed since it was taken."""
    import hashlib
    if not os.path.exists(path):
        return None
    h = hashlib.sha256()
    for f in sources:
        with open(os.path.join(ROOT, "paper_2609_19611_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    stored, traffic = None, None
    for line in open(path):
        parts = line.split()
        if len(parts) == 2 and parts[0] == "kernel_sources_sha256":
            stored = parts[1]
        if len(parts) == 3 and parts[0] == "traffic_bytes_per_launch" and parts[1] == workload:
            traffic = int(parts[2])
    return traffic if stored == h.hexdigest() else None


def _median_ms(fn, steps, warmup, stream):
    """Median of `steps` timed calls of fn (HIP events on `stream`)."""
    import torch
    for _ in range(warmup):
        fn()
    torch.cuda.synchronize()
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(steps)]
    for a, b in ev:
        a.record(stream)
        fn()
        b.record(stream)
    torch.cuda.synchronize()
    return float(np.median([a.elapsed_time(b) for a, b in ev]))


def same_buffer_fill(ids, cnt, stream, steps=5, warmup=2):
    """Write rate of torch's fill over the enumeration's own output arrays
    (the same bytes at the same addresses).  Plain write rates fall with the
    size written (about 6.5 TB/s over 2 GiB, 5.7-6.0 TB/s over 35 GB on the
    same boxes), so this, not a 2 GiB fill, is the ceiling a writer of
    these rows is held to."""
    ms = _median_ms(lambda: (ids.fill_(7), cnt.fill_(7)), steps, warmup, stream)
    return (ids.numel() * ids.element_size() + cnt.numel() * cnt.element_size()) / (ms * 1e-3) / 1e9


def row_fill(ids, cnt, offsets, n, block, lds, stream, steps=5, warmup=2):
    """Write rate of a kernel that writes the same rows with no per-location
    work (the enumeration's grid, block size, LDS per block and lane shifts;
    lib/libdirigo_rowfill, a measurement reference built beside the
    library), or None when it is not built.  Plain fills run in address
    order; a one-block-per-row writer of these rows is what this figure
    times."""
    import ctypes
    path = os.path.join(ROOT, "paper_2609_19611_amd", "lib", "libdirigo_rowfill.so")
    if not os.path.exists(path):
        return None
    L = ctypes.CDLL(path)
    L.dgr_row_fill.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64, ctypes.c_int,
                               ctypes.c_uint32, ctypes.c_void_p]

    def call():
        rc = L.dgr_row_fill(ids.data_ptr(), cnt.data_ptr(), offsets.data_ptr(), n, block, lds,
                            ctypes.c_void_p(stream.cuda_stream))
        if rc:
            raise RuntimeError(f"dgr_row_fill failed: {rc}")
    ms = _median_ms(call, steps, warmup, stream)
    return (ids.numel() * ids.element_size() + cnt.numel() * cnt.element_size()) / (ms * 1e-3) / 1e9


def placement_spread(B, g, d_locs, offsets, ws, total, stream, sets=3, steps=7):
    """The enumeration and torch's fill of its output arrays in `sets` more
    allocations of the same output arrays (untimed for the headline): a
    writer of one row per block is sensitive to where the output's physical
    pages fall, which the allocator decides, while an address-ordered fill
    is not."""
    import torch
    # (All sets held at once, so that each is a distinct allocation.)
    bufs = [(torch.empty(total, dtype=torch.int32, device="cuda"), torch.empty(total, dtype=torch.int32, device="cuda"))
            for _ in range(sets)]
    out = []
    for ids, cnt in bufs:
        ms = _median_ms(lambda: B.dg_enumerate(g, d_locs, offsets, ids, cnt, ws), steps, 2, stream)
        fill = _median_ms(lambda: (ids.fill_(7), cnt.fill_(7)), steps, 2, stream)
        out.append({"enumerate_ms": ms, "fill_ms": fill, "frac_of_fill": fill / ms})
    del bufs
    torch.cuda.empty_cache()
    return out


def same_buffer_fill_dag(arrays, stream, steps=5, warmup=2):
    """Write rate of torch's fill over the DAG's own output arrays (nodes,
    first edges, edges, multiplicities: the same bytes at the same
    addresses)."""
    ms = _median_ms(lambda: [a.fill_(7) for a in arrays], steps, warmup, stream)
    return sum(a.numel() * a.element_size() for a in arrays) / (ms * 1e-3) / 1e9


def secondary_enumeration(B, W, name, fill_gbps, steps=10, warmup=3):
    """Single-pass enumeration of another workload: median call time of
    `steps` calls, rates and the HBM fraction (algorithmic bytes)."""
    import torch
    stream = torch.cuda.current_stream()
    g = B.dg_graph_parse(W.CONFIGS[name]["text"]())
    locs = W.config_locations(name)
    d_locs = torch.as_tensor(locs, dtype=torch.int64, device="cuda")
    n = len(locs)
    ws = B.workspace(g, n)
    off = torch.empty(n + 1, dtype=torch.int64, device="cuda")
    total = B.dg_enumerate_sizes(g, d_locs, off, ws)
    ids = torch.empty(total, dtype=torch.int32, device="cuda")
    cnt = torch.empty(total, dtype=torch.int32, device="cuda")
    ms = _median_ms(lambda: B.dg_enumerate(g, d_locs, off, ids, cnt, ws), steps, warmup, stream)
    alg = 16 * n + 8 * total
    gbps = alg / (ms * 1e-3) / 1e9
    same = same_buffer_fill(ids, cnt, stream)
    info = B.dg_graph_info(g)
    rows = row_fill(ids, cnt, off, n, info["block_threads"], info["lds_bytes"], stream)
    del ids, cnt
    torch.cuda.empty_cache()
    return {"workload": f"{name}: " + W.CONFIGS[name]["desc"], "locations": n, "entries": total,
            "ms_per_call": ms, "statistic": f"median of {steps} calls (dg_enumerate, whole call)",
            "entries_per_s": total / (ms * 1e-3), "locations_per_s": n / (ms * 1e-3),
            "achieved_GBps": gbps, "frac_of_hbm_peak": gbps / HBM_PEAK_GBS, "frac_of_measured_fill": gbps / fill_gbps,
            "same_buffer_fill_GBps": same, "frac_of_same_buffer_fill": gbps / same,
            "row_fill_GBps": rows, "frac_of_row_fill": gbps / rows if rows else None}


def secondary_compare(B, W, steps=5, warmup=2):
    """The pair check: the clean split-K variant alone (median of 10 calls)
    and the step of 17 comparisons (clean + 16 faults; median of `steps`)."""
    import concurrent.futures as cf
    import torch
    stream = torch.cuda.current_stream()
    ref = B.dg_graph_parse(W.c5_reference_text())
    variants = [B.dg_graph_parse(W.c5_variant_text())] + [B.dg_graph_parse(W.c5_variant_text(fault=f))
                                                          for f in W.c5_faults()]
    locs = W.config_locations("c5")
    d_locs = torch.as_tensor(locs, dtype=torch.int64, device="cuda")
    n = len(locs)

    def load(v):  # compiles the pair's specialised kernel (one location, own buffers)
        B.compare_locations(ref, v, locs[:1])
    with cf.ThreadPoolExecutor(8) as ex:
        list(ex.map(load, variants))
    torch.cuda.synchronize()
    ws = B.workspace(ref, n)
    status = torch.empty(n, dtype=torch.uint8, device="cuda")
    mism = torch.empty(n, dtype=torch.int64, device="cuda")
    clean = _median_ms(lambda: B.dg_compare(ref, variants[0], d_locs, status, mism, ws), 10, 2, stream)
    step = _median_ms(lambda: [B.dg_compare(ref, v, d_locs, status, mism, ws) for v in variants], steps, warmup,
                      stream)
    return {"workload": "c5: " + W.CONFIGS["c5"]["desc"], "locations": n,
            "clean_ms_per_compare": clean, "clean_locations_per_s": n / (clean * 1e-3),
            "step_ms_17_compares": step, "locations_per_s_17_compares": 17 * n / (step * 1e-3),
            "statistic": "median of 10 calls (clean) and of %d steps (17 compares)" % steps}


def secondary_dag(B, W, name, every=8, steps=5, warmup=1):
    """Expression DAGs of every `every`-th listed location of a workload:
    the fill kernel's median over `steps` launches (sizes pass and buffers
    beforehand, untimed), its HBM fraction (algorithmic bytes) and the row
    writer of its edge rows on the same buffers."""
    import torch
    stream = torch.cuda.current_stream()
    g = B.dg_graph_parse(W.CONFIGS[name]["text"]())
    locs = W.config_locations(name)[::every]
    d_locs = torch.as_tensor(locs, dtype=torch.int64, device="cuda")
    n = len(locs)
    ws = torch.empty(max(B.dg_workspace_size(g, n), 1), dtype=torch.uint8, device="cuda")
    noff = torch.empty(n + 1, dtype=torch.int64, device="cuda")
    eoff = torch.empty(n + 1, dtype=torch.int64, device="cuda")
    nn, ne = B.dg_dag_sizes(g, d_locs, noff, eoff, ws)
    out = [torch.empty(max(m, 1), dtype=torch.int32, device="cuda") for m in (nn, nn, ne, ne)]
    ms = _median_ms(lambda: B.dg_dag_fill(g, d_locs, noff, eoff, *out, ws), steps, warmup, stream)
    alg = 24 * n + 8 * nn + 8 * ne
    gbps = alg / (ms * 1e-3) / 1e9
    info = B.dg_graph_info(g)
    rows = row_fill(out[2], out[3], eoff, n, info["dag_block_threads"], info["dag_lds_bytes"], stream)
    del out
    torch.cuda.empty_cache()
    return {"workload": f"{name}: " + W.CONFIGS[name]["desc"] + " (expression DAGs)", "locations": n,
            "nodes": nn, "edges": ne, "fill_ms": ms,
            "statistic": f"median of {steps} launches (dg_dag_fill, whole call)",
            "kernels": "specialized" if info["dag_specialized"] == 1 else "precompiled",
            "achieved_GBps": gbps, "frac_of_hbm_peak": gbps / HBM_PEAK_GBS,
            "edge_row_fill_GBps": rows, "frac_of_edge_row_fill": gbps / rows if rows else None}


def git_sha():
    try:
        return subprocess.check_output(["git", "rev-parse", "--short", "HEAD"], cwd=ROOT,
                                       stderr=subprocess.DEVNULL).decode().strip()
    except Exception:
        return None


def cpu_baseline(workload, text_a, text_b, locs, target_s):
    """The oracle, as it stands, on a bounded prefix of the same location list."""
    import oracle
    threads = min(16, os.cpu_count() or 1)
    if workload == "c5":
        ga, gb = oracle.Graph(text_a), oracle.Graph(text_b)
        m = min(256, len(locs))
        while True:
            t0 = time.perf_counter()
            oracle.compare(ga, gb, locs[:m], threads=threads)
            dt = time.perf_counter() - t0
            if dt > 0.5 * target_s or m >= len(locs):
                break
            m = min(len(locs), int(m * min(64.0, max(2.0, 0.8 * target_s / max(dt, 1e-3)))))
        return {"value": m / dt, "unit": "locations/s", "cores": threads, "kind": "oracle",
                "sample": f"first {m} of {len(locs)} locations, one compare (clean variant)",
                "seconds": round(dt, 3)}
    g = oracle.Graph(text_a)
    m = min(16, len(locs))
    while True:
        t0 = time.perf_counter()
        off, _, _ = g.enumerate(locs[:m], threads=threads)
        dt = time.perf_counter() - t0
        if dt > 0.5 * target_s or m >= len(locs):
            break
        m = min(len(locs), int(m * min(64.0, max(2.0, 0.8 * target_s / max(dt, 1e-3)))))
    reps = 1
    if dt < 1.0:
        # The whole list takes under a second: repeat it for about a second.
        reps = int(min(1000, max(2, 1.0 / max(dt, 1e-4))))
        t0 = time.perf_counter()
        for _ in range(reps):
            off, _, _ = g.enumerate(locs[:m], threads=threads)
        dt = time.perf_counter() - t0
    sample = f"first {m} of {len(locs)} locations" + (f", {reps} passes" if reps > 1 else "")
    return {"value": float(off[-1]) * reps / dt, "unit": "entries/s", "cores": threads, "kind": "oracle",
            "sample": sample, "locations_per_s": m * reps / dt, "seconds": round(dt, 3)}


def stream_full_output(args, B, g, cfg, info, text):
    """Every location of the output, rows streamed through a bounded buffer;
    the consumer folds each chunk into a checksum on its stream."""
    import torch
    numel = info["output_numel"]
    buf = torch.empty(int(args.stream_gib * (1 << 30)), dtype=torch.uint8, device="cuda")
    streams = (torch.cuda.Stream(), torch.cuda.Stream())
    max_chunk = 1 << 17
    sums = []
    stats = {"entries": 0, "chunks": 0}

    def consume(first, off, ids, cnt, stream):
        # A light consumer, enqueued on the chunk's stream (current here):
        # a checksum over every 1024th count; no host wait.
        sums.append(torch.sum(cnt[::1024], dtype=torch.int64))
        stats["entries"] += ids.numel()
        stats["chunks"] += 1

    def step():
        sums.clear()
        stats["entries"] = stats["chunks"] = 0
        B.dg_enumerate_stream(g, 0, numel, buf, max_chunk, consume, streams)
        return stats["entries"], int(sum(int(x) for x in sums))

    for _ in range(max(1, args.warmup)):
        step()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        entries, checksum = step()
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    ms = elapsed * 1000 / args.steps
    line = {
        "metric": "footprint entries/sec enumerated (whole output streamed through a bounded buffer)",
        "value": entries / (elapsed / args.steps), "unit": "entries/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": ms, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "u32", "data": "synthetic (shapes only; footprints are data independent)",
        "config": {"workload": f"{args.workload}: " + cfg["desc"] + " (full output, streamed)", "locations": numel,
                   "entries_per_step": entries, "locations_per_s": numel / (elapsed / args.steps),
                   "buffer_gib": args.stream_gib, "chunks": stats["chunks"], "sampled_count_checksum": checksum,
                   "algorithmic_GBps": (16 * numel + 8 * entries) / (elapsed / args.steps) / 1e9},
        "roofline": {"bound": "hbm", "kernel": "dg_enumerate", "achieved": None, "peak": HBM_PEAK_GBS,
                     "unit": "GB/s", "frac": None, "traffic": None},
    }
    line["git"] = git_sha()
    print(json.dumps(line), flush=True)


def dag_bench(args, B, g, cfg, locs, text):
    """Expression DAGs of res(y[l]) for every listed location: sizes pass,
    scans and fill per step, buffers sized once beforehand."""
    import torch
    dev = torch.device("cuda", 0)
    d_locs = torch.as_tensor(locs, dtype=torch.int64, device=dev)
    n = len(locs)
    ws = torch.empty(max(B.dg_workspace_size(g, n), 1), dtype=torch.uint8, device=dev)
    noff = torch.empty(n + 1, dtype=torch.int64, device=dev)
    eoff = torch.empty(n + 1, dtype=torch.int64, device=dev)
    nn, ne = B.dg_dag_sizes(g, d_locs, noff, eoff, ws)
    nodes = torch.empty(max(nn, 1), dtype=torch.int32, device=dev)
    node_edge = torch.empty(max(nn, 1), dtype=torch.int32, device=dev)
    edges = torch.empty(max(ne, 1), dtype=torch.int32, device=dev)
    mults = torch.empty(max(ne, 1), dtype=torch.int32, device=dev)
    stream = torch.cuda.current_stream()
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(args.steps)]

    def step(i=None):
        B.dg_dag_sizes(g, d_locs, noff, eoff, ws)
        if i is not None:
            ev[i][0].record(stream)
        B.dg_dag_fill(g, d_locs, noff, eoff, nodes, node_edge, edges, mults, ws)
        if i is not None:
            ev[i][1].record(stream)

    for _ in range(max(1, args.warmup)):
        step()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        step(i)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    fill_ms = float(np.mean([a.elapsed_time(b) for a, b in ev]))
    fill_ms_median = float(np.median([a.elapsed_time(b) for a, b in ev]))
    same = same_buffer_fill_dag((nodes, node_edge, edges, mults), stream)
    info = B.dg_graph_info(g)
    kinds = "specialized" if info["dag_specialized"] == 1 else "precompiled"
    # The edge and multiplicity rows written by the row-writer reference with
    # the DAG kernels' grid, block size and LDS (nodes aside: 8 B per node).
    rows = row_fill(edges, mults, eoff, n, info["dag_block_threads"], info["dag_lds_bytes"], stream)
    # Algorithmic bytes of the fill: 8 (location) + 16 (two offsets) per
    # location, 8 per node (id + first edge), 8 per edge (child + multiplicity).
    alg = 24 * n + 8 * nn + 8 * ne
    achieved = alg / (fill_ms_median * 1e-3) / 1e9
    line = {
        "metric": "expression-DAG edges/sec emitted (sizes + fill; nodes and locations/sec in config)",
        "value": ne / (elapsed / args.steps), "unit": "edges/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": elapsed * 1000 / args.steps, "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "u32",
        "data": "synthetic (shapes only; footprints are data independent)",
        "config": {"workload": f"{args.workload}: " + cfg["desc"] + " (expression DAGs)", "locations": n,
                   "nodes_per_step": nn, "edges_per_step": ne, "locations_per_s": n / (elapsed / args.steps)},
        "roofline": {"bound": "hbm", "kernel": "dg_dag_fill" if kinds == "specialized" else "k_dag_fill",
                     "achieved": achieved, "peak": HBM_PEAK_GBS,
                     "unit": "GB/s", "frac": achieved / HBM_PEAK_GBS,
                     "traffic": measured_traffic(args.workload, DAG_TRAFFIC_FILE, DAG_SOURCES),
                     "traffic_unit": "HBM bytes per launch (rocprofv3 FETCH_SIZE x2 + WRITE_SIZE x1)",
                     "kernel_ms": fill_ms_median, "kernel_ms_mean": fill_ms,
                     "kernel_ms_statistic": f"median of {args.steps} launches", "algorithmic_bytes": alg,
                     "same_buffer_fill_GBps": same, "frac_of_same_buffer_fill": achieved / same,
                     "edge_row_fill_GBps": rows, "frac_of_edge_row_fill": achieved / rows if rows else None,
                     "kernels": kinds},
    }
    # The same fill in two more allocations of its output arrays (not part
    # of the headline): its rate depends on where their physical pages fall.
    del nodes, node_edge, edges, mults
    torch.cuda.empty_cache()
    others = [[torch.empty(max(m, 1), dtype=torch.int32, device=dev) for m in (nn, nn, ne, ne)] for _ in range(2)]
    line["roofline"]["other_allocations"] = [
        {"fill_ms": t, "frac": alg / (t * 1e-3) / 1e9 / HBM_PEAK_GBS}
        for t in (_median_ms(lambda: B.dg_dag_fill(g, d_locs, noff, eoff, *o, ws), 5, 1, stream) for o in others)]
    del others
    torch.cuda.empty_cache()
    if not args.no_cpu_baseline:
        import oracle
        m = max(1, min(n, 64))
        t1 = time.perf_counter()
        oracle.Graph(text).dag(locs[:m], threads=os.cpu_count() or 1)
        dt = time.perf_counter() - t1
        line["cpu_baseline"] = {"value": m / dt, "unit": "locations/s", "cores": os.cpu_count() or 1,
                                "kind": "oracle", "sample": f"first {m} of {n} locations"}
    line["git"] = git_sha()
    print(json.dumps(line), flush=True)


def merge_bench(args, B):
    """The running example as whole programs (both start with the same
    convolution): a step is dg_compare of the merged pair, common prefix
    trimmed, over all 131,072 output locations.  The same comparison of the
    untrimmed obligation (inputs matched only) and the merge itself are
    timed beside it."""
    import torch
    from paper_2609_19611_amd import workloads as W
    dev = torch.device("cuda", 0)
    torch.cuda.set_device(dev)
    a = B.dg_graph_parse(W.paper_program_text(False))
    b = B.dg_graph_parse(W.paper_program_text(True))
    t0 = time.perf_counter()
    ta, tb, k = B.dg_graph_merge(a, b, True)
    merge_ms = (time.perf_counter() - t0) * 1e3
    ua, ub, _ = B.dg_graph_merge(a, b, False)
    n = B.dg_graph_info(ta)["output_numel"]
    locs = torch.arange(n, dtype=torch.int64, device=dev)
    ws = torch.empty(max(B.dg_workspace_size(ta, n), B.dg_workspace_size(ua, n), 1), dtype=torch.uint8,
                     device=dev)
    status = torch.empty(n, dtype=torch.uint8, device=dev)
    mism = torch.empty(n, dtype=torch.int64, device=dev)

    def timed(x, y, steps, warmup):
        for _ in range(max(1, warmup)):
            m = B.dg_compare(x, y, locs, status, mism, ws)
        torch.cuda.synchronize()
        t1 = time.perf_counter()
        for _ in range(steps):
            m = B.dg_compare(x, y, locs, status, mism, ws)
        torch.cuda.synchronize()
        return (time.perf_counter() - t1) / steps, m

    dt, mism_trim = timed(ta, tb, args.steps, args.warmup)
    du, mism_full = timed(ua, ub, max(1, args.steps // 5), 1)
    line = {
        "metric": "output locations/sec compared after MERGE (common prefix trimmed)",
        "value": n / dt, "unit": "locations/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": dt * 1e3, "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "u32",
        "data": "synthetic (shapes only; footprints are data independent)",
        "config": {"workload": "paper running example as whole programs: x[128,3,64,64] -> conv(16, k3 p1) -> "
                               "min(C) -> sum(H) -> gelu -> +b vs the fused min/sum kernel (h < 32)",
                   "locations": n, "trimmed_ops": k, "merge_host_ms": merge_ms,
                   "mismatching_locations_trimmed": int(mism_trim),
                   "mismatching_locations_untrimmed": int(mism_full),
                   "untrimmed_locations_per_s": n / du, "untrimmed_ms_per_compare": du * 1e3,
                   "speedup_from_trimming": du / dt},
        "roofline": {"bound": "alu", "achieved": None, "peak": None, "unit": None, "frac": None, "traffic": None},
    }
    if not args.no_cpu_baseline:
        import oracle
        oa, ob, _ = oracle.merge(oracle.Graph(W.paper_program_text(False)), oracle.Graph(W.paper_program_text(True)))
        ga, gb = oracle.Graph(oa), oracle.Graph(ob)
        m = 4096
        t1 = time.perf_counter()
        oracle.compare(ga, gb, list(range(m)), threads=os.cpu_count() or 1)
        d = time.perf_counter() - t1
        line["cpu_baseline"] = {"value": m / d, "unit": "locations/s", "cores": os.cpu_count() or 1,
                                "kind": "oracle", "sample": f"first {m} of {n} locations, trimmed pair"}
    line["git"] = git_sha()
    print(json.dumps(line), flush=True)


def order_bench(args, B):
    """The location order of the c5 split-K variant (33,554,432 output
    locations): a step is dg_order_permute over every permutation position
    with the prefix's locations left out (device-resident, synchronous).
    Then, per seeded fault, the rank of the first mismatching location under
    the heuristic order, the plain permutation and the sequential order."""
    import torch
    from paper_2609_19611_amd import workloads as W
    dev = torch.device("cuda", 0)
    torch.cuda.set_device(dev)
    ref = B.dg_graph_parse(W.c5_reference_text())
    var = B.dg_graph_parse(W.c5_variant_text())
    n = B.dg_graph_info(var)["output_numel"]
    seed = 5
    prefix = B.dg_order_prefix(var)
    out = torch.empty(n, dtype=torch.int64, device=dev)
    ws = torch.empty(max(1, B.dg_order_workspace_size(len(prefix))), dtype=torch.uint8, device=dev)
    stream = torch.cuda.current_stream()
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(args.steps)]

    def step(i=None):
        if i is not None:
            ev[i][0].record(stream)
        w = B.dg_order_permute(n, seed, prefix, 0, n, out, ws)
        if i is not None:
            ev[i][1].record(stream)
        return w

    for _ in range(max(1, args.warmup)):
        step()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        w = step(i)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    call_ms = float(np.median([a.elapsed_time(b) for a, b in ev]))
    assert w + len(prefix) == n

    # Rank of the first mismatch: compare the reference with each faulty
    # variant over growing prefixes of an order until one mismatches.
    heur = torch.cat([torch.tensor(prefix, dtype=torch.int64, device=dev), out[:w]])
    perm = torch.empty(n, dtype=torch.int64, device=dev)
    B.dg_order_permute(n, seed, [], 0, n, perm, ws)
    seq = torch.arange(n, dtype=torch.int64, device=dev)
    cws = torch.empty(max(B.dg_workspace_size(ref, n), 1), dtype=torch.uint8, device=dev)
    status = torch.empty(n, dtype=torch.uint8, device=dev)
    mism = torch.empty(n, dtype=torch.int64, device=dev)

    def first_mismatch(v, order):
        lo, k = 0, 64
        while lo < n:
            hi = min(n, lo + k)
            m = B.dg_compare(ref, v, order[lo:hi], status, mism, cws)
            if m:
                return lo + int(mism[0].item())
            lo, k = hi, k * 4
        return None

    ranks = []
    # The 16 seeded faults, then the sparse ones (only the last output row, or
    # only the last row and column together, mismatch).
    for f in list(W.c5_faults()) + list(W.C5_SPARSE_FAULTS):
        v = B.dg_graph_parse(W.c5_variant_text(fault=f))
        ranks.append({"fault": f if isinstance(f, str) else "/".join(str(x) for x in f),
                      "heuristic": first_mismatch(v, heur),
                      "permutation": first_mismatch(v, perm), "sequential": first_mismatch(v, seq)})
    # ALU roofline: 24 32-bit operations per Feistel round (two 64-bit
    # multiplies, three 64-bit shifts, five 64-bit xors and ands), four rounds
    # per encryption, on average D / n encryptions per position (cycle walking
    # on the domain D = 4^h), against 256 CUs x 4 SIMDs x 16 lanes x 2.4 GHz.
    h = 0
    while (1 << (2 * h)) < n:
        h += 1
    ops = 24 * 4 * ((1 << (2 * h)) / n) * n
    achieved = ops / (call_ms * 1e-3) / 1e12
    line = {
        "metric": "output locations/sec ordered (keyed permutation of every output location, prefix left out)",
        "value": n / (elapsed / args.steps), "unit": "locations/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": elapsed * 1000 / args.steps, "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "int64",
        "data": "synthetic (shapes only; the order depends on shapes and the seed)",
        "config": {"workload": "c5 split-K variant output [64,128,64,64]: location order", "locations": n,
                   "seed": seed, "prefix": len(prefix), "first_mismatch_rank": ranks},
        "roofline": {"bound": "alu", "kernel": "k_order_write", "achieved": achieved, "peak": ALU_PEAK_TOPS,
                     "unit": "Tops/s (int32)", "frac": achieved / ALU_PEAK_TOPS, "traffic": None,
                     "call_ms": call_ms, "algorithmic_ops": ops, "hbm_bytes_written": 8 * w},
    }
    if not args.no_cpu_baseline:
        import oracle
        m = 2_000_000
        t1 = time.perf_counter()
        oracle.permutation(n, seed, 0, m)
        dt = time.perf_counter() - t1
        line["cpu_baseline"] = {"value": m / dt, "unit": "locations/s", "cores": 1, "kind": "oracle",
                                "sample": f"first {m} of {n} permutation positions"}
    line["git"] = git_sha()
    print(json.dumps(line), flush=True)


def main():
    args = parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU; --gpus {args.gpus} is not supported: each GPU would run an "
              "independent shard of the location list (no collective on the hot path), so the whole-job "
              "rate is N times the one-GPU rate measured here.", file=sys.stderr)
        sys.exit(2)

    if args.dag and (args.wide or args.two_pass or args.full_output):
        print("--dag takes no other mode", file=sys.stderr)
        sys.exit(2)
    if args.wide and (args.two_pass or args.full_output or args.workload == "c5"):
        print("--wide times the single-pass enumeration of c1-c4 only", file=sys.stderr)
        sys.exit(2)

    if args.write_sweep:
        write_sweep(args.steps, args.warmup)
        return
    if args.copy_gib > 0:
        copy_calibration(args.copy_gib, args.steps, args.warmup)
        return
    if args.order or args.merge:
        from paper_2609_19611_amd import binding as B
        (order_bench if args.order else merge_bench)(args, B)
        return

    import torch
    from paper_2609_19611_amd import binding as B
    from paper_2609_19611_amd import workloads as W

    cfg = W.CONFIGS[args.workload]
    text = cfg["text"]()
    locs = W.config_locations(args.workload)
    dev = torch.device("cuda", 0)
    torch.cuda.set_device(dev)
    stream = torch.cuda.current_stream()
    d_locs = torch.as_tensor(locs, dtype=torch.int64, device=dev)
    n = len(locs)
    g = B.dg_graph_parse(text)
    info = B.dg_graph_info(g)

    if args.dag:
        dag_bench(args, B, g, cfg, locs if args.workload != "c3" else locs[::8], text)
        return

    if args.workload == "c5":
        variants = [B.dg_graph_parse(W.c5_variant_text())] + [B.dg_graph_parse(W.c5_variant_text(fault=f))
                                                              for f in W.c5_faults()]
        if args.full_output:
            n = info["output_numel"]
        ws = torch.empty(max(B.dg_workspace_size(g, n), 1), dtype=torch.uint8, device=dev)
        status = torch.empty(n, dtype=torch.uint8, device=dev)
        mism = torch.empty(n, dtype=torch.int64, device=dev)

        if args.full_output:
            # A step verifies the clean variant at every output location;
            # the faulty variants, timed apart, stop at their first mismatch.
            variants_timed = variants[:1]
        else:
            variants_timed = variants

        def step():
            k = 0
            for v in variants_timed:
                if args.full_output:
                    k += B.dg_compare_range(g, v, 0, n, status, mism, ws)
                else:
                    k += B.dg_compare(g, v, d_locs, status, mism, ws)
            return k

        for _ in range(args.warmup):
            step()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(args.steps):
            mismatches = step()
        torch.cuda.synchronize()
        elapsed = time.perf_counter() - t0
        ms = elapsed * 1000 / args.steps
        compares = len(variants_timed)
        value = n * compares / (elapsed / args.steps)
        extra = {}
        roofline = {"bound": "alu", "achieved": None, "peak": None, "unit": None, "frac": None, "traffic": None}
        if not args.full_output:
            # The clean variant alone, whose every location compares whole
            # rows: entries compared are both graphs' row entries (their
            # sizes, untimed), priced at COMPARE_OPS_PER_ENTRY int32 ops.
            offs = torch.empty(n + 1, dtype=torch.int64, device=dev)
            entries = B.dg_enumerate_sizes(g, d_locs, offs, ws) + B.dg_enumerate_sizes(variants[0], d_locs, offs, ws)
            ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
                  for _ in range(args.steps)]
            for i in range(args.steps):
                ev[i][0].record(stream)
                B.dg_compare(g, variants[0], d_locs, status, mism, ws)
                ev[i][1].record(stream)
            torch.cuda.synchronize()
            clean_ms = float(np.median([x.elapsed_time(y) for x, y in ev]))
            achieved = COMPARE_OPS_PER_ENTRY * entries / (clean_ms * 1e-3) / 1e12
            extra = {"clean_ms_per_compare": clean_ms, "clean_entries_compared": entries,
                     "clean_entries_compared_per_s": entries / (clean_ms * 1e-3),
                     "clean_locations_per_s": n / (clean_ms * 1e-3)}
            roofline = {"bound": "alu", "kernel": "dg_compare (clean variant, whole call)", "achieved": achieved,
                        "peak": ALU_PEAK_TOPS, "unit": "Tops/s (int32)", "frac": achieved / ALU_PEAK_TOPS,
                        "traffic": None, "kernel_ms": clean_ms,
                        "kernel_ms_statistic": f"median of {args.steps} calls",
                        "model": f"{COMPARE_OPS_PER_ENTRY} int32 ops per row entry of either graph"}
        if args.full_output:
            fault_ms = []
            for v in variants[1:]:
                B.dg_compare_range(g, v, 0, 1, status, mism, ws)  # loads the pair's kernel (untimed)
                torch.cuda.synchronize()
                t1 = time.perf_counter()
                B.dg_compare_range(g, v, 0, n, status, mism, ws, max_mismatch=1)
                fault_ms.append((time.perf_counter() - t1) * 1000)
            extra = {"faulty_variants": len(fault_ms), "ms_to_first_mismatch_mean": float(np.mean(fault_ms)),
                     "ms_to_first_mismatch_max": float(np.max(fault_ms))}
        line = {
            "metric": "output locations/sec compared (two-graph footprint check)",
            "value": value, "unit": "locations/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
            "ms_per_step": ms, "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "u32",
            "data": "synthetic (shapes only; footprints are data independent)",
            "config": {"workload": "c5: " + cfg["desc"] + (" (full output)" if args.full_output else ""),
                       "locations": n, "compares_per_step": compares,
                       "mismatching_locations_last_step": int(mismatches), **extra},
            "roofline": roofline,
        }
        if not args.no_cpu_baseline:
            line["cpu_baseline"] = cpu_baseline("c5", text, W.c5_variant_text(), locs, args.cpu_seconds)
        line["git"] = git_sha()
        print(json.dumps(line), flush=True)
        return

    if args.full_output:
        stream_full_output(args, B, g, cfg, info, text)
        return

    ws = torch.empty(max(B.dg_workspace_size(g, n), 1), dtype=torch.uint8, device=dev)
    offsets = torch.empty(n + 1, dtype=torch.int64, device=dev)
    # Size the output buffers once (untimed); every timed step then computes
    # the offsets and rows from scratch.
    total = B.dg_enumerate_sizes(g, d_locs, offsets, ws)
    word = torch.int64 if args.wide else torch.int32
    ids = torch.empty(max(total, 1), dtype=word, device=dev)
    cnt = torch.empty(max(total, 1), dtype=word, device=dev)
    kern_ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
               for _ in range(args.steps)]

    if args.two_pass:
        kernel = "k_fill"

        def step(i=None):
            t = B.dg_enumerate_sizes(g, d_locs, offsets, ws)
            if i is not None:
                kern_ev[i][0].record(stream)
            B.dg_enumerate_fill(g, d_locs, offsets, ids, cnt, ws)
            if i is not None:
                kern_ev[i][1].record(stream)
            return t
    else:
        kernel = "k_enumerate_wide" if args.wide else "k_enumerate"
        enumerate_call = B.dg_enumerate_wide if args.wide else B.dg_enumerate

        def step(i=None):
            if i is not None:
                kern_ev[i][0].record(stream)
            t = enumerate_call(g, d_locs, offsets, ids, cnt, ws)
            if i is not None:
                kern_ev[i][1].record(stream)
            return t

    for _ in range(max(1, args.warmup)):
        step()
    torch.cuda.synchronize()
    # The first call compiled the graph's specialised kernels (unless
    # DIRIGO_JIT=0); the timed kernel is named accordingly.
    specialized = B.dg_graph_info(g)["specialized"] == 1
    if specialized:
        kernel = "dg_" + kernel[2:]
    t0 = time.perf_counter()
    for i in range(args.steps):
        t = step(i)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    assert t == total
    kern_times = [a.elapsed_time(b) for a, b in kern_ev]
    kern_ms = float(np.median(kern_times))
    ms = elapsed * 1000 / args.steps
    # Algorithmic bytes per location: 8 (location) + 8 (offset) + 8 per entry
    # (uint32 id + uint32 count; 16 with 64-bit ids and counts).
    alg_bytes = 16 * n + (16 if args.wide else 8) * total
    achieved = alg_bytes / (kern_ms * 1e-3) / 1e9
    line = {
        "metric": "footprint entries/sec enumerated (with output locations/sec and % of HBM peak)",
        "value": total / (elapsed / args.steps), "unit": "entries/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": ms, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "u64" if args.wide else "u32",
        "data": "synthetic (shapes only; footprints are data independent)",
        "config": {"workload": f"{args.workload}: " + cfg["desc"], "locations": n, "entries_per_step": total,
                   "locations_per_s": n / (elapsed / args.steps), "block_threads": info["block_threads"],
                   "lds_bytes": info["lds_wide_bytes" if args.wide else "lds_bytes"],
                   "path": "two-pass" if args.two_pass else ("single-pass, 64-bit" if args.wide else "single-pass"),
                   "kernels": "specialized" if specialized else "interpreted"},
        "roofline": {"bound": "hbm", "kernel": kernel, "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": achieved / HBM_PEAK_GBS,
                     "traffic": measured_traffic(args.workload) if kernel == "dg_enumerate" else None,
                     "traffic_unit": "HBM bytes per launch (rocprofv3 FETCH_SIZE x2 + WRITE_SIZE x1)",
                     "kernel_ms": kern_ms, "kernel_ms_mean": float(np.mean(kern_times)),
                     "kernel_ms_statistic": f"median of {args.steps} launches", "algorithmic_bytes": alg_bytes},
    }
    # The bandwidth plain torch kernels reach on this machine (after the timed
    # region), beside the spec peak: a fill of the same output arrays, and
    # a 2 GiB fill and copy.
    same = same_buffer_fill(ids, cnt, stream)
    rows = None if args.wide else row_fill(ids, cnt, offsets, n, info["block_threads"], info["lds_bytes"], stream)
    del ids, cnt
    spread = None
    if args.workload == "c4" and not (args.two_pass or args.wide) and not args.no_secondary:
        torch.cuda.empty_cache()
        spread = placement_spread(B, g, d_locs, offsets, ws, total, stream)
    rates = write_rates(2.0, 5, 2)
    line["roofline"]["same_buffer_fill_GBps"] = same
    line["roofline"]["frac_of_same_buffer_fill"] = achieved / same
    line["roofline"]["row_fill_GBps"] = rows
    line["roofline"]["frac_of_row_fill"] = achieved / rows if rows else None
    if spread:
        # The same call in three more allocations of its output arrays (not
        # part of the headline): the rate depends on the physical placement.
        line["roofline"]["other_allocations"] = spread
    line["roofline"]["measured_fill_GBps"] = rates["fill_GBps_write"]
    line["roofline"]["measured_fill_bytes"] = rates["bytes"]
    line["roofline"]["measured_copy_GBps"] = rates["copy_GBps_read_plus_write"]
    line["roofline"]["frac_of_measured_fill"] = achieved / rates["fill_GBps_write"]
    if args.workload == "c4" and not (args.two_pass or args.wide) and not args.no_secondary:
        # The other headline figures, timed after the main one: the
        # conv-transpose + softmax enumeration, the pair check and the
        # conv-transpose's expression DAGs.
        line["secondary"] = {"c3": secondary_enumeration(B, W, "c3", rates["fill_GBps_write"]),
                             "c5": secondary_compare(B, W),
                             "c3_dag": secondary_dag(B, W, "c3")}
    if not args.no_cpu_baseline:
        line["cpu_baseline"] = cpu_baseline(args.workload, text, None, locs, args.cpu_seconds)
    line["git"] = git_sha()
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
