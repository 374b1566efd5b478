"""The bench's write-rate reference (lib/libdirigo_rowfill.so, dgr_row_fill)
writes exactly the rows it is given: row i's entries p get (p, i), nothing
outside [offsets[0], offsets[n]) changes, for ragged rows at any alignment,
both block sizes."""

import ctypes
import os

import numpy as np
import pytest
import torch

pytestmark = pytest.mark.gpu

LIB = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "paper_2609_19611_amd", "lib",
                   "libdirigo_rowfill.so")


@pytest.mark.parametrize("block", [64, 256])
def test_row_fill_writes_exactly_the_rows(block):
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    L = ctypes.CDLL(LIB)
    L.dgr_row_fill.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64, ctypes.c_int,
                               ctypes.c_uint32, ctypes.c_void_p]
    rng = np.random.default_rng(block)
    sizes = rng.integers(0, 700, 300)
    sizes[::17] = 0
    lead, tail = 13, 29
    off = np.concatenate([[0], np.cumsum(sizes)]) + lead
    total = int(off[-1]) + tail
    dev = torch.device("cuda", 0)
    ids = torch.full((total,), -1, dtype=torch.int32, device=dev)
    cnt = torch.full((total,), -1, dtype=torch.int32, device=dev)
    d_off = torch.as_tensor(off, dtype=torch.int64, device=dev)
    stream = torch.cuda.current_stream()
    assert L.dgr_row_fill(ids.data_ptr(), cnt.data_ptr(), d_off.data_ptr(), len(sizes), block, 4096,
                          ctypes.c_void_p(stream.cuda_stream)) == 0
    torch.cuda.synchronize()
    want_ids = np.full(total, -1, dtype=np.int64)
    want_cnt = np.full(total, -1, dtype=np.int64)
    for i, s in enumerate(sizes):
        p = np.arange(off[i], off[i] + s)
        want_ids[p] = p
        want_cnt[p] = i
    assert np.array_equal(ids.cpu().numpy().astype(np.int64), want_ids)
    assert np.array_equal(cnt.cpu().numpy().astype(np.int64), want_cnt)
    assert L.dgr_row_fill(ids.data_ptr(), cnt.data_ptr(), d_off.data_ptr(), 4, 128, 0, None) == -1
