"""tq_read_probe, the bench's streaming-read measurement (not part of the
method), through the C ABI: it reads without writing and rejects bad sizes."""
import ctypes

import pytest
import torch

import paper_2603_26110_amd as tq

pytestmark = pytest.mark.gpu


def test_read_probe_reads_and_leaves_sink():
    data = torch.arange(3 * 2 ** 20, dtype=torch.int32, device="cuda")
    sink = torch.zeros(4096, dtype=torch.int32, device="cuda")
    for blocks in (1, 7, 1024, 4096):
        tq.read_probe(data, blocks, sink)
    torch.cuda.synchronize()
    assert int(sink.abs().sum()) == 0


def test_read_probe_rejects_bad_sizes():
    L = tq._load()
    data = torch.zeros(64, dtype=torch.int32, device="cuda")
    sink = torch.zeros(16, dtype=torch.int32, device="cuda")
    s = torch.cuda.current_stream().cuda_stream
    assert L.tq_read_probe(ctypes.c_void_p(data.data_ptr()), 100, 4, ctypes.c_void_p(sink.data_ptr()),
                           ctypes.c_void_p(s)) != 0
    assert L.tq_read_probe(ctypes.c_void_p(data.data_ptr()), 256, 0, ctypes.c_void_p(sink.data_ptr()),
                           ctypes.c_void_p(s)) != 0
    assert L.tq_read_probe(ctypes.c_void_p(data.data_ptr() + 4), 240, 4, ctypes.c_void_p(sink.data_ptr()),
                           ctypes.c_void_p(s)) != 0
    assert L.tq_read_probe(ctypes.c_void_p(data.data_ptr()), 256, 4, ctypes.c_void_p(sink.data_ptr()),
                           ctypes.c_void_p(s)) == 0
    torch.cuda.synchronize()
