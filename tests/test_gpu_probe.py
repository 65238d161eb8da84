"""The benchmark's streaming-read probe (libtkprobe, not the attention ABI)
reads every 32-bit word of its buffer exactly once: the XOR of its per-thread
sink words equals the XOR of all words of the buffer, for the grid the bench
uses, with and without the non-temporal hint, and for ragged sizes and grids."""
import ctypes
import os

import numpy as np
import pytest
import torch

from gpu_cases import device, say

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
PROBE = os.path.join(ROOT, "paper_2603_04427_amd", "libtkprobe.so")


def probe():
    lib = ctypes.CDLL(PROBE)  # built beside libtkattn; a missing probe fails the test
    lib.tkprobe_threads.restype = ctypes.c_int
    lib.tkprobe_stream_read.restype = ctypes.c_int
    lib.tkprobe_stream_read.argtypes = [ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p, ctypes.c_int,
                                        ctypes.c_int, ctypes.c_void_p]
    return lib


@pytest.mark.parametrize("nbytes,grid,nt", [(16 * 1000003, 256, 0), (16 * 1000003, 256, 1), (4096, 7, 1),
                                            (16, 1, 0), (16 * 513, 3, 1)])
def test_stream_probe_reads_every_word_once(nbytes, grid, nt):
    dev = device()
    lib = probe()
    g = torch.Generator().manual_seed(nbytes + grid + nt)
    host = torch.randint(-(2 ** 31), 2 ** 31 - 1, (nbytes // 4,), dtype=torch.int32, generator=g)
    buf = host.to(dev)
    sink = torch.zeros(grid * lib.tkprobe_threads(), dtype=torch.int32, device=dev)
    say(f"stream probe: {nbytes} bytes, {grid} workgroups, non_temporal={nt}")
    rc = lib.tkprobe_stream_read(ctypes.c_void_p(buf.data_ptr()), nbytes, ctypes.c_void_p(sink.data_ptr()), grid, nt,
                                 ctypes.c_void_p(torch.cuda.current_stream().cuda_stream))
    assert rc == 0
    torch.cuda.synchronize()
    got = np.bitwise_xor.reduce(sink.cpu().numpy())
    want = np.bitwise_xor.reduce(host.numpy())
    assert got == want
