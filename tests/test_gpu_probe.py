"""The bandwidth probes that bench.py measures its ceilings with: the row-pattern copy takes
rows from a queue, like the fused pass, so every row must be copied exactly once whatever
order the workgroups take them in; the small-block copy must copy every 16-byte vector."""

import ctypes
import os

import pytest
import torch

pytestmark = pytest.mark.gpu
ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _probe():
    lib = ctypes.CDLL(os.path.join(ROOT, "paper_2609_32444_amd", "libcis_probe.so"))
    lib.cis_probe_bandwidth.argtypes = [ctypes.c_int, ctypes.c_void_p, ctypes.c_void_p,
                                        ctypes.c_int64, ctypes.c_int64, ctypes.c_int,
                                        ctypes.c_void_p, ctypes.c_void_p]
    return lib


@pytest.mark.parametrize("mode,rows,row_bytes", [(0, 5000, 303872), (0, 3, 65536),
                                                 (3, 777, 4112)])
def test_probe_copies_every_row(mode, rows, row_bytes):
    lib = _probe()
    gen = torch.Generator(device="cuda")
    gen.manual_seed(rows)
    src = torch.randint(0, 256, (rows * row_bytes,), dtype=torch.uint8, device="cuda",
                        generator=gen)
    dst = torch.zeros_like(src)
    # 1024 sink words and the row queue's 64-bit counter, filled with junk: the call must
    # clear the counter itself
    sink = torch.full((1026,), -1, dtype=torch.int32, device="cuda")
    grid = torch.cuda.get_device_properties(0).multi_processor_count
    stream = torch.cuda.current_stream().cuda_stream
    for _ in range(2):  # a second call on the same sink starts from a cleared counter again
        dst.zero_()
        rc = lib.cis_probe_bandwidth(mode, src.data_ptr(), dst.data_ptr(), rows, row_bytes,
                                     grid, sink.data_ptr(), stream)
        assert rc == 0
        torch.cuda.synchronize()
        assert torch.equal(dst, src)


def test_probe_rejects_misaligned_sink():
    lib = _probe()
    buf = torch.zeros(1 << 16, dtype=torch.uint8, device="cuda")
    sink = torch.zeros(1030, dtype=torch.int32, device="cuda")
    rc = lib.cis_probe_bandwidth(0, buf.data_ptr(), buf.data_ptr(), 1, 4096, 1,
                                 sink.data_ptr() + 4, torch.cuda.current_stream().cuda_stream)
    assert rc == -2
