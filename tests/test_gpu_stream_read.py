"""GPU check of the streaming-read reference (nnjit_stream_read), the
measurement helper that times what one launch can stream from HBM.

Its kernel folds every 32-bit word a thread reads into one XOR and stores
that value (to the thread's workgroup's sink word) only when it equals one
constant.  A zero buffer with a single 16-byte chunk holding the constant
therefore names the workgroup that read that chunk: with G workgroups of 256
threads, chunk c is read by thread c mod 256G, so exactly sink word
(c mod 256G) / 256 changes.  Chunks in the first pass, later passes of the
four-deep loop and the remainder loop, and the last chunk, are each read
exactly where the grid-stride order puts them; a chunk that is never read,
or read by the wrong workgroup, leaves the sink wrong.
"""
import pytest

import paper_2309_08978_amd as nj

pytestmark = pytest.mark.gpu

MAGIC = 0x9E3779B9
MAGIC_I32 = MAGIC - (1 << 32)   # the same bits as a signed 32-bit value


def test_stream_read_reads_every_chunk_where_the_grid_puts_it():
    import torch
    wgs = 8
    stride = 256 * wgs                      # chunks per pass of the grid
    n16 = 3 * 4 * stride + 37               # three full four-deep passes, then 37 in the remainder loop
    chunks = [0, 1, 255, 256, stride - 1, stride, 4 * stride + 5, 2 * 4 * stride + 300, 12 * stride, n16 - 1]
    buf = torch.zeros(n16 * 4, dtype=torch.int32, device="cuda:0")
    sink = torch.empty(wgs, dtype=torch.int32, device="cuda:0")
    for c in chunks:
        buf.zero_()
        buf[4 * c] = MAGIC_I32
        sink.fill_(7)
        assert nj.nnjit_stream_read(buf, n16 * 16, sink, wgs) == nj.NNJIT_OK, nj.nnjit_last_error()
        torch.cuda.synchronize()
        expect = [7] * wgs
        expect[(c % stride) // 256] = MAGIC_I32
        assert sink.cpu().tolist() == expect, f"chunk {c}"


def test_stream_read_on_zeros_writes_nothing():
    import torch
    for wgs in (1, 64, 4096):
        buf = torch.zeros(1 << 20, dtype=torch.int32, device="cuda:0")
        sink = torch.full((wgs,), 7, dtype=torch.int32, device="cuda:0")
        assert nj.nnjit_stream_read(buf, buf.numel() * 4, sink, wgs) == nj.NNJIT_OK
        torch.cuda.synchronize()
        assert bool((sink == 7).all())
