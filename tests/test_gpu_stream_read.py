"""The streaming-read reference kernel (the bandwidth a read-only kernel
reaches on this GPU) reads every 16-byte chunk of its buffer exactly once:
a buffer of zeros with one 32-bit word set to the kernel's fixed fold value
makes exactly that word's lane write the sink."""
import pytest

pytestmark = pytest.mark.gpu

MAGIC = 0x9E3779B9


@pytest.mark.parametrize("unroll,blocks", [(4, 1), (8, 8), (16, 32), (8, 3)])
def test_every_chunk_is_read_once(gpu_lib, unroll, blocks):
    import torch
    n_words = (64 << 20) // 4 + 4 * 37  # not a multiple of the workgroup ranges
    buf = torch.zeros(n_words, dtype=torch.int32, device="cuda")
    sink = torch.zeros(1, dtype=torch.int32, device="cuda")
    gpu_lib.stream_read(buf, sink, unroll=unroll, blocks_per_cu=blocks)
    torch.cuda.synchronize()
    assert int(sink.item()) == 0
    magic = MAGIC - (1 << 32)  # as int32
    for pos in (0, 3, n_words // 2 + 1, n_words - 1, n_words - 5):
        buf.zero_()
        buf[pos] = magic
        sink.zero_()
        gpu_lib.stream_read(buf, sink, unroll=unroll, blocks_per_cu=blocks)
        torch.cuda.synchronize()
        assert int(sink.item()) == magic, f"word {pos} not read exactly once"
