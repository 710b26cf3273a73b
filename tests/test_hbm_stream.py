"""The HBM read stream (dwkv_hbm_read) on the GPU through the C ABI: the xor
of the sink words it writes equals the xor of the buffer's 32-bit words,
computed on the host, bit for bit; sink words past the block count are left
alone.  Sizes cover an empty buffer, a single 16-byte word, a partial last
round, and buffers larger than a round of every block."""
import numpy as np
import pytest

from gpu_util import announce, torch_gpu

pytestmark = pytest.mark.gpu

SENTINEL = 0x5A5A5A5A


@pytest.mark.parametrize("n_bytes", [0, 16, 48, 32768 + 16, 5 * (1 << 20) + 48, 96 * (1 << 20) + 32768 * 3 + 16])
def test_hbm_read_xor(n_bytes):
    torch = torch_gpu()
    from paper_2607_06523_amd import hbm_read, hbm_read_blocks
    blocks = hbm_read_blocks()
    rng = np.random.default_rng(n_bytes % 1000 + 7)
    words = rng.integers(0, 1 << 32, size=n_bytes // 4, dtype=np.uint64).astype(np.uint32)
    buf = torch.from_numpy(words.view(np.int32).copy()).cuda() if n_bytes else torch.empty(0, dtype=torch.int32,
                                                                                          device="cuda")
    sink = torch.full((blocks + 4,), SENTINEL, dtype=torch.int32, device="cuda")
    announce(f"hbm_read bytes={n_bytes}")
    hbm_read(buf, sink)
    got = sink.cpu().numpy().view(np.uint32)
    torch.cuda.synchronize()
    want = np.bitwise_xor.reduce(words) if n_bytes else np.uint32(0)
    assert np.bitwise_xor.reduce(got[:blocks]) == want
    assert np.all(got[blocks:] == SENTINEL)
