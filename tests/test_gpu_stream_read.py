"""The read-only streaming kernel that bench.py measures read-bound kernels
against (rs3_stream_read): every 16-byte chunk read exactly once, by thread
chunk % RS3_STREAM_READ_THREADS, and xor-reduced per thread."""
import numpy as np
import pytest

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")


@pytest.mark.parametrize("n16", [3 * 262144 + 12345, 5])
def test_stream_read_xor_per_thread(n16):
    import paper_2608_22526_amd as rs3
    nth = rs3.RS3_STREAM_READ_THREADS
    rng = np.random.default_rng(n16)
    data = rng.integers(0, 2 ** 32, size=(n16, 4), dtype=np.uint64).astype(np.uint32)
    src = torch.from_numpy(data.view(np.int32).reshape(-1)).cuda()
    out = torch.full((nth,), -1, dtype=torch.int32, device="cuda")
    rs3.stream_read(src, n16 * 16, out)
    torch.cuda.synchronize()
    got = out.cpu().numpy().view(np.uint32)
    words = np.bitwise_xor.reduce(data, axis=1)              # xor of each chunk's four words
    pad = np.zeros(-(-n16 // nth) * nth, np.uint32)
    pad[:n16] = words
    exp = np.bitwise_xor.reduce(pad.reshape(-1, nth), axis=0)
    assert np.array_equal(got, exp)


def test_stream_read_rejects_unaligned():
    import paper_2608_22526_amd as rs3
    src = torch.zeros(64, dtype=torch.int32, device="cuda")
    out = torch.zeros(rs3.RS3_STREAM_READ_THREADS, dtype=torch.int32, device="cuda")
    with pytest.raises(rs3.Rs3Error):
        rs3.stream_read(src, 100, out)
