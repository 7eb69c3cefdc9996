"""The read-stream measurement aid reads every 16-byte vector of its buffer exactly once:
the XOR of all the words it writes equals the XOR of the buffer's 32-bit words (each
wave folds what it read with XOR, and XOR is order-free), for buffers that fill the
grid-stride loop and ones with a ragged tail, on small and large grids."""
import numpy as np
import pytest

from paper_2606_08382_amd import starkv as S

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("n_vec,wg", [(1, 1), (37, 1), (256 * 17 + 5, 3), (1 << 16, 64),
                                      ((1 << 20) + 123, 2048)])
def test_read_stream_reads_every_vector_once(n_vec, wg):
    import torch
    rng = np.random.default_rng(n_vec * 31 + wg)
    host = rng.integers(0, 2**32, size=4 * n_vec, dtype=np.uint32)
    src = torch.from_numpy(host.view(np.int32)).cuda()
    sink = torch.zeros(wg * 4, dtype=torch.int32, device="cuda")
    S.starkv_read_stream(src, 16 * n_vec, sink, wg)
    torch.cuda.synchronize()
    got = np.bitwise_xor.reduce(sink.cpu().numpy().view(np.uint32))
    assert got == np.bitwise_xor.reduce(host)
