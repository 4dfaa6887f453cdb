"""The streaming-read measurement kernel (acceptmoe_stream_read) reads every
byte it is given: its per-workgroup XOR checksums equal the host's over the
same shares, including a ragged tail and workgroups left without a share."""
import numpy as np
import pytest
import torch

from paper_2608_02989_amd import ops

pytestmark = pytest.mark.gpu


def host_checksums(words: np.ndarray, nbytes: int, grid: int) -> np.ndarray:
    n16 = nbytes // 16
    per = (n16 + grid - 1) // grid
    pieces = words[: n16 * 4].reshape(n16, 4)
    out = np.zeros(grid, np.uint32)
    for b in range(grid):
        lo, hi = b * per, min((b + 1) * per, n16)
        if lo < hi:
            out[b] = np.bitwise_xor.reduce(pieces[lo:hi].reshape(-1))
    return out


@pytest.mark.parametrize("nbytes,grid", [(16, 1), (16 * 1000 + 48, 7), (16 * 300, 512), (1 << 20, 256),
                                         ((1 << 22) + 16 * 5, 1000)])
def test_stream_read_checksums(gpu, nbytes, grid):
    print(f"[stream_read] bytes={nbytes} grid={grid}", flush=True)
    rng = np.random.default_rng(nbytes + grid)
    words = rng.integers(0, 2**32, size=(nbytes + 64) // 4, dtype=np.uint64).astype(np.uint32)
    src = torch.from_numpy(words.view(np.int32)).cuda()
    sink = torch.full((grid,), -1, dtype=torch.int32, device="cuda")
    ops.stream_read(src, nbytes, sink, grid)
    torch.cuda.synchronize()
    got = sink.cpu().numpy().view(np.uint32)
    np.testing.assert_array_equal(got, host_checksums(words, nbytes, grid))
