"""The streaming-read measurement kernel reads every dword of its buffer
exactly once: the XOR of its per-workgroup sink words equals the XOR of the
buffer, for ragged partitions of the chunks over the workgroups."""
import numpy as np
import pytest
import torch

from paper_2608_08020_amd.gambit import GambitError, stream_read

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("nontemporal", [False, True])
@pytest.mark.parametrize("chunks,grid", [(1, 1), (37, 1), (37, 5), (37, 37), (300, 64)])
def test_every_dword_read_once(nontemporal, chunks, grid):
    print(f"stream_read chunks={chunks} grid={grid} nt={nontemporal}", flush=True)
    rng = np.random.default_rng(chunks * 100 + grid)
    host = rng.integers(-2**31, 2**31, size=chunks * 65536 // 4, dtype=np.int64).astype(np.int32)
    buf = torch.from_numpy(host).cuda()
    sink = torch.zeros(grid, dtype=torch.int32, device="cuda")
    stream_read(buf, nontemporal, grid, sink)
    got = np.bitwise_xor.reduce(sink.cpu().numpy().view(np.uint32))
    want = np.bitwise_xor.reduce(host.view(np.uint32))
    assert got == want


def test_rejects_bad_sizes():
    buf = torch.zeros(65536 // 4 + 4, dtype=torch.int32, device="cuda")
    sink = torch.zeros(4, dtype=torch.int32, device="cuda")
    with pytest.raises(GambitError):
        stream_read(buf, False, 1, sink)           # not a multiple of 64 KiB
    with pytest.raises(GambitError):
        stream_read(buf[:65536 // 4], False, 2, sink)  # more workgroups than chunks
