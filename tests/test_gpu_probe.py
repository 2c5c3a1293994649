"""The bandwidth probes move the bytes they report: the copy copies, the
write writes its constant everywhere, the row probe stores the XOR of the
rows it read at the same offsets of every destination row and nothing
beyond the rows' length."""
import pytest
import torch

from paper_2507_07114_amd import probe

pytestmark = pytest.mark.gpu
DEV = "cuda"


def test_copy_read_and_write_probes():
    n = (1 << 20) + 48  # a ragged last workgroup
    src = torch.randint(0, 2**31 - 1, (n,), dtype=torch.int32, device=DEV)
    dst = torch.zeros_like(src)
    sink = torch.zeros(probe.SINK_BYTES, dtype=torch.uint8, device=DEV)
    assert probe.hbm_probe_copy(src, dst) == 8 * n
    assert probe.hbm_probe_read(src, sink) == 4 * n
    want = src.clone()
    assert probe.hbm_probe_write(src[: n // 2]) == 2 * n
    torch.cuda.synchronize()
    assert torch.equal(dst, want)
    assert torch.all(src[: n // 2].view(torch.float32) == 1.0)
    assert torch.equal(src[n // 2:], want[n // 2:])
    assert torch.equal(sink, torch.zeros_like(sink))


def test_rows_probe_stores_the_xor_of_the_rows():
    rows, ld, row = 6, 4096 * 3 + 64, 4096 * 2 + 512 + 16  # int32 elements; ragged last tile
    src = torch.randint(0, 2**31 - 1, (rows, ld), dtype=torch.int32, device=DEV)
    dst = torch.full((rows, ld), -7, dtype=torch.int32, device=DEV)
    sink = torch.zeros(probe.SINK_BYTES, dtype=torch.uint8, device=DEV)
    moved = probe.hbm_probe_rows(src, 5, dst, 4, row * 4, sink)
    torch.cuda.synchronize()
    assert moved == 9 * row * 4
    want = src[0, :row].clone()
    for i in range(1, 5):
        want ^= src[i, :row]
    for i in range(4):
        assert torch.equal(dst[i, :row], want), i
    assert torch.all(dst[:4, row:] == -7) and torch.all(dst[4:] == -7)
