"""GPU: the direct global->LDS copy the multi-channel kernels stage their
filter rows with.  A 16-byte-per-lane copy puts lane l's four floats at
4l .. 4l + 3 past its LDS destination, also when that destination is 4, 8
or 12 bytes past a 16-byte boundary (the kernels keep filter rows at an odd
pitch for conflict-free reads), and writes nothing else."""
import pytest
import torch

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("shift", [0, 1, 2, 3])
def test_16_byte_lds_copy_layout(shift):
    from paper_2212_00404_amd import peaks
    out = peaks.lds_dma_layout(shift)
    want = torch.zeros(264)
    want[shift:shift + 256] = torch.arange(256, dtype=torch.float32) + 1.0
    assert torch.equal(out, want), (shift, out[:12], out[shift + 250:shift + 258])
