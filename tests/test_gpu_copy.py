"""The streaming copy the bench reports as the practical HBM ceiling: bit
exact for sizes below, at and far above one sweep of the grid, including
ragged tails, and leaves the bytes past the end untouched."""
import pytest
import torch

import paper_2607_27090_amd as isl

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("units", [1, 7, 1000, 524_288, 524_288 + 13, 4_194_304 * 3 + 5])
def test_stream_copy_bit_exact(units):
    g = torch.Generator(device="cuda").manual_seed(units)
    src = torch.randint(-2 ** 31, 2 ** 31 - 1, (units * 4,), generator=g, dtype=torch.int32,
                        device="cuda")
    dst = torch.full((units * 4 + 4,), 0x5A5A5A5A, dtype=torch.int32, device="cuda")
    isl.is_stream_copy(dst[:units * 4], src)
    torch.cuda.synchronize()
    assert torch.equal(dst[:units * 4], src)
    assert bool((dst[units * 4:] == 0x5A5A5A5A).all())
