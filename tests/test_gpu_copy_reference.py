"""The device-copy reference (a measurement aid, not part of the method)
copies every byte in both access modes, including a ragged tail."""

import pytest
import torch

from paper_2302_13451_amd import binding as bd

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("mode", [0, 1])
@pytest.mark.parametrize("n16", [1, 63, 257, 64 * 4 * 1000 + 17, 3 << 20])
def test_copy_reference_copies_every_byte(mode, n16):
    print("copy reference mode=%d pieces=%d" % (mode, n16), flush=True)
    g = torch.Generator(device="cpu").manual_seed(n16)
    src = torch.randint(-2 ** 31, 2 ** 31 - 1, (4 * n16,), generator=g, dtype=torch.int32).cuda()
    dst = torch.full((4 * n16 + 8,), 7, dtype=torch.int32, device="cuda")
    bd.copy_reference(src, dst[:4 * n16], mode)
    torch.cuda.synchronize()
    assert torch.equal(dst[:4 * n16], src)
    assert torch.all(dst[4 * n16:] == 7)
