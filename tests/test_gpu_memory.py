"""Memory per training vector of one attention layer's forward + backward
(Sec. "Lower Memory Usage", Fig. 5): SA through the library against masked
acausal attention (MAA) in PyTorch at d = 64, N_T = 1000.

What is fixed here is exact: the library allocates nothing and keeps no score,
weight or mask tensor, so SA's peak is the sum of its own tensors (q, k, v,
dout, out, lse, dq, dk, dv) whatever the receptive field, while MAA keeps
T x T matrices and so needs several times more at every width."""

import pytest

import bench
from paper_2302_13451_amd import accounting as acc

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("H", [8, 16])
def test_sa_memory_is_its_tensors_at_every_width(H):
    B, T, d, La = 2, 1000, 64, 8
    tensors = B * acc.sa_training_tensor_bytes(T, H, d)
    alone = bench.sa_tensors_memory(B, T, H, d)  # the same tensors, no kernel
    # the caching allocator may keep a large block whole (2 MiB granules)
    assert tensors <= alone <= tensors + 9 * (2 << 20)
    for W in (10, 250, 490):
        got = bench.sa_training_memory(B, T, H, d, W - 1 - La, La)
        print("SA H=%d W=%d: %d bytes, the tensors alone %d (%d exact)" % (H, W, got, alone, tensors),
              flush=True)
        assert got == alone


def test_maa_needs_more_memory_than_sa():
    B, T, d, H, La = 2, 1000, 64, 8, 8
    for W in (10, 490):
        sa = bench.sa_training_memory(B, T, H, d, W - 1 - La, La)
        maa = bench.maa_training_memory(B, T, H, d, W - 1 - La, La)
        print("W=%d: SA %d, MAA %d bytes" % (W, sa, maa), flush=True)
        # MAA holds at least the float32 T x T scores of every head
        assert maa >= B * H * T * T * 4
        assert maa > 4 * sa
