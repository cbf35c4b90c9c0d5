"""GPU parity of sa_backward (and the forward that feeds it) against the fp64
oracle on identical inputs, with the upstream gradient drawn N(0, 1)."""

import numpy as np
import pytest
import torch

from paper_2302_13451_amd import binding as bd
from paper_2302_13451_amd.inputs import sa_inputs
from parity import assert_close, f64, to_gpu

pytestmark = pytest.mark.gpu


def run(oracle_mod, B, T, H, d, Lb, La, dtype, seed, lengths, scale="rsqrt_d", pad=0.0):
    print("backward case B=%d T=%d H=%d d=%d Lb=%d La=%d %s seed=%d" % (B, T, H, d, Lb, La,
                                                                       dtype, seed), flush=True)
    x = sa_inputs(B, T, H, d, seed, dtype=dtype, scale=scale, lengths=lengths, pad_value=pad)
    q, k, v, do = (to_gpu(x[n], dtype) for n in ("q", "k", "v", "dout"))
    ln = x["lengths"].cuda()
    out, lse = bd.sa_forward(q, k, v, Lb, La, ln)
    dq, dk, dv = bd.sa_backward(q, k, v, out, lse, do, Lb, La, ln)
    torch.cuda.synchronize()
    clean = {n: np.nan_to_num(f64(x[n])) for n in ("q", "k", "v", "dout")}
    ref = oracle_mod.sa_backward(clean["q"], clean["k"], clean["v"], clean["dout"], Lb, La,
                                 x["lengths"].numpy())
    return (f64(dq), f64(dk), f64(dv)), ref, x


def check(got, ref, dtype):
    # a zero band has dq = dk = 0 exactly; rounding noise is bounded by the
    # scale of dv (= dout there)
    zero_atol = 1e-5 * float(np.max(np.abs(ref[2])))
    for name, g, r in zip(("dq", "dk", "dv"), got, ref):
        assert_close(g, r, dtype, name, elementwise=False, zero_atol=zero_atol)


def test_config1_shape_float32(oracle_mod):
    got, ref, _ = run(oracle_mod, 1, 64, 2, 32, 8, 2, "f32", 1, "full", "unit")
    check(got, ref, "f32")


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("B,T,H,d,Lb,La,lengths", [
    (3, 200, 2, 64, 37, 5, (50, 200)),
    (2, 131, 3, 32, 64, 8, (1, 131)),
    (2, 257, 2, 64, 0, 9, (100, 257)),
    (2, 190, 1, 64, 70, 0, (64, 190)),
    (2, 97, 2, 32, 200, 200, (30, 97)),
    (1, 40, 2, 64, 0, 0, "full"),
    # a window that just fills one staged segment of 144 frames (64 + Lb + La),
    # and one that needs the multi-segment sweep
    (2, 260, 2, 64, 72, 8, (70, 260)),
    (2, 300, 2, 64, 100, 20, (50, 300)),
    (1, 600, 2, 32, 250, 60, (300, 600)),
    # empty sequences between others, and more sequences than a wave has lanes
    (6, 130, 2, 64, 30, 8, (0, 130, 0, 64, 1, 0)),
    (66, 70, 1, 64, 20, 4, (0, 70)),
    (65, 50, 1, 32, 30, 30, (1, 50)),
])
@pytest.mark.parametrize("scale", ["rsqrt_d", "unit"])
def test_backward_parity(oracle_mod, dtype, B, T, H, d, Lb, La, lengths, scale):
    got, ref, _ = run(oracle_mod, B, T, H, d, Lb, La, dtype, 7, lengths, scale)
    check(got, ref, dtype)


def test_config3_full_size(oracle_mod):
    """SA forward+backward bf16, B=16, T=800, H=12, d=64, Lb=64, La=8, lengths
    U[400, 800] with tail padding."""
    got, ref, _ = run(oracle_mod, 16, 800, 12, 64, 64, 8, "bf16", 3, (400, 800))
    check(got, ref, "bf16")


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_backward_padded_frames_are_never_read(oracle_mod, dtype):
    got, ref, x = run(oracle_mod, 3, 230, 2, 64, 40, 6, dtype, 12, (60, 229), "unit",
                      pad=float("nan"))
    check(got, ref, dtype)
    for g in got:
        for b, L in enumerate(x["lengths"].tolist()):
            assert np.all(g[b, L:] == 0)


def test_backward_deterministic():
    x = sa_inputs(4, 333, 3, 64, 14, dtype="bf16", lengths=(100, 333))
    q, k, v, do = (to_gpu(x[n], "bf16") for n in ("q", "k", "v", "dout"))
    ln = x["lengths"].cuda()
    out, lse = bd.sa_forward(q, k, v, 50, 7, ln)
    g1 = bd.sa_backward(q, k, v, out, lse, do, 50, 7, ln)
    g2 = bd.sa_backward(q, k, v, out, lse, do, 50, 7, ln)
    for a, b in zip(g1, g2):
        assert torch.equal(a, b)
