"""GPU parity of sa_backward (and the forward that feeds it) against the fp64
oracle on identical inputs, with the upstream gradient drawn N(0, 1).

Two kinds of case:

* supplied output: the backward gets the oracle's forward output rounded to the
  element type and its log-sum-exp in float; the oracle computes the gradient
  for that same output (the term dout . out of the softmax Jacobian product
  taken from it). Both sides then compute one function of identical inputs,
  and every (sequence, head) slice is held to the tolerance normwise and
  element by element (float32 against the element, bfloat16 against the
  scale of the element's row: see parity.assert_slices_close).
* end to end: the GPU forward feeds the GPU backward, against the exact
  gradient. In float32 this is held to the same per-slice, per-element bar.
  In bfloat16 the rounding of `out` to bfloat16 moves dq and dk by itself (the
  oracle, given its own output rounded to bfloat16, differs from the exact
  gradient by up to 2.3e-2 of a slice's maximum), so end-to-end bfloat16
  cases are held per output tensor, normwise.
"""

import numpy as np
import pytest
import torch

from paper_2302_13451_amd import binding as bd
from paper_2302_13451_amd.inputs import sa_inputs
from parity import TORCH_DTYPE, assert_close, assert_slices_close, f64, round_to, to_gpu

pytestmark = pytest.mark.gpu


def _inputs(B, T, H, d, Lb, La, dtype, seed, lengths, scale, pad, tag):
    print("backward %s case B=%d T=%d H=%d d=%d Lb=%d La=%d %s seed=%d" % (
        tag, B, T, H, d, Lb, La, dtype, seed), flush=True)
    x = sa_inputs(B, T, H, d, seed, dtype=dtype, scale=scale, lengths=lengths, pad_value=pad)
    g = {n: to_gpu(x[n], dtype) for n in ("q", "k", "v", "dout")}
    clean = {n: np.nan_to_num(f64(x[n])) for n in ("q", "k", "v", "dout")}
    return x, g, clean


def run(oracle_mod, B, T, H, d, Lb, La, dtype, seed, lengths, scale="rsqrt_d", pad=0.0):
    """End to end: GPU forward, GPU backward, exact oracle gradient."""
    x, g, clean = _inputs(B, T, H, d, Lb, La, dtype, seed, lengths, scale, pad, "end-to-end")
    ln = x["lengths"].cuda()
    out, lse = bd.sa_forward(g["q"], g["k"], g["v"], Lb, La, ln)
    dq, dk, dv = bd.sa_backward(g["q"], g["k"], g["v"], out, lse, g["dout"], Lb, La, ln)
    torch.cuda.synchronize()
    ref = oracle_mod.sa_backward(clean["q"], clean["k"], clean["v"], clean["dout"], Lb, La,
                                 x["lengths"].numpy())
    return (f64(dq), f64(dk), f64(dv)), ref, x


def run_supplied(oracle_mod, B, T, H, d, Lb, La, dtype, seed, lengths, scale="rsqrt_d", pad=0.0):
    """The backward alone, both sides given the oracle's forward output
    (rounded to the element type) and log-sum-exp."""
    x, g, clean = _inputs(B, T, H, d, Lb, La, dtype, seed, lengths, scale, pad, "supplied-output")
    L = x["lengths"].numpy()
    y, lse = oracle_mod.sa_forward(clean["q"], clean["k"], clean["v"], Lb, La, L)
    y = round_to(y, dtype)
    out = torch.from_numpy(y).to(TORCH_DTYPE[dtype]).cuda()
    lse_g = torch.from_numpy(lse).float().cuda()
    dq, dk, dv = bd.sa_backward(g["q"], g["k"], g["v"], out, lse_g, g["dout"], Lb, La,
                                x["lengths"].cuda())
    torch.cuda.synchronize()
    ref = oracle_mod.sa_backward(clean["q"], clean["k"], clean["v"], clean["dout"], Lb, La, L,
                                 y=y)
    return (f64(dq), f64(dk), f64(dv)), ref, x


def _zero_atol(ref):
    # a zero band has dq = dk = 0 exactly; rounding noise is bounded by the
    # scale of dv (= dout there)
    return 1e-5 * float(np.max(np.abs(ref[2])))


def check_slices(got, ref, dtype, lengths, elementwise=True):
    # float32 gradients element by element; bfloat16 ones against their row's
    # scale (parity.assert_slices_close)
    for name, g, r in zip(("dq", "dk", "dv"), got, ref):
        assert_slices_close(g, r, dtype, lengths, name, elementwise=elementwise,
                            zero_atol=_zero_atol(ref), row_scale=dtype == "bf16")


def check_end_to_end(got, ref, dtype, lengths):
    if dtype == "f32":
        check_slices(got, ref, dtype, lengths)
    else:
        for name, g, r in zip(("dq", "dk", "dv"), got, ref):
            assert_close(g, r, dtype, name, elementwise=False, zero_atol=_zero_atol(ref))


def test_config1_shape_float32(oracle_mod):
    got, ref, x = run(oracle_mod, 1, 64, 2, 32, 8, 2, "f32", 1, "full", "unit")
    check_slices(got, ref, "f32", x["lengths"])
    got, ref, x = run_supplied(oracle_mod, 1, 64, 2, 32, 8, 2, "f32", 1, "full", "unit")
    check_slices(got, ref, "f32", x["lengths"])


SHAPES = [
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
]


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("B,T,H,d,Lb,La,lengths", SHAPES)
@pytest.mark.parametrize("scale", ["rsqrt_d", "unit"])
def test_backward_parity(oracle_mod, dtype, B, T, H, d, Lb, La, lengths, scale):
    got, ref, x = run_supplied(oracle_mod, B, T, H, d, Lb, La, dtype, 7, lengths, scale)
    check_slices(got, ref, dtype, x["lengths"])
    got, ref, x = run(oracle_mod, B, T, H, d, Lb, La, dtype, 7, lengths, scale)
    check_end_to_end(got, ref, dtype, x["lengths"])


def test_config3_full_size(oracle_mod):
    """SA forward+backward bf16, B=16, T=800, H=12, d=64, Lb=64, La=8, lengths
    U[400, 800] with tail padding: the backward alone per slice and element,
    and the GPU forward feeding it."""
    got, ref, x = run_supplied(oracle_mod, 16, 800, 12, 64, 64, 8, "bf16", 3, (400, 800))
    check_slices(got, ref, "bf16", x["lengths"])
    got, ref, x = run(oracle_mod, 16, 800, 12, 64, 64, 8, "bf16", 3, (400, 800))
    check_end_to_end(got, ref, "bf16", x["lengths"])


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_backward_padded_frames_are_never_read(oracle_mod, dtype):
    got, ref, x = run_supplied(oracle_mod, 3, 230, 2, 64, 40, 6, dtype, 12, (60, 229), "unit",
                               pad=float("nan"))
    check_slices(got, ref, dtype, x["lengths"])
    got, ref, x = run(oracle_mod, 3, 230, 2, 64, 40, 6, dtype, 12, (60, 229), "unit",
                      pad=float("nan"))
    check_end_to_end(got, ref, dtype, x["lengths"])
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
