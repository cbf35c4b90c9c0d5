"""GPU parity of the two-branch llsa_backward (and the llsa_forward that
feeds it) against the fp64 oracle's exact adjoint of the LLSA forward, on
identical inputs, with the upstream gradient of both outputs drawn N(0, 1).

As for the SA backward (test_gpu_backward), each case runs twice: with the
oracle's forward output (rounded to bfloat16) and log-sum-exp supplied to
both sides, held per (branch, sequence, head) slice normwise and element by
element against the scale of its row; and end to end (GPU forward into GPU
backward) against the exact gradient, per branch tensor normwise: the bfloat16
rounding of `out` alone moves a slice of dq by up to 2.3e-2 of its maximum
(the oracle's own figure)."""

import numpy as np
import pytest
import torch

from paper_2302_13451_amd import binding as bd
from paper_2302_13451_amd.inputs import llsa_inputs
from parity import TORCH_DTYPE, assert_close, assert_slices_close, f64, round_to, to_gpu

pytestmark = pytest.mark.gpu


def _inputs(B, T, H, d, Lb, La, seed, lengths, scale, pad, tag, dtype="bf16"):
    print("llsa backward %s case B=%d T=%d H=%d d=%d Lb=%d La=%d %s seed=%d" % (
        tag, B, T, H, d, Lb, La, dtype, seed), flush=True)
    x = llsa_inputs(B, T, H, d, seed, dtype=dtype, scale=scale, lengths=lengths, pad_value=pad,
                    with_dout=True)
    g = {n: to_gpu(x[n], dtype) for n in ("q", "k", "v", "dout")}
    clean = {n: np.nan_to_num(f64(x[n])) for n in ("q", "k", "v", "dout")}
    return x, g, clean


def run(oracle_mod, B, T, H, d, Lb, La, seed, lengths, scale="rsqrt_d", pad=0.0, dtype="bf16"):
    x, g, clean = _inputs(B, T, H, d, Lb, La, seed, lengths, scale, pad, "end-to-end", dtype)
    ln = x["lengths"].cuda()
    out, lse = bd.llsa_forward(g["q"], g["k"], g["v"], Lb, La, ln)
    dq, dk, dv = bd.llsa_backward(g["q"], g["k"], g["v"], out, lse, g["dout"], Lb, La, ln)
    torch.cuda.synchronize()
    ref = oracle_mod.llsa_two_branch_backward(clean["q"], clean["k"], clean["v"], clean["dout"], Lb,
                                              La, x["lengths"].numpy())
    return (f64(dq), f64(dk), f64(dv)), ref, x["lengths"].tolist()


def run_supplied(oracle_mod, B, T, H, d, Lb, La, seed, lengths, scale="rsqrt_d", pad=0.0,
                 dtype="bf16"):
    x, g, clean = _inputs(B, T, H, d, Lb, La, seed, lengths, scale, pad, "supplied-output", dtype)
    L = x["lengths"].numpy()
    y, lse = oracle_mod.llsa_two_branch(clean["q"], clean["k"], clean["v"], Lb, La, L)
    y = round_to(y, dtype)
    out = torch.from_numpy(y).to(TORCH_DTYPE[dtype]).cuda()
    dq, dk, dv = bd.llsa_backward(g["q"], g["k"], g["v"], out, torch.from_numpy(lse).float().cuda(),
                                  g["dout"], Lb, La, x["lengths"].cuda())
    torch.cuda.synchronize()
    ref = oracle_mod.llsa_two_branch_backward(clean["q"], clean["k"], clean["v"], clean["dout"], Lb,
                                              La, L, y=y)
    return (f64(dq), f64(dk), f64(dv)), ref, x["lengths"].tolist()


def _zero_atol(ref):
    return 1e-5 * float(np.max(np.abs(ref[2])))


def check_slices(got, ref, lengths, elementwise=True, dtype="bf16"):
    for name, g, r in zip(("dq", "dk", "dv"), got, ref):
        assert_slices_close(g, r, dtype, lengths, name, elementwise=elementwise,
                            zero_atol=_zero_atol(ref), row_scale=dtype == "bf16")


def check_end_to_end(got, ref, lengths=None, dtype="bf16"):
    if dtype == "f32":
        check_slices(got, ref, lengths, dtype="f32")
        return
    for name, g, r in zip(("dq", "dk", "dv"), got, ref):
        for br, bname in ((0, "causal"), (1, "look-ahead")):
            assert_close(g[br], r[br], "bf16", "%s %s" % (name, bname), elementwise=False,
                         zero_atol=_zero_atol(ref))


@pytest.mark.parametrize("B,T,H,d,Lb,La,lengths", [
    (2, 200, 2, 64, 37, 5, (50, 200)),
    (2, 150, 2, 32, 64, 8, (1, 150)),
    (2, 130, 2, 64, 20, 0, (70, 130)),
    (2, 170, 3, 64, 0, 9, (100, 170)),
    (1, 99, 2, 64, 10, 1, "full"),
    (2, 190, 2, 64, 64, 8, (60, 190)),
    (2, 160, 2, 64, 24, 16, (60, 160)),
    (2, 120, 1, 64, 15, 25, (33, 120)),
    (2, 100, 1, 32, 80, 20, (30, 100)),
    # empty sequences between others, and more sequences than a wave has lanes
    (6, 140, 2, 64, 40, 8, (0, 140, 0, 70, 1, 0)),
    (66, 80, 1, 64, 30, 4, (0, 80)),
])
@pytest.mark.parametrize("scale", ["rsqrt_d", "unit"])
def test_llsa_backward_parity(oracle_mod, B, T, H, d, Lb, La, lengths, scale):
    got, ref, L = run_supplied(oracle_mod, B, T, H, d, Lb, La, 51, lengths, scale)
    check_slices(got, ref, L)
    got, ref, L = run(oracle_mod, B, T, H, d, Lb, La, 51, lengths, scale)
    check_end_to_end(got, ref)


def test_llsa_backward_padded_frames_are_never_read(oracle_mod):
    got, ref, L = run_supplied(oracle_mod, 3, 180, 2, 64, 30, 6, 52, (40, 179), pad=float("nan"))
    check_slices(got, ref, L)
    got, ref, L = run(oracle_mod, 3, 180, 2, 64, 30, 6, 52, (40, 179), pad=float("nan"))
    for g in got:
        assert np.all(np.isfinite(g))
    check_end_to_end(got, ref)
    for g in got:
        for b, n in enumerate(L):
            assert np.all(g[:, b, n:] == 0.0)


# More 64-frame tiles than the persistent kernel has workgroups (256), so each
# walks several (sequence, head) slices: steps that continue their
# predecessor's bands and steps that start a new slice, with branch C (La > 0)
# and without (La = 0), and windows on both sides of its ring geometry.
@pytest.mark.parametrize("B,T,H,d,Lb,La,lengths", [
    (16, 640, 8, 64, 37, 5, (1, 640)),
    (12, 700, 10, 64, 20, 0, (100, 700)),
    (16, 600, 8, 64, 24, 16, (50, 600)),
    (20, 520, 12, 64, 64, 8, (0, 520)),
    (16, 600, 8, 64, 64, 16, (50, 600)),
])
def test_llsa_backward_persistent(oracle_mod, B, T, H, d, Lb, La, lengths):
    got, ref, L = run_supplied(oracle_mod, B, T, H, d, Lb, La, 57, lengths)
    check_slices(got, ref, L)


def test_llsa_backward_persistent_padded_frames_are_never_read(oracle_mod):
    """NaN in every padding frame, with several slices per workgroup of the
    persistent kernel (steps that continue and steps that start a slice)."""
    got, ref, L = run_supplied(oracle_mod, 24, 400, 12, 64, 64, 8, 58, (50, 399), pad=float("nan"))
    for g in got:
        assert np.all(np.isfinite(g))
    check_slices(got, ref, L)
    for g in got:
        for b, n in enumerate(L):
            assert np.all(g[:, b, n:] == 0.0)


def test_config4_backward_full_size(oracle_mod):
    """LLSA backward bf16, B=16, T=800, H=12, d=64, Lb=64, La=8, lengths U[400, 800]."""
    got, ref, L = run_supplied(oracle_mod, 16, 800, 12, 64, 64, 8, 4, (400, 800))
    check_slices(got, ref, L)
    got, ref, L = run(oracle_mod, 16, 800, 12, 64, 64, 8, 4, (400, 800))
    check_end_to_end(got, ref)


# Windows past one staged segment and float32 (the vector-ALU kernel), and the
# boundaries from both sides: Lb = 32, La = 16 still stages (MFMA); Lb = 64,
# La = 16 does not stage but fits the persistent kernel's rings at bfloat16
# (MFMA for up to 64 sequences at d = 64); Lb = 70, La = 20 fits neither.
@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("B,T,H,d,Lb,La,lengths", [
    (2, 200, 2, 64, 70, 20, (60, 200)),
    (2, 190, 2, 64, 32, 16, (60, 190)),
    (2, 190, 2, 64, 64, 16, (60, 190)),
    (2, 150, 1, 32, 120, 30, (40, 150)),
    (3, 90, 2, 64, 5, 0, (0, 90, 17)),
    (66, 40, 1, 64, 8, 3, (0, 40)),
])
def test_llsa_backward_every_window(oracle_mod, dtype, B, T, H, d, Lb, La, lengths):
    got, ref, L = run_supplied(oracle_mod, B, T, H, d, Lb, La, 56, lengths, "unit", dtype=dtype)
    check_slices(got, ref, L, dtype=dtype)
    got, ref, L = run(oracle_mod, B, T, H, d, Lb, La, 56, lengths, "unit", dtype=dtype)
    check_end_to_end(got, ref, L, dtype)


def test_llsa_backward_float32_config4_shape(oracle_mod):
    """float32 at the LLSA workload's window, B=4, T=800, H=12, d=64, Lb=64, La=8."""
    got, ref, L = run_supplied(oracle_mod, 4, 800, 12, 64, 64, 8, 57, (400, 800), dtype="f32")
    check_slices(got, ref, L, dtype="f32")
