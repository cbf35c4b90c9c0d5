"""GPU parity of the two-branch llsa_forward against the fp64 oracle (the
paper's LLSA in the general channel form with channels 0..La-1 held by the
causal branch and channel La by the look-ahead branch)."""

import numpy as np
import pytest
import torch

from paper_2302_13451_amd import binding as bd
from paper_2302_13451_amd.inputs import llsa_inputs
from parity import assert_lse_close, assert_slices_close, f64, to_gpu

pytestmark = pytest.mark.gpu


def run(oracle_mod, B, T, H, d, Lb, La, dtype, seed, lengths, scale="rsqrt_d", pad=0.0):
    print("llsa case B=%d T=%d H=%d d=%d Lb=%d La=%d %s seed=%d" % (B, T, H, d, Lb, La, dtype,
                                                                   seed), flush=True)
    x = llsa_inputs(B, T, H, d, seed, dtype=dtype, scale=scale, lengths=lengths, pad_value=pad)
    q, k, v = (to_gpu(x[n], dtype) for n in ("q", "k", "v"))
    out, lse = bd.llsa_forward(q, k, v, Lb, La, x["lengths"].cuda())
    torch.cuda.synchronize()
    clean = {n: np.nan_to_num(f64(x[n])) for n in ("q", "k", "v")}
    yr, lr = oracle_mod.llsa_two_branch(clean["q"], clean["k"], clean["v"], Lb, La,
                                        x["lengths"].numpy())
    return f64(out), lse.cpu().numpy(), yr, lr, x["lengths"].numpy()


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("B,T,H,d,Lb,La,lengths", [
    (2, 200, 2, 64, 37, 5, (50, 200)),
    (2, 150, 2, 32, 64, 8, (1, 150)),
    (2, 130, 2, 64, 20, 0, (70, 130)),
    (2, 170, 3, 64, 0, 9, (100, 170)),
    (1, 99, 2, 64, 10, 1, "full"),
    (2, 70, 1, 32, 300, 300, (10, 70)),
    # the largest look-ahead the persistent kernel takes, and one past it;
    # empty sequences between others; more sequences than a wave has lanes
    (2, 190, 2, 64, 64, 16, (60, 190)),
    (2, 190, 2, 64, 64, 17, (60, 190)),
    (6, 140, 2, 64, 40, 8, (0, 140, 0, 70, 1, 0)),
    (66, 80, 1, 64, 30, 4, (0, 80)),
])
@pytest.mark.parametrize("scale", ["rsqrt_d", "unit"])
def test_llsa_parity(oracle_mod, dtype, B, T, H, d, Lb, La, lengths, scale):
    out, lse, yr, lr, ln = run(oracle_mod, B, T, H, d, Lb, La, dtype, 31, lengths, scale)
    assert_slices_close(out, yr, dtype, ln, "out (causal, look-ahead)")
    assert_lse_close(lse, lr, dtype)


def test_config4_full_size(oracle_mod):
    """LLSA forward bf16, B=16, T=800, H=12, d=64, Lb=64, La=8, lengths U[400, 800]."""
    out, lse, yr, lr, ln = run(oracle_mod, 16, 800, 12, 64, 64, 8, "bf16", 4, (400, 800))
    assert_slices_close(out, yr, "bf16", ln, "out (causal, look-ahead)")
    assert_lse_close(lse, lr, "bf16")


def test_llsa_padded_frames_are_never_read(oracle_mod):
    out, lse, yr, lr, ln = run(oracle_mod, 3, 180, 2, 64, 30, 6, "bf16", 33, (40, 179),
                               pad=float("nan"))
    assert_slices_close(out, yr, "bf16", ln, "out")
    assert_lse_close(lse, lr, "bf16")


def test_llsa_dependency_horizon():
    """Perturbing any frame after t leaves the causal output of t bit-identical,
    and any frame after t + La leaves the look-ahead output of t bit-identical."""
    B, T, H, d, Lb, La = 1, 160, 2, 64, 24, 6
    x = llsa_inputs(B, T, H, d, 34, dtype="bf16", scale="unit")
    q, k, v = (to_gpu(x[n], "bf16") for n in ("q", "k", "v"))
    base, _ = bd.llsa_forward(q, k, v, Lb, La)
    for tau in (40, 97, 130):
        qp, kp, vp = q.clone(), k.clone(), v.clone()
        for t_ in (qp, kp, vp):
            t_[:, :, tau] += 1.0
        pert, _ = bd.llsa_forward(qp, kp, vp, Lb, La)
        diff = (pert != base).any(dim=-1).any(dim=-1)[:, 0].cpu()  # [branch][T]
        assert not diff[0, :tau].any()
        assert not diff[1, :tau - La].any()
        assert diff[0, tau] and diff[1, tau - La]
