"""GPU parity of llsa_paper_forward (the paper's LLSA with La + 1 channels,
each computed with its own query, Eq. 14/15 in the convention of Fig. 4)
against the fp64 oracle's general channel form, which the Fig. 4 worked
example pins."""

import numpy as np
import pytest
import torch

from paper_2302_13451_amd import binding as bd
from paper_2302_13451_amd.inputs import llsa_inputs
from parity import assert_close, assert_lse_close, f64, to_gpu

pytestmark = pytest.mark.gpu


def run(oracle_mod, B, T, H, d, Lb, La, dtype, seed, lengths, scale="rsqrt_d", pad=0.0):
    print("llsa paper case B=%d T=%d H=%d d=%d Lb=%d La=%d %s seed=%d" % (
        B, T, H, d, Lb, La, dtype, seed), flush=True)
    x = llsa_inputs(B, T, H, d, seed, dtype=dtype, scale=scale, lengths=lengths, pad_value=pad,
                    channels=La + 1)
    q, k, v = (to_gpu(x[n], dtype) for n in ("q", "k", "v"))
    out, lse = bd.llsa_paper_forward(q, k, v, Lb, La, x["lengths"].cuda())
    torch.cuda.synchronize()
    clean = {n: np.nan_to_num(f64(x[n])) for n in ("q", "k", "v")}
    yr, lr = oracle_mod.llsa_paper(clean["q"], clean["k"], clean["v"], Lb, La,
                                   x["lengths"].numpy())
    return f64(out), lse.cpu().numpy(), yr, lr, x["lengths"].numpy()


def check(out, lse, yr, lr, dtype):
    for c in range(out.shape[0]):
        assert_close(out[c], yr[c], dtype, "channel %d out" % c)
    assert_lse_close(lse, lr, dtype)


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("B,T,H,d,Lb,La,lengths", [
    (2, 150, 2, 64, 30, 1, (40, 150)),   # the paper's two-channel module
    (2, 130, 2, 32, 21, 3, (1, 130)),
    (2, 120, 3, 64, 64, 8, (50, 120)),
    (1, 90, 2, 64, 0, 4, "full"),        # band of one frame
    (2, 100, 1, 64, 17, 0, (30, 100)),   # one channel: plain causal SA
    (3, 9, 2, 64, 5, 12, (0, 9, 4)),     # look-ahead longer than the sequences
    (66, 40, 1, 32, 10, 2, (0, 40)),
])
@pytest.mark.parametrize("scale", ["rsqrt_d", "unit"])
def test_llsa_paper_parity(oracle_mod, dtype, B, T, H, d, Lb, La, lengths, scale):
    check(*run(oracle_mod, B, T, H, d, Lb, La, dtype, 41, lengths, scale)[:4], dtype)


def test_llsa_paper_config4_shape(oracle_mod):
    """bf16, B=4, T=800, H=12, d=64, Lb=64, La=8 (nine channels), lengths
    U[400, 800]."""
    check(*run(oracle_mod, 4, 800, 12, 64, 64, 8, "bf16", 5, (400, 800))[:4], "bf16")


def test_llsa_paper_padded_frames_are_never_read(oracle_mod):
    out, lse, yr, lr, ln = run(oracle_mod, 3, 160, 2, 64, 24, 5, "bf16", 43, (40, 159),
                               pad=float("nan"))
    check(out, lse, yr, lr, "bf16")
    for b, L in enumerate(ln):
        assert (out[:, b, L:] == 0).all()
        assert np.isneginf(lse[:, b, :, L:]).all()


def test_llsa_paper_one_channel_is_causal_sa():
    """With La = 0 the module is SA with the window t-Lb .. t: bit-identical to
    sa_forward, which runs the same band kernel."""
    x = llsa_inputs(2, 140, 2, 64, 44, dtype="bf16", lengths=(60, 140), channels=1)
    q, k, v = (to_gpu(x[n], "bf16") for n in ("q", "k", "v"))
    ln = x["lengths"].cuda()
    out, lse = bd.llsa_paper_forward(q, k, v, 33, 0, ln)
    ref, lref = bd.sa_forward(q[0], k[0], v[0], 33, 0, ln)
    assert torch.equal(out[0], ref)
    assert torch.equal(lse[0], lref)


def test_llsa_paper_dependency_horizon():
    """Channel c of frame t reads inputs up to frame t + c only: perturbing
    frame tau of every channel leaves channel c bit-identical at t < tau - c."""
    B, T, H, d, Lb, La = 1, 150, 2, 64, 20, 5
    x = llsa_inputs(B, T, H, d, 45, dtype="bf16", scale="unit", channels=La + 1)
    q, k, v = (to_gpu(x[n], "bf16") for n in ("q", "k", "v"))
    base, _ = bd.llsa_paper_forward(q, k, v, Lb, La)
    for tau in (30, 88, 140):
        qp, kp, vp = q.clone(), k.clone(), v.clone()
        for t_ in (qp, kp, vp):
            t_[:, :, tau] += 1.0
        pert, _ = bd.llsa_paper_forward(qp, kp, vp, Lb, La)
        diff = (pert != base).any(dim=-1).any(dim=-1)[:, 0].cpu()  # [channel][T]
        for c in range(La + 1):
            assert not diff[c, :max(0, tau - c)].any()
            assert diff[c, max(0, tau - c)]


def test_llsa_paper_rejects_bad_arguments():
    x = llsa_inputs(1, 20, 1, 64, 46, dtype="bf16", channels=3)
    q, k, v = (to_gpu(x[n], "bf16") for n in ("q", "k", "v"))
    with pytest.raises(bd.SAError):
        bd.llsa_paper_forward(q, k, v, 4, 3)  # three channels, La = 3 needs four
    big = torch.zeros(66, 1, 4, 1, 64, dtype=torch.bfloat16, device="cuda")
    with pytest.raises(bd.SAError):
        bd.llsa_paper_forward(big, big, big, 4, 65)  # La beyond the maximum
