"""GPU parity of llsa_paper_forward (the paper's LLSA with La + 1 channels,
each computed with its own query, Eq. 14/15 in the convention of Fig. 4)
against the fp64 oracle's general channel form, which the Fig. 4 worked
example pins."""

import numpy as np
import pytest
import torch

from paper_2302_13451_amd import binding as bd
from paper_2302_13451_amd.inputs import llsa_inputs
from parity import assert_close, assert_lse_close, assert_slices_close, f64, round_to, to_gpu

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


def check(out, lse, yr, lr, lengths, dtype):
    assert_slices_close(out, yr, dtype, lengths, "out")
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
    (2, 110, 2, 64, 30, 15, (40, 110)),  # the widest look-ahead of the one-tile diagonal pass
    (2, 110, 2, 32, 30, 16, (40, 110)),  # and one past it
    # bfloat16 look-backs of 80 frames and more take the band passes and the
    # merge instead of the one-pass kernel: both sides of that switch, and
    # wide look-backs with short and long look-aheads
    (2, 200, 2, 64, 79, 8, (60, 200)),
    (2, 200, 2, 64, 80, 8, (60, 200)),
    (2, 200, 2, 64, 90, 8, (60, 200)),
    (2, 220, 2, 32, 100, 4, (1, 220)),
    (2, 260, 2, 64, 150, 15, (100, 260)),
    (2, 140, 2, 64, 120, 1, (90, 140)),
])
@pytest.mark.parametrize("scale", ["rsqrt_d", "unit"])
def test_llsa_paper_parity(oracle_mod, dtype, B, T, H, d, Lb, La, lengths, scale):
    check(*run(oracle_mod, B, T, H, d, Lb, La, dtype, 41, lengths, scale), dtype)


def test_llsa_paper_config4_shape(oracle_mod):
    """bf16, B=16, T=800, H=12, d=64, Lb=64, La=8 (nine channels), lengths
    U[400, 800]: the benchmarked shape, every (channel, sequence, head) slice
    element by element."""
    check(*run(oracle_mod, 16, 800, 12, 64, 64, 8, "bf16", 5, (400, 800)), "bf16")


def test_llsa_paper_padded_frames_are_never_read(oracle_mod):
    out, lse, yr, lr, ln = run(oracle_mod, 3, 160, 2, 64, 24, 5, "bf16", 43, (40, 159),
                               pad=float("nan"))
    check(out, lse, yr, lr, ln, "bf16")
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


# ---------------------------------------------------------------------------
# backward


# Each backward case runs twice, as for the SA backward: with the oracle's
# forward output (rounded to bfloat16) and log-sum-exp supplied to both sides,
# per (channel, sequence, head) slice normwise and element by element against
# the row's scale; and end to end against the exact gradient, per channel
# tensor normwise (the rounding of `out` to bfloat16 alone moves a slice of dq
# by about 2e-2 of its maximum).
def run_bwd(oracle_mod, B, T, H, d, Lb, La, seed, lengths, scale="rsqrt_d", pad=0.0,
            supplied=False, dtype="bf16"):
    print("llsa paper backward %s case B=%d T=%d H=%d d=%d Lb=%d La=%d %s seed=%d" % (
        "supplied-output" if supplied else "end-to-end", B, T, H, d, Lb, La, dtype, seed),
        flush=True)
    x = llsa_inputs(B, T, H, d, seed, dtype=dtype, scale=scale, lengths=lengths, pad_value=pad,
                    with_dout=True, channels=La + 1)
    q, k, v, do = (to_gpu(x[n], dtype) for n in ("q", "k", "v", "dout"))
    ln = x["lengths"].cuda()
    clean = {n: np.nan_to_num(f64(x[n])) for n in ("q", "k", "v", "dout")}
    L = x["lengths"].numpy()
    y = None
    if supplied:
        y, lse = oracle_mod.llsa_paper(clean["q"], clean["k"], clean["v"], Lb, La, L)
        y = round_to(y, dtype)
        out, lse = torch.from_numpy(y).to(q.dtype).cuda(), torch.from_numpy(lse).float().cuda()
    else:
        out, lse = bd.llsa_paper_forward(q, k, v, Lb, La, ln)
    dq, dk, dv = bd.llsa_paper_backward(q, k, v, out, lse, do, Lb, La, ln)
    torch.cuda.synchronize()
    ref = oracle_mod.llsa_paper_backward(clean["q"], clean["k"], clean["v"], clean["dout"], Lb, La,
                                         L, y=y)
    return (f64(dq), f64(dk), f64(dv)), ref, x["lengths"].tolist()


def check_bwd(got, ref, lengths, mode="supplied", dtype="bf16"):
    """mode: "supplied" (per slice and element) or "tensors" (per channel
    tensor; float32 end to end is held per slice and element too)."""
    zero_atol = 1e-5 * float(np.max(np.abs(ref[2])))
    for name, g, r in zip(("dq", "dk", "dv"), got, ref):
        if mode == "tensors" and dtype == "bf16":
            for c in range(g.shape[0]):
                assert_close(g[c], r[c], "bf16", "%s channel %d" % (name, c), elementwise=False,
                             zero_atol=zero_atol)
        else:
            assert_slices_close(g, r, dtype, lengths, name, zero_atol=zero_atol,
                                row_scale=dtype == "bf16")


def run_check_bwd(oracle_mod, B, T, H, d, Lb, La, seed, lengths, scale="rsqrt_d", pad=0.0,
                  dtype="bf16"):
    got, ref, L = run_bwd(oracle_mod, B, T, H, d, Lb, La, seed, lengths, scale, pad, supplied=True,
                          dtype=dtype)
    check_bwd(got, ref, L, "supplied", dtype)
    got, ref, L = run_bwd(oracle_mod, B, T, H, d, Lb, La, seed, lengths, scale, pad, dtype=dtype)
    check_bwd(got, ref, L, "tensors", dtype)
    return got, L


@pytest.mark.parametrize("B,T,H,d,Lb,La,lengths", [
    (2, 150, 2, 64, 30, 1, (40, 150)),   # the paper's two-channel module
    (2, 130, 2, 32, 21, 3, (1, 130)),
    (2, 190, 2, 64, 64, 8, (50, 190)),   # nine channels, the widest band at La = 8
    (2, 120, 2, 64, 37, 4, (60, 120)),   # odd channel count: the last pair has one output
    (1, 90, 2, 64, 0, 5, "full"),        # band of one frame
    (2, 100, 1, 64, 17, 0, (30, 100)),   # one channel: the SA backward
    (2, 160, 2, 64, 24, 16, (60, 160)),
    (2, 140, 1, 64, 13, 33, (50, 140)),  # pairs past the first 16 rows of the bands
    (2, 150, 1, 32, 150, 50, (70, 150)),
    (3, 9, 2, 64, 5, 12, (0, 9, 4)),     # look-ahead longer than the sequences
    (66, 40, 1, 32, 10, 2, (0, 40)),
    (2, 110, 2, 64, 40, 15, (40, 110)),  # the widest look-ahead of the one-tile diagonal pass
    (2, 110, 2, 32, 40, 16, (40, 110)),  # and one past it
    (2, 200, 2, 64, 80, 8, (60, 200)),   # wide bands at nine channels
    (2, 200, 2, 64, 81, 8, (60, 200)),
    (3, 300, 2, 32, 75, 11, (300, 1, 170)),
])
@pytest.mark.parametrize("scale", ["rsqrt_d", "unit"])
def test_llsa_paper_backward_parity(oracle_mod, B, T, H, d, Lb, La, lengths, scale):
    run_check_bwd(oracle_mod, B, T, H, d, Lb, La, 52, lengths, scale)


def test_llsa_paper_backward_config4_shape(oracle_mod):
    """bf16, B=16, T=800, H=12, d=64, Lb=64, La=8 (nine channels), lengths
    U[400, 800]: the benchmarked shape."""
    run_check_bwd(oracle_mod, 16, 800, 12, 64, 64, 8, 6, (400, 800))


def test_llsa_paper_backward_padded_frames_are_never_read(oracle_mod):
    got, lengths = run_check_bwd(oracle_mod, 3, 180, 2, 64, 30, 6, 53, (40, 179),
                                 pad=float("nan"))
    for g in got:
        for b, L in enumerate(lengths):
            assert (g[:, b, L:] == 0).all()


def test_llsa_paper_backward_one_channel_is_sa_backward():
    """La = 0: bit-identical to sa_backward with the window t-Lb .. t."""
    x = llsa_inputs(2, 140, 2, 64, 54, dtype="bf16", lengths=(60, 140), with_dout=True,
                    channels=1)
    q, k, v, do = (to_gpu(x[n], "bf16") for n in ("q", "k", "v", "dout"))
    ln = x["lengths"].cuda()
    out, lse = bd.llsa_paper_forward(q, k, v, 33, 0, ln)
    got = bd.llsa_paper_backward(q, k, v, out, lse, do, 33, 0, ln)
    ref = bd.sa_backward(q[0], k[0], v[0], out[0], lse[0], do[0], 33, 0, ln)
    for g, r in zip(got, ref):
        assert torch.equal(g[0], r)


# Windows the band pass cannot stage (the vector-ALU kernel), float32, and
# the staged-window boundary: Lb + La = 64 stages, 65 with La = 16 does not.
@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("B,T,H,d,Lb,La,lengths", [
    (1, 200, 1, 64, 70, 20, "full"),
    (2, 130, 2, 64, 48, 16, (40, 130)),
    (2, 130, 2, 64, 49, 16, (40, 130)),
    (2, 120, 1, 32, 150, 40, (50, 120)),
    (2, 100, 2, 64, 20, 3, (0, 100)),
])
def test_llsa_paper_backward_every_window(oracle_mod, dtype, B, T, H, d, Lb, La, lengths):
    run_check_bwd(oracle_mod, B, T, H, d, Lb, La, 58, lengths, "unit", dtype=dtype)
