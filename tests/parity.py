"""Helpers shared by the GPU parity tests: move seeded inputs to the GPU in the
kernel's element type, run the oracle on the identical (rounded) values, and
compare with the tolerance the path is held to."""

import numpy as np
import torch

# relative tolerance, normwise: max|got - ref| / max|ref| (and elementwise
# |got - ref| <= tol * (|ref| + rms(ref)))
TOL = {"f32": 1e-5, "bf16": 2e-2}
TORCH_DTYPE = {"f32": torch.float32, "bf16": torch.bfloat16}


def to_gpu(x: torch.Tensor, dtype: str) -> torch.Tensor:
    return x.to(TORCH_DTYPE[dtype]).contiguous().cuda()


def f64(x: torch.Tensor) -> np.ndarray:
    return x.detach().to(torch.float64).cpu().numpy()


def assert_close(got, ref, dtype: str, what: str = "", elementwise: bool = True,
                 zero_atol: float = 0.0):
    """Normwise relative error max|got - ref| / max|ref| <= tol (the criterion
    the path is held to). With ``elementwise`` also every element within
    tol * (|ref| + rms(ref)); gradients skip this, because the error the
    bfloat16 forward output brings into D = dout . out scales with |D|, not with
    the element. An all-zero reference requires max|got| <= zero_atol."""
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    assert got.shape == ref.shape, (what, got.shape, ref.shape)
    assert np.all(np.isfinite(got)), "%s: non-finite values" % what
    tol = TOL[dtype]
    scale = np.max(np.abs(ref))
    if scale == 0.0:
        assert np.max(np.abs(got)) <= zero_atol, "%s: %.3g > %.3g" % (
            what, np.max(np.abs(got)), zero_atol)
        return
    err = np.max(np.abs(got - ref)) / scale
    assert err <= tol, "%s: normwise relative error %.3g > %.1g" % (what, err, tol)
    if not elementwise:
        return
    rms = float(np.sqrt(np.mean(ref ** 2)))
    bad = np.abs(got - ref) > tol * (np.abs(ref) + rms)
    assert not bad.any(), "%s: %d elements outside tolerance, first at %s" % (
        what, int(bad.sum()), np.argwhere(bad)[0])


def assert_lse_close(got, ref, dtype: str, what: str = "lse"):
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    np.testing.assert_array_equal(np.isneginf(got), np.isneginf(ref), err_msg=what)
    fin = np.isfinite(ref)
    # log-sum-exp enters the backward as exp(s - lse): its absolute error is the
    # relative error of the recomputed weights (bf16), relative for float32
    if dtype == "bf16":
        np.testing.assert_allclose(got[fin], ref[fin], rtol=0, atol=1e-3, err_msg=what)
    else:
        np.testing.assert_allclose(got[fin], ref[fin], rtol=1e-5, atol=1e-5, err_msg=what)
