"""Helpers shared by the GPU parity tests: move seeded inputs to the GPU in the
kernel's element type, run the oracle on the identical (rounded) values, and
compare with the tolerance the path is held to."""

import numpy as np
import torch

# relative tolerance, normwise: max|got - ref| / max|ref| (and elementwise
# |got - ref| <= tol * (|ref| + rms(ref))), per output tensor or per
# (sequence, head) slice
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


def assert_slices_close(got, ref, dtype: str, lengths, what: str = "", elementwise: bool = True,
                        zero_atol: float = 0.0, row_scale: bool = False):
    """The criterion per (sequence, head) slice: for tensors ``[..., B, T, H,
    d]`` every slice ``[..., b, :len_b, h, :]`` (one per leading index) must
    have max|got - ref| <= tol * max|ref| over that slice, and, with
    ``elementwise``, every element within tol * (|ref| + rms of the slice's
    ref), or with ``row_scale`` within tol * (max|ref| over the element's row
    + rms of the slice's ref): a bfloat16 gradient element is a sum of
    bfloat16-rounded products the size of its row, so its error scales with
    the row (the first rows of a sequence carry weights near 1 and gradients
    many times the slice's rms). A slice whose reference is zero requires
    max|got| <= zero_atol. Rows past a sequence's end must be exactly zero in
    ``got``."""
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    assert got.shape == ref.shape, (what, got.shape, ref.shape)
    assert np.all(np.isfinite(got)), "%s: non-finite values" % what
    tol = TOL[dtype]
    B, T, H, d = got.shape[-4:]
    g = got.reshape((-1, B, T, H, d))
    r = ref.reshape((-1, B, T, H, d))
    lengths = [int(x) for x in np.asarray(lengths).reshape(-1)]
    for c in range(g.shape[0]):
        for b in range(B):
            L = min(max(lengths[b], 0), T)
            assert np.all(g[c, b, L:] == 0), "%s: padding rows of [%d, %d] not zero" % (what, c, b)
            if L == 0:
                continue
            gs = g[c, b, :L].transpose(1, 0, 2)  # [H][L][d]
            rs = r[c, b, :L].transpose(1, 0, 2)
            scale = np.abs(rs).reshape(H, -1).max(axis=1)
            err = np.abs(gs - rs)
            emax = err.reshape(H, -1).max(axis=1)
            for h in range(H):
                if scale[h] == 0.0:
                    assert emax[h] <= zero_atol, "%s [%d, b=%d, h=%d]: %.3g > %.3g" % (
                        what, c, b, h, emax[h], zero_atol)
                    continue
                rel = emax[h] / scale[h]
                assert rel <= tol, "%s [%d, b=%d, h=%d]: slice error %.3g > %.1g" % (
                    what, c, b, h, rel, tol)
                if elementwise:
                    rms = float(np.sqrt(np.mean(rs[h] ** 2)))
                    if row_scale:
                        bound = tol * (np.abs(rs[h]).max(axis=1, keepdims=True) + rms)
                    else:
                        bound = tol * (np.abs(rs[h]) + rms)
                    bad = err[h] > bound
                    assert not bad.any(), "%s [%d, b=%d, h=%d]: %d elements outside tolerance, " \
                        "first at (t, i) = %s" % (what, c, b, h, int(bad.sum()),
                                                  np.argwhere(bad)[0])


def round_to(x: np.ndarray, dtype: str) -> np.ndarray:
    """x rounded to the element type (nearest even), back in float64."""
    return torch.from_numpy(np.ascontiguousarray(x)).to(TORCH_DTYPE[dtype]).double().numpy()


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
