"""Pins of the CPU oracle's LLSA backward: the exact adjoint of the LLSA
forward (Eq. 14/15; the paper's Eq. 16 gives only its value part). It is
checked against what the mathematics fixes, not against itself:

* central finite differences of the oracle's own forward, L = sum_o dy_o . y_o,
  for the two-branch form, the paper's (A+1)-channel form and the literal
  index form of Eq. 14, with ragged lengths;
* reduction to the SA backward (Eq. 7-13, pinned on its own): with equal
  branches the look-ahead output is SA with (Lb, La) and the causal one SA
  with (Lb + La, 0), so the branch gradients sum to the two SA gradients;
* padding: rows past a sequence's end get zero gradients, and padded inputs
  (NaN here) never reach a valid one.
"""

import numpy as np
import pytest


def _rand(rng, shape):
    return rng.standard_normal(shape)


def _loss(oracle_mod, fwd, q, k, v, dy):
    y, _ = fwd(q, k, v)
    return float(np.sum(y * dy))


def _fd_check(oracle_mod, fwd, bwd, q, k, v, dy, h=1e-6, tol=2e-7):
    dq, dk, dv = bwd(q, k, v, dy)
    for name, x, g in (("q", q, dq), ("k", k, dk), ("v", v, dv)):
        num = np.zeros_like(x)
        it = np.nditer(x, flags=["multi_index"])
        for _ in it:
            i = it.multi_index
            old = x[i]
            x[i] = old + h
            lp = _loss(oracle_mod, fwd, q, k, v, dy)
            x[i] = old - h
            lm = _loss(oracle_mod, fwd, q, k, v, dy)
            x[i] = old
            num[i] = (lp - lm) / (2 * h)
        err = np.max(np.abs(num - g))
        assert err < tol, "d%s differs from finite differences by %g" % (name, err)


@pytest.mark.parametrize("Lb,La,lengths", [(3, 2, [9, 6]), (2, 1, [9, 9]), (4, 3, [5, 9]), (3, 0, [9, 7])])
def test_two_branch_backward_matches_finite_differences(oracle_mod, Lb, La, lengths):
    rng = np.random.default_rng(11 + Lb + 3 * La)
    shape = (2, 2, 9, 1, 3)
    q, k, v, dy = (_rand(rng, shape) for _ in range(4))
    fwd = lambda q, k, v: oracle_mod.llsa_two_branch(q, k, v, Lb, La, lengths, threads=1)
    bwd = lambda q, k, v, dy: oracle_mod.llsa_two_branch_backward(q, k, v, dy, Lb, La, lengths, threads=1)
    _fd_check(oracle_mod, fwd, bwd, q, k, v, dy)


@pytest.mark.parametrize("convention", ["text", "eq14"])
def test_paper_channel_form_backward_matches_finite_differences(oracle_mod, convention):
    Lb, La, lengths = 2, 2, [8, 5]
    rng = np.random.default_rng(5 if convention == "text" else 6)
    shape = (La + 1, 2, 8, 1, 3)
    q, k, v = (_rand(rng, shape) for _ in range(3))
    dy = _rand(rng, shape)
    chans = list(range(La + 1))
    fwd = lambda q, k, v: oracle_mod.llsa_forward(q, k, v, chans, chans, chans, Lb, La, lengths,
                                                   convention, threads=1)
    bwd = lambda q, k, v, dy: oracle_mod.llsa_backward(q, k, v, dy, chans, chans, chans, Lb, La,
                                                       lengths, convention, threads=1)
    _fd_check(oracle_mod, fwd, bwd, q, k, v, dy)


@pytest.mark.parametrize("Lb,La", [(5, 3), (4, 1), (0, 2), (6, 0)])
def test_equal_branches_reduce_to_sa_backward(oracle_mod, Lb, La):
    rng = np.random.default_rng(40 + Lb + La)
    B, T, H, d = 2, 13, 2, 4
    lengths = [13, 9]
    q = _rand(rng, (2, B, T, H, d))
    k1, v1 = _rand(rng, (B, T, H, d)), _rand(rng, (B, T, H, d))
    k = np.stack([k1, k1])
    v = np.stack([v1, v1])
    dy = _rand(rng, (2, B, T, H, d))
    dq, dk, dv = oracle_mod.llsa_two_branch_backward(q, k, v, dy, Lb, La, lengths, threads=1)
    # look-ahead output: SA (Lb, La); causal output: SA (Lb + La, 0)
    dqL, dkL, dvL = oracle_mod.sa_backward(q[1], k1, v1, dy[1], Lb, La, lengths, threads=1)
    dqC, dkC, dvC = oracle_mod.sa_backward(q[0], k1, v1, dy[0], Lb + La, 0, lengths, threads=1)
    np.testing.assert_allclose(dq[1], dqL, rtol=0, atol=1e-12)
    np.testing.assert_allclose(dq[0], dqC, rtol=0, atol=1e-12)
    np.testing.assert_allclose(dk[0] + dk[1], dkL + dkC, rtol=0, atol=1e-12)
    np.testing.assert_allclose(dv[0] + dv[1], dvL + dvC, rtol=0, atol=1e-12)


def test_one_output_gradient_touches_only_its_query(oracle_mod):
    rng = np.random.default_rng(3)
    q, k, v, dy = (_rand(rng, (2, 1, 10, 1, 4)) for _ in range(4))
    dy[0] = 0.0  # only the look-ahead output carries a gradient
    dq, dk, dv = oracle_mod.llsa_two_branch_backward(q, k, v, dy, 3, 2, [10], threads=1)
    assert np.all(dq[0] == 0.0)
    # the look-ahead output reads branch C only for frames after t: frame 0 of
    # branch C is never read by it
    assert np.all(dk[0][:, 0] == 0.0) and np.all(dv[0][:, 0] == 0.0)
    assert np.any(dq[1] != 0.0)


def test_padding_rows_zero_and_padded_inputs_unread(oracle_mod):
    rng = np.random.default_rng(8)
    B, T, H, d = 2, 11, 1, 4
    lengths = [11, 6]
    q, k, v, dy = (_rand(rng, (2, B, T, H, d)) for _ in range(4))
    for x in (q, k, v, dy):
        x[:, 1, 6:] = np.nan
    dq, dk, dv = oracle_mod.llsa_two_branch_backward(q, k, v, dy, 3, 2, lengths, threads=1)
    for g in (dq, dk, dv):
        assert np.all(np.isfinite(g))
        assert np.all(g[:, 1, 6:] == 0.0)


def _fd_check_lse(fwd, bwd, q, k, v, dy, c, h=1e-6, tol=2e-7):
    """Finite differences of L = sum_o dy_o . y_o - sum_(o,t) c_(o,t) lse_(o,t)."""
    dq, dk, dv = bwd(q, k, v, dy)

    def loss():
        y, lse = fwd(q, k, v)
        fin = np.isfinite(lse)
        return float(np.sum(y * dy) - np.sum(np.where(fin, c * np.where(fin, lse, 0.0), 0.0)))

    for name, x, g in (("q", q, dq), ("k", k, dk), ("v", v, dv)):
        num = np.zeros_like(x)
        it = np.nditer(x, flags=["multi_index"])
        for _ in it:
            i = it.multi_index
            old = x[i]
            x[i] = old + h
            lp = loss()
            x[i] = old - h
            lm = loss()
            x[i] = old
            num[i] = (lp - lm) / (2 * h)
        err = np.max(np.abs(num - g))
        assert err < tol, "d%s differs from finite differences by %g" % (name, err)


@pytest.mark.parametrize("form", ["two-branch", "paper"])
def test_supplied_output_gradient(oracle_mod, form):
    """With a supplied output y' = y + delta, the Jacobian product of every row
    moves by -a_j (dy . delta) = the gradient of -(dy . delta) lse (d lse / d z_j
    = a_j): the gradient matches finite differences of
    sum dy . y - sum c lse, c = dy . delta held constant. With delta = 0 it is
    the exact gradient."""
    Lb, La, lengths = 3, 2, [9, 6]
    rng = np.random.default_rng(17 if form == "paper" else 18)
    nb = La + 1 if form == "paper" else 2
    shape = (nb, 2, 9, 1, 3)
    q, k, v, dy = (_rand(rng, shape) for _ in range(4))
    if form == "paper":
        fwd = lambda q, k, v: oracle_mod.llsa_paper(q, k, v, Lb, La, lengths, threads=1)
        bwd = lambda q, k, v, dy, y=None: oracle_mod.llsa_paper_backward(
            q, k, v, dy, Lb, La, lengths, threads=1, y=y)
    else:
        fwd = lambda q, k, v: oracle_mod.llsa_two_branch(q, k, v, Lb, La, lengths, threads=1)
        bwd = lambda q, k, v, dy, y=None: oracle_mod.llsa_two_branch_backward(
            q, k, v, dy, Lb, La, lengths, threads=1, y=y)
    y, _ = fwd(q, k, v)
    for g, r in zip(bwd(q, k, v, dy, y), bwd(q, k, v, dy)):
        np.testing.assert_allclose(g, r, rtol=1e-11, atol=1e-13)
    delta = 0.3 * _rand(rng, y.shape)
    c = np.transpose((dy * delta).sum(axis=-1), (0, 1, 3, 2))  # [nout][B][H][T], as lse
    _fd_check_lse(fwd, lambda q, k, v, dy: bwd(q, k, v, dy, y + delta), q, k, v, dy, c)
