"""Pins of the CPU oracle's two-branch LLSA streaming step (infer_llsa,
Section "Low Latency Streaming Attention", Eq. 14/15): driving the two
branches' rings one step at a time, with branch C's frame u and branch L's
frame u - La arriving at step u, must emit the causal output of every frame
as it arrives and the look-ahead output La steps later, each equal to the
two-branch LLSA output of the whole sequence; stacked layers keep the
look-ahead latency at La frames while stacked SA layers add La per layer
(Tab. 3)."""

import numpy as np
import pytest

from paper_2302_13451_amd.inputs import llsa_inputs


def drive(oracle_mod, x, Lb, La, R, lengths, steps, start=None):
    """Feeds [2][S][T][H][d] inputs (index 0 = branch C, 1 = branch L) and
    returns per-step outputs and emitted frames of both outputs."""
    _, S, T, H, d = x["q"].shape
    st = oracle_mod.LlsaStreamOracle(S, H, d, Lb, La, R, lengths)
    if start is not None:
        st.step_ctr[:] = start
    q, k, v = (x[n] for n in ("q", "k", "v"))
    zero = np.zeros((S, H, d))
    oc = np.zeros((steps, S, H, d))
    ol = np.zeros((steps, S, H, d))
    ec = np.zeros((steps, S), dtype=np.int32)
    el = np.zeros((steps, S), dtype=np.int32)
    for n in range(steps):
        fc, fl = [], []
        for s in range(S):
            u = n + (0 if start is None else start[s])
            fc.append(u if 0 <= u < T else None)
            fl.append(u - La if 0 <= u - La < T else None)
        pick = lambda a, br, fr: np.stack([a[br, s, f] if f is not None else zero[s]  # noqa: E731
                                           for s, f in enumerate(fr)])
        oc[n], ec[n], ol[n], el[n] = st.step(pick(q, 0, fc), pick(k, 0, fc), pick(v, 0, fc),
                                             pick(q, 1, fl), pick(k, 1, fl), pick(v, 1, fl))
    return oc, ec, ol, el, st


@pytest.mark.parametrize("Lb,La,R_extra", [(4, 2, 0), (3, 0, 0), (0, 3, 2), (6, 1, 5), (5, 4, 0)])
def test_llsa_stream_equals_two_branch_forward_bitwise(oracle_mod, Lb, La, R_extra):
    S, T, H, d = 3, 12, 2, 4
    lengths = [7, 12, 1]
    x = llsa_inputs(S, T, H, d, 110, dtype="f32", scale="unit", lengths=lengths)
    x = {n: x[n].double().numpy() for n in ("q", "k", "v")}
    steps = T + La + 2
    oc, ec, ol, el, st = drive(oracle_mod, x, Lb, La, Lb + La + 1 + R_extra, lengths, steps)
    assert np.array_equal(st.step_ctr, np.full(S, steps))
    y, _ = oracle_mod.llsa_two_branch(x["q"], x["k"], x["v"], Lb, La, lengths, threads=1)
    for s, L in enumerate(lengths):
        # the causal output of frame u at step u, the look-ahead one La steps later
        assert all(ec[n, s] == (n if n < L else -1) for n in range(steps))
        assert all(el[n, s] == (n - La if La <= n < L + La else -1) for n in range(steps))
        np.testing.assert_array_equal(oc[:L, s], y[0, s, :L])
        np.testing.assert_array_equal(ol[La:La + L, s], y[1, s, :L])
        assert np.all(oc[ec[:, s] < 0, s] == 0) and np.all(ol[el[:, s] < 0, s] == 0)


def test_llsa_stream_never_reads_padding(oracle_mod):
    S, T, H, d, Lb, La = 2, 10, 1, 4, 3, 2
    lengths = [6, 10]
    x = llsa_inputs(S, T, H, d, 111, dtype="f32", scale="unit", lengths=lengths,
                    pad_value=float("nan"))
    x = {n: x[n].double().numpy() for n in ("q", "k", "v")}
    oc, ec, ol, el, _ = drive(oracle_mod, x, Lb, La, Lb + La + 1, lengths, T + La)
    assert np.all(np.isfinite(oc)) and np.all(np.isfinite(ol))


def test_llsa_stream_staggered_start(oracle_mod):
    """A stream whose counter starts negative joins later: same rows, shifted."""
    S, T, H, d, Lb, La = 2, 8, 1, 3, 2, 2
    x = llsa_inputs(S, T, H, d, 112, dtype="f32", scale="unit")
    x = {n: x[n].double().numpy() for n in ("q", "k", "v")}
    x = {n: np.stack([a[:, 0], a[:, 0]], axis=1) for n, a in x.items()}  # same sequence twice
    delay = 3
    oc, ec, ol, el, _ = drive(oracle_mod, x, Lb, La, Lb + La + 1, [T, T], T + La + delay,
                              start=[0, -delay])
    np.testing.assert_array_equal(oc[delay:, 1], oc[:T + La, 0])
    np.testing.assert_array_equal(ol[delay:, 1], ol[:T + La, 0])
    assert np.all(ec[:delay, 1] == -1) and np.all(el[:delay + La, 1] == -1)


def test_stacked_llsa_keeps_la_latency_stacked_sa_adds_la_per_layer(oracle_mod):
    """Three stacked layers with a fixed linear map between them. LLSA: layer
    l + 1 takes branch C's frame u from layer l's causal output of step u and
    branch L's frame u - La from its look-ahead output of step u, so the top
    layer's look-ahead output of frame t appears at step t + La, and equals the
    stacked batch computation. SA: each layer emits frame t La steps after its
    input frame t, so the top layer's frame t appears at step t + 3 La."""
    T, H, d, Lb, La, layers = 14, 2, 4, 3, 2, 3
    rng = np.random.default_rng(113)
    x = rng.standard_normal((T, H, d))
    W = [rng.standard_normal((3, H * d, H * d)) / np.sqrt(H * d) for _ in range(layers)]

    def proj(l, y):  # y [..., H, d] -> (q, k, v) of layer l
        f = y.reshape(y.shape[:-2] + (H * d,))
        return [(f @ W[l][i]).reshape(y.shape) for i in range(3)]

    # batch reference: both branches of layer 0 see the input
    yc = yl = x
    for l in range(layers):
        pc, pl = proj(l, yc), proj(l, yl)
        q, k, v = (np.stack([pc[i], pl[i]])[:, None] for i in range(3))
        y, _ = oracle_mod.llsa_two_branch(q, k, v, Lb, La, threads=1)
        yc, yl = y[0, 0], y[1, 0]
    # streaming: every layer stepped once per input frame
    sts = [oracle_mod.LlsaStreamOracle(1, H, d, Lb, La, Lb + La + 1, [T]) for _ in range(layers)]
    top = {}
    zero = np.zeros((H, d))
    for n in range(T + La):
        fc = x[n] if n < T else zero          # branch C of layer 0: frame n
        fl = x[n - La] if n >= La else zero   # branch L of layer 0: frame n - La
        for l, st in enumerate(sts):
            pc, pl = proj(l, fc), proj(l, fl)
            oc, ec, ol, el = st.step(*[p[None] for p in pc], *[p[None] for p in pl])
            fc, fl = oc[0], ol[0]
        if el[0] >= 0:
            top[int(el[0])] = (n, fl.copy())
    assert sorted(top) == list(range(T))
    for t, (n, y) in top.items():
        assert n == t + La
        np.testing.assert_allclose(y, yl[t], rtol=1e-12, atol=1e-12)
    # stacked SA: layer l's frame t arrives when the layer below emits it, at
    # step t + l La, so its counter starts at -l La; the top layer emits frame
    # t at step t + layers La
    sas = [oracle_mod.StreamOracle(1, H, d, Lb, La, Lb + La + 1, [T]) for _ in range(layers)]
    for l, st in enumerate(sas):
        st.step_ctr[0] = -l * La
    seen = {}
    for n in range(T + layers * La):
        f = x[n] if n < T else zero
        for l, st in enumerate(sas):
            p = proj(l, f)
            o, e = st.step(*[a[None] for a in p])
            f = o[0]
        if e[0] >= 0:
            seen[int(e[0])] = n
    assert seen == {t: t + layers * La for t in range(T)}
