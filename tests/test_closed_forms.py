"""Closed forms the paper prints, checked against this package's accounting
(the counts the benchmark divides by measured time)."""

import os

import numpy as np
import pytest

from paper_2302_13451_amd import accounting as acc

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def read_kv(name):
    out = {}
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            line = line.strip()
            if line and not line.startswith("#"):
                k, v = line.split()
                out[k] = int(v)
    return out


def test_masking_waste_example():
    """Section "Masked Acausal Attention": N_T = 6000, 120 ones per mask."""
    g = read_kv("maa_waste_example.txt")
    T, W = g["frames"], g["receptive_field"]
    assert acc.dense_scores(T) == g["scores_computed"]
    assert acc.band_scores_unclipped(T, W) == g["scores_used"]
    assert acc.dense_scores(T) - acc.band_scores_unclipped(T, W) == g["scores_replaced"]


def brute_pairs(L, Lb, La):
    return sum(min(L - 1, t + La) - max(0, t - Lb) + 1 for t in range(L))


@pytest.mark.parametrize("Lb,La", [(0, 0), (64, 8), (32, 8), (3, 17), (500, 500), (0, 9)])
def test_window_width_sum_closed_form(Lb, La):
    for L in [0, 1, 2, 5, 8, 9, 40, 73, 74, 400, 800]:
        assert acc.window_width_sum([L], Lb, La) == brute_pairs(L, Lb, La), L


def test_window_width_sum_interior_formula():
    """For L >= Lb + La + 1 the count is (Lb+La+1) L - Lb(Lb+1)/2 - La(La+1)/2."""
    Lb, La = 64, 8
    for L in (73, 600, 800):
        assert acc.window_width_sum([L], Lb, La) == (Lb + La + 1) * L - Lb * (Lb + 1) // 2 - La * (La + 1) // 2


def test_sa_cost_is_linear_in_the_band_and_masked_cost_quadratic():
    """Section "Lower Compute Bound": O(d N_T (A+B+1)) vs O(d N_T^2)."""
    T = 4000
    w1 = acc.window_width_sum([T], 10, 10)
    w2 = acc.window_width_sum([T], 20, 20)
    assert abs(w2 / w1 - 41 / 21) < 0.01
    assert acc.dense_scores(2 * T) == 4 * acc.dense_scores(T)


def test_llsa_width_sums():
    lengths = [400, 555, 800]
    c, l = acc.llsa_width_sums(lengths, 64, 8)
    assert c == sum(brute_pairs(L, 72, 0) for L in lengths)
    assert l == sum(brute_pairs(L, 64, 8) for L in lengths)


def test_byte_accounting():
    lengths = np.array([400, 800])
    f = 1200
    assert acc.sa_forward_bytes(lengths, 12, 64) == 4 * f * 12 * 64 * 2 + 4 * f * 12
    assert acc.sa_backward_bytes(lengths, 12, 64) == 8 * f * 12 * 64 * 2 + 4 * f * 12


def test_llsa_paper_width_sums_brute_force():
    """Pairs of the (La+1)-channel LLSA per channel, counted frame by frame:
    channel c of frame t reads t+c-La-Lb .. t+c clipped to [0, len)."""
    lengths = [0, 1, 7, 30, 64]
    for Lb, La in ((0, 1), (5, 3), (12, 8), (40, 2)):
        got = acc.llsa_paper_width_sums(lengths, Lb, La)
        for c in range(La + 1):
            want = sum(len([tau for tau in range(t + c - La - Lb, t + c + 1) if 0 <= tau < L])
                       for L in lengths for t in range(L))
            assert got[c] == want, (Lb, La, c)
    # with two channels the paper's module is the two-branch one
    assert acc.llsa_paper_width_sums(lengths, 9, 1) == list(acc.llsa_width_sums(lengths, 9, 1))
