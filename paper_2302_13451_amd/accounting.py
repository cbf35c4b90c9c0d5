"""Work and traffic accounting for the band-attention kernels.

These are the algorithmic counts the benchmark divides by measured time: only
the useful band work is counted (no recomputation, no tile waste), and only
valid frames are counted as traffic (zero-filling of padding frames is not).

* Band size: SA restricts each query to the keys t-B .. t+A (Eq. 4), clipped
  here to the valid frames [0, len). ``window_width_sum`` is the exact number
  of (query, key) pairs over a sequence.
* Cost: SA computes O(d_k N_T (A+B+1)) work against O(d_k N_T^2) for masked
  acausal attention (Section "Lower Compute Bound"); ``dense_scores`` and
  ``band_scores_unclipped`` give the two score counts of the worked example in
  Section "Masked Acausal Attention".
"""

from __future__ import annotations

from typing import Iterable

ELEM_BYTES = {"bf16": 2, "f32": 4}


def _seq_width_sum(L: int, Lb: int, La: int) -> int:
    """Sum over t in [0, L) of min(L-1, t+La) - max(0, t-Lb) + 1 (closed form)."""
    if L <= 0:
        return 0
    m = max(0, L - La)  # rows whose look-ahead is not cut by the sequence end
    upper = m * (m - 1) // 2 + m * (La + 1) + (L - m) * L
    n = max(0, L - 1 - Lb)  # rows whose look-back is not cut by the sequence start
    lower = n * (n + 1) // 2
    return upper - lower


def window_width_sum(lengths: Iterable[int], Lb: int, La: int) -> int:
    """Number of (query, key) pairs of SA over all sequences (one head)."""
    return sum(_seq_width_sum(int(L), int(Lb), int(La)) for L in lengths)


def llsa_width_sums(lengths: Iterable[int], Lb: int, La: int):
    """(causal output, look-ahead output) pair counts of the two-branch LLSA.

    The causal output reads [t-La-Lb, t]; the look-ahead output reads
    [t-Lb, t+La]; both clipped to [0, len)."""
    lengths = list(lengths)
    return (window_width_sum(lengths, Lb + La, 0), window_width_sum(lengths, Lb, La))


def dense_scores(T: int) -> int:
    """Scores computed by masked acausal attention for one sequence and head."""
    return T * T


def band_scores_unclipped(T: int, W: int) -> int:
    """Scores used when every mask vector holds W ones (edges not clipped)."""
    return T * W


def sa_forward_flops(lengths, H: int, d: int, Lb: int, La: int) -> int:
    """2 flops per multiply-add for q.k and for a.v over every band pair."""
    return 4 * d * H * window_width_sum(lengths, Lb, La)


def sa_backward_flops(lengths, H: int, d: int, Lb: int, La: int) -> int:
    """dP = dO V^T, dV = P^T dO, dQ = dS K, dK = dS^T Q over every band pair
    (the recomputation of the scores is not counted)."""
    return 8 * d * H * window_width_sum(lengths, Lb, La)


def llsa_forward_flops(lengths, H: int, d: int, Lb: int, La: int) -> int:
    c, l = llsa_width_sums(lengths, Lb, La)
    return 4 * d * H * (c + l)


def llsa_backward_flops(lengths, H: int, d: int, Lb: int, La: int) -> int:
    """The SA backward's products over both outputs' windows."""
    c, l = llsa_width_sums(lengths, Lb, La)
    return 8 * d * H * (c + l)


def llsa_paper_width_sums(lengths: Iterable[int], Lb: int, La: int):
    """Pair counts of the (La+1)-channel LLSA, one per output channel c: the
    window t+c-La-Lb .. t+c clipped to [0, len)."""
    lengths = list(lengths)
    return [window_width_sum(lengths, La + Lb - c, c) for c in range(La + 1)]


def llsa_paper_forward_flops(lengths, H: int, d: int, Lb: int, La: int) -> int:
    return 4 * d * H * sum(llsa_paper_width_sums(lengths, Lb, La))


def llsa_paper_backward_flops(lengths, H: int, d: int, Lb: int, La: int) -> int:
    return 8 * d * H * sum(llsa_paper_width_sums(lengths, Lb, La))


def valid_frames(lengths) -> int:
    return sum(int(L) for L in lengths)


def sa_forward_bytes(lengths, H: int, d: int, dtype: str = "bf16", with_lse: bool = True) -> int:
    """q, k, v read and out written once per valid frame; lse written (fp32)."""
    f = valid_frames(lengths)
    e = ELEM_BYTES[dtype]
    return 4 * f * H * d * e + (4 * f * H if with_lse else 0)


def sa_backward_bytes(lengths, H: int, d: int, dtype: str = "bf16") -> int:
    """q, k, v, out, dout and lse read; dq, dk, dv written; once per valid frame."""
    f = valid_frames(lengths)
    e = ELEM_BYTES[dtype]
    return 8 * f * H * d * e + 4 * f * H


def llsa_forward_bytes(lengths, H: int, d: int, dtype: str = "bf16", with_lse: bool = True) -> int:
    """Both branches' q, k, v read, both outputs (and lse) written."""
    f = valid_frames(lengths)
    e = ELEM_BYTES[dtype]
    return 8 * f * H * d * e + (2 * 4 * f * H if with_lse else 0)


def llsa_backward_bytes(lengths, H: int, d: int, dtype: str = "bf16") -> int:
    """Both outputs' q, out, dout and lse and both branches' k, v read; dq, dk,
    dv of both written; once per valid frame."""
    f = valid_frames(lengths)
    e = ELEM_BYTES[dtype]
    return 16 * f * H * d * e + 2 * 4 * f * H


def llsa_paper_forward_bytes(lengths, H: int, d: int, La: int, dtype: str = "bf16") -> int:
    """Every channel's q, k, v read and out and lse written once per valid
    frame: La + 1 times the SA forward's bytes."""
    return (La + 1) * sa_forward_bytes(lengths, H, d, dtype)


def llsa_paper_backward_bytes(lengths, H: int, d: int, La: int, dtype: str = "bf16") -> int:
    """La + 1 times the SA backward's bytes."""
    return (La + 1) * sa_backward_bytes(lengths, H, d, dtype)


def sa_training_tensor_bytes(T: int, H: int, d: int, dtype: str = "bf16") -> int:
    """Bytes of every tensor of one sequence in an SA layer's forward +
    backward through the library: q, k, v, dout, out, dq, dk, dv and lse (no
    score, weight or mask tensor is kept)."""
    return 8 * T * H * d * ELEM_BYTES[dtype] + 4 * T * H


def stream_step_pairs(window_widths: Iterable[int], H: int) -> int:
    return H * sum(int(w) for w in window_widths)


def stream_step_bytes(window_widths: Iterable[int], appended: int, H: int, d: int,
                      dtype: str = "bf16") -> int:
    """One streaming step: each emitting stream reads its query and the keys and
    values of its window and writes its output row; each accepting stream reads
    its new frame (q, k, v) and writes it into the rings."""
    e = ELEM_BYTES[dtype]
    widths = [int(w) for w in window_widths]
    emit = len(widths)
    row = H * d * e
    return (2 * emit * row + 2 * sum(widths) * row  # query + out + window keys/values
            + appended * 6 * row)               # new frame read + ring writes


def stream_step_flops(window_widths: Iterable[int], H: int, d: int) -> int:
    return 4 * d * stream_step_pairs(window_widths, H)


def llsa_stream_step_bytes(window_widths: Iterable[int], appended: int, H: int, d: int,
                           dtype: str = "bf16") -> int:
    """One two-branch LLSA streaming step: each emitting stream reads its two
    queries and the keys and values of the shared window and writes its two
    output rows; each accepting stream reads the new key and value of both
    branches and writes them into the rings."""
    e = ELEM_BYTES[dtype]
    widths = [int(w) for w in window_widths]
    row = H * d * e
    return (4 * len(widths) * row + 2 * sum(widths) * row  # queries + outputs + window
            + appended * 8 * row)                         # two branches' k, v in and out


def llsa_stream_step_flops(window_widths: Iterable[int], H: int, d: int) -> int:
    """Two outputs (causal and look-ahead) over each emitting stream's window."""
    return 2 * 4 * d * stream_step_pairs(window_widths, H)
