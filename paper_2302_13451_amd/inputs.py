"""Seeded synthetic inputs shared by the tests, the smoke check and the benchmark.

This module only draws random numbers and lays them out; it holds none of the
attention arithmetic. Both the GPU path and the CPU oracle consume what it
returns, so that the two sides always see bit-identical inputs.

Recipe (speech-shaped stand-ins for the paper's LibriSpeech features, which are
not used): draws are float32 N(0, 1) from ``torch.Generator('cpu')`` seeded
with ``seed``, in the fixed order q, k, v, dout, lengths; q, k and v are divided
by sqrt(d) when ``scale == "rsqrt_d"`` (multiplied by ``peak`` for the "peaky"
variant), then rounded to bfloat16 (round-to-nearest-even) when ``dtype`` is
``"bf16"``. Frames at or beyond a sequence's length are overwritten with
``pad_value`` (0 by default; NaN for the canary tests that prove padded frames
are never read).
"""

from __future__ import annotations

import math
from typing import Optional, Sequence, Tuple, Union

import torch

LengthSpec = Union[None, str, Tuple[int, int], Sequence[int]]


def _round(x: torch.Tensor, dtype: str) -> torch.Tensor:
    if dtype == "bf16":
        return x.to(torch.bfloat16).to(torch.float32)
    if dtype == "f32":
        return x
    raise ValueError("dtype must be 'bf16' or 'f32'")


def _scale(scale, d: int) -> float:
    if scale == "rsqrt_d":
        return 1.0 / math.sqrt(d)
    if scale == "unit":
        return 1.0
    return float(scale)


def _draw_lengths(g: torch.Generator, n: int, T: int, lengths: LengthSpec) -> torch.Tensor:
    if lengths is None or lengths == "full":
        return torch.full((n,), T, dtype=torch.int32)
    if isinstance(lengths, tuple) and len(lengths) == 2:
        lo, hi = lengths
        return torch.randint(int(lo), int(hi) + 1, (n,), generator=g, dtype=torch.int64).to(torch.int32)
    arr = torch.as_tensor(list(lengths), dtype=torch.int32)
    if arr.shape != (n,):
        raise ValueError("explicit lengths must have one entry per sequence")
    return arr


def _pad(x: torch.Tensor, lengths: torch.Tensor, value: float, time_dim: int) -> torch.Tensor:
    T = x.shape[time_dim]
    t = torch.arange(T).view([1] * time_dim + [T] + [1] * (x.dim() - time_dim - 1))
    shape = [1] * x.dim()
    shape[time_dim - 1] = lengths.shape[0]
    pad = t >= lengths.view(shape).to(torch.int64)
    return torch.where(pad, torch.full_like(x, value), x)


def sa_inputs(B: int, T: int, H: int, d: int, seed: int, *, dtype: str = "bf16",
              scale="rsqrt_d", peak: float = 1.0, lengths: LengthSpec = "full",
              pad_value: float = 0.0, with_dout: bool = True) -> dict:
    """q, k, v (and dout) as float32 CPU tensors ``[B][T][H][d]`` holding values
    exactly representable in ``dtype``; ``lengths`` as int32 ``[B]``."""
    g = torch.Generator(device="cpu").manual_seed(int(seed))
    s = _scale(scale, d) * float(peak)
    q = torch.randn(B, T, H, d, generator=g) * s
    k = torch.randn(B, T, H, d, generator=g) * s
    v = torch.randn(B, T, H, d, generator=g) * s
    dout = torch.randn(B, T, H, d, generator=g) if with_dout else None
    ln = _draw_lengths(g, B, T, lengths)
    out = {"q": q, "k": k, "v": v, "dout": dout}
    for name in list(out):
        if out[name] is None:
            continue
        x = _round(out[name], dtype)
        out[name] = _pad(x, ln, pad_value, 1)
    out["lengths"] = ln
    return out


def llsa_inputs(B: int, T: int, H: int, d: int, seed: int, *, dtype: str = "bf16",
                scale="rsqrt_d", peak: float = 1.0, lengths: LengthSpec = "full",
                pad_value: float = 0.0, with_dout: bool = False, channels: int = 2) -> dict:
    """Multi-branch q, k, v as float32 CPU tensors ``[channels][B][T][H][d]``
    (two branches by default: index 0 = causal branch, 1 = look-ahead branch;
    ``channels = La + 1`` for the paper's channel form); ``lengths`` int32
    ``[B]``; with ``with_dout`` also the gradient of every output, ``dout``
    N(0, 1) of the same shape, drawn after the lengths (so q, k, v and the
    lengths do not depend on it)."""
    g = torch.Generator(device="cpu").manual_seed(int(seed))
    s = _scale(scale, d) * float(peak)
    q = torch.randn(channels, B, T, H, d, generator=g) * s
    k = torch.randn(channels, B, T, H, d, generator=g) * s
    v = torch.randn(channels, B, T, H, d, generator=g) * s
    ln = _draw_lengths(g, B, T, lengths)
    out = {"q": q, "k": k, "v": v}
    if with_dout:
        out["dout"] = torch.randn(channels, B, T, H, d, generator=g)
    for name in list(out):
        out[name] = _pad(_round(out[name], dtype), ln, pad_value, 2)
    out["lengths"] = ln
    return out


def stream_inputs(steps: int, S: int, H: int, d: int, seed: int, *, dtype: str = "bf16",
                  scale="rsqrt_d", lengths: Optional[Sequence[int]] = None) -> dict:
    """Frames fed to a streaming step: q, k, v float32 ``[steps][S][H][d]``;
    ``lengths`` int32 ``[S]`` or None for open-ended streams."""
    g = torch.Generator(device="cpu").manual_seed(int(seed))
    s = _scale(scale, d)
    q = _round(torch.randn(steps, S, H, d, generator=g) * s, dtype)
    k = _round(torch.randn(steps, S, H, d, generator=g) * s, dtype)
    v = _round(torch.randn(steps, S, H, d, generator=g) * s, dtype)
    ln = None if lengths is None else torch.as_tensor(list(lengths), dtype=torch.int32)
    return {"q": q, "k": k, "v": v, "lengths": ln}
