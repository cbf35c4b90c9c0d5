"""Streaming inference through a stack of attention layers, one frame per step.

Each layer maps its input features (``[S][H*d]`` per frame) to q, k and v with
a fixed linear map (``W[l]``: ``[3][H*d][H*d]``), then runs one streaming
attention step through the library:

* ``"sa"``: ``sa_stream_step``. A layer emits frame t La steps after frame t
  entered it, so frame t enters layer l at step t + l La and leaves the top of
  an L-layer stack at step t + L La: the look-ahead latency grows with depth.
* ``"llsa"``: ``llsa_stream_step`` (the two-branch LLSA, Eq. 14/15). At step u
  every layer takes branch C's frame u and branch L's frame u - La and emits
  its causal output of frame u and its look-ahead output of frame u - La,
  which are the next layer's branch C and branch L frames of the same step.
  The model input feeds branch C with frame u and branch L with frame u - La
  (kept in a ring of La + 1 input frames), so the top look-ahead output of
  frame t leaves at step t + La for any depth.

Every step of the attention runs in the library's kernels; the projections
are torch matrix products (model plumbing around the measured path).
"""

from __future__ import annotations

from typing import List, Optional

import torch

from . import binding as bd


class StackedStream:
    def __init__(self, kind: str, W: List[torch.Tensor], S: int, H: int, d: int, Lb: int,
                 La: int, lengths=None, dtype=torch.bfloat16, device="cuda"):
        if kind not in ("sa", "llsa"):
            raise ValueError("kind must be 'sa' or 'llsa'")
        self.kind, self.S, self.H, self.d, self.Lb, self.La = kind, S, H, d, Lb, La
        self.W = [w.to(device=device, dtype=dtype).contiguous() for w in W]
        self.layers = len(W)
        if kind == "sa":
            self.states = [bd.StreamState(S, H, d, Lb, La, lengths=lengths, dtype=dtype,
                                          device=device) for _ in W]
            for l, st in enumerate(self.states):
                st.step_ctr.fill_(-l * La)  # frame t enters layer l at step t + l La
        else:
            self.states = [bd.LlsaStreamState(S, H, d, Lb, La, lengths=lengths, dtype=dtype,
                                              device=device) for _ in W]
            # the model input's last La + 1 frames, for branch L of the first layer
            self.inputs = torch.zeros((La + 1, S, H * d), dtype=dtype, device=device)
        self.u = 0

    def _proj(self, l: int, x: torch.Tensor):
        f = x.reshape(self.S, self.H * self.d)
        return [(f @ self.W[l][i]).view(self.S, self.H, self.d) for i in range(3)]

    def step(self, x: Optional[torch.Tensor]):
        """Feeds the model input's frame u (``[S][H][d]``; None past the end of
        every stream) and returns ``(out [S][H][d], emitted [S])``: the top
        layer's output and the frame it belongs to (-1: none this step)."""
        if x is None:
            x = torch.zeros((self.S, self.H, self.d), dtype=self.W[0].dtype,
                            device=self.W[0].device)
        u = self.u
        self.u += 1
        if self.kind == "sa":
            f = x
            for l, st in enumerate(self.states):
                q, k, v = self._proj(l, f)
                f, em = bd.sa_stream_step(st, q, k, v)
            return f, em
        self.inputs[u % (self.La + 1)] = x.reshape(self.S, -1)
        fc = x
        fl = self.inputs[(u - self.La) % (self.La + 1)].view(self.S, self.H, self.d)
        for l, st in enumerate(self.states):
            qc, kc, vc = self._proj(l, fc)
            ql, kl, vl = self._proj(l, fl)
            fc, _, fl, em = bd.llsa_stream_step(st, qc, kc, vc, ql, kl, vl)
        return fl, em
