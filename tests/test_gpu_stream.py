"""GPU parity of sa_stream_step: the ring-buffer streaming step against the
oracle's ring simulation, against SA over the whole sequence at the streaming
benchmark shape, and under HIP-graph replay."""

import numpy as np
import pytest
import torch

from paper_2302_13451_amd import binding as bd
from paper_2302_13451_amd.inputs import stream_inputs
from parity import TORCH_DTYPE, assert_close, f64

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("S,H,d,Lb,La,R_extra,lengths", [
    (3, 2, 64, 6, 2, 0, [9, 20, 1]),
    (4, 12, 64, 64, 8, 0, [100, 85, 3, 0]),
    (2, 3, 32, 5, 0, 3, [30, 12]),
    (2, 9, 32, 0, 4, 1, [17, 25]),
    (2, 2, 64, 70, 1, 0, None),
])
def test_stream_matches_oracle_ring(oracle_mod, dtype, S, H, d, Lb, La, R_extra, lengths):
    print("stream case S=%d H=%d d=%d Lb=%d La=%d %s" % (S, H, d, Lb, La, dtype), flush=True)
    R = Lb + La + 1 + R_extra
    steps = (max(lengths) if lengths else 90) + La + 2
    x = stream_inputs(steps, S, H, d, 41, dtype=dtype, scale="unit", lengths=lengths)
    st = bd.StreamState(S, H, d, Lb, La, R, lengths, dtype=TORCH_DTYPE[dtype])
    ref = oracle_mod.StreamOracle(S, H, d, Lb, La, R, lengths)
    qg, kg, vg = (x[n].to(TORCH_DTYPE[dtype]).cuda() for n in ("q", "k", "v"))
    for u in range(steps):
        out, em = bd.sa_stream_step(st, qg[u], kg[u], vg[u])
        ro, re = ref.step(f64(x["q"][u]), f64(x["k"][u]), f64(x["v"][u]))
        assert np.array_equal(em.cpu().numpy(), re), u
        assert_close(f64(out), ro, dtype, "step %d" % u)
    assert np.array_equal(st.step_ctr.cpu().numpy(), ref.step_ctr)


def test_config5_full_size_against_sa(oracle_mod):
    """64 open-ended streams, H=12, d=64, ring of 64 past + 8 look-ahead + the
    current frame, 1000 steps: every emitted row equals SA's row of the whole
    sequence."""
    S, H, d, Lb, La, steps = 64, 12, 64, 64, 8, 1000
    R = Lb + La + 1
    x = stream_inputs(steps, S, H, d, 5, dtype="bf16")
    st = bd.StreamState(S, H, d, Lb, La, R)
    qg, kg, vg = (x[n].to(torch.bfloat16).cuda() for n in ("q", "k", "v"))
    outs = torch.empty(steps, S, H, d, dtype=torch.bfloat16, device="cuda")
    ems = torch.empty(steps, S, dtype=torch.int32, device="cuda")
    for u in range(steps):
        out, em = bd.sa_stream_step(st, qg[u], kg[u], vg[u], out=outs[u])
        ems[u] = em
    ems = ems.cpu().numpy()
    want = np.where(np.arange(steps) >= La, np.arange(steps) - La, -1)
    assert np.array_equal(ems, np.repeat(want[:, None], S, axis=1))
    seq = lambda n: f64(x[n]).transpose(1, 0, 2, 3)  # noqa: E731  [S][steps][H][d]
    y, _ = oracle_mod.sa_forward(seq("q"), seq("k"), seq("v"), Lb, La)
    got = f64(outs[La:]).transpose(1, 0, 2, 3)       # rows 0 .. steps-La-1
    assert_close(got, y[:, :steps - La], "bf16", "stream rows")


def test_graph_replay_advances_and_matches_eager():
    S, H, d, Lb, La, n_capture, replays = 8, 4, 64, 16, 4, 5, 4
    R = Lb + La + 1
    steps = n_capture * replays
    x = stream_inputs(steps, S, H, d, 6, dtype="bf16")
    qg, kg, vg = (x[n].to(torch.bfloat16).cuda() for n in ("q", "k", "v"))
    eager = bd.StreamState(S, H, d, Lb, La, R)
    want = []
    for u in range(steps):
        o, e = bd.sa_stream_step(eager, qg[u], kg[u], vg[u])
        want.append((o.clone(), e.clone()))
    st = bd.StreamState(S, H, d, Lb, La, R)
    inq = torch.zeros(n_capture, S, H, d, dtype=torch.bfloat16, device="cuda")
    ink, inv = torch.zeros_like(inq), torch.zeros_like(inq)
    outs = torch.zeros_like(inq)
    ems = torch.zeros(n_capture, S, dtype=torch.int32, device="cuda")
    # warm the library up on a side state before capture
    side = bd.StreamState(S, H, d, Lb, La, R)
    bd.sa_stream_step(side, inq[0], ink[0], inv[0])
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        for i in range(n_capture):
            _, e = bd.sa_stream_step(st, inq[i], ink[i], inv[i], out=outs[i])
            ems[i].copy_(e)
    for r in range(replays):
        sl = slice(r * n_capture, (r + 1) * n_capture)
        inq.copy_(qg[sl])
        ink.copy_(kg[sl])
        inv.copy_(vg[sl])
        graph.replay()
        torch.cuda.synchronize()
        for i in range(n_capture):
            o, e = want[r * n_capture + i]
            assert torch.equal(outs[i], o), (r, i)
            assert torch.equal(ems[i], e), (r, i)
    assert torch.all(st.step_ctr == steps)
