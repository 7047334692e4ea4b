"""The forward and backward calls under HIP graph capture.

The path launches kernels only: the library allocates nothing, never
synchronises outside vp_ce_check, and clears its workspace header with a kernel
(no memset node).  A graph captured from one forward + backward must therefore
replay to exactly the eager result.  The graph is replayed several times with
eager work of the same library and host synchronisations in between, and every
replay is compared bit for bit with the eager run.
"""
import numpy as np
import pytest

import workloads as wl

pytestmark = pytest.mark.gpu


def test_forward_backward_replay_in_a_graph():
    import torch

    import paper_2609_14306_amd as vp
    from helpers import to_device

    inp = wl.make_inputs("longctx_bf16_T32768_d2880_V201088_P8_ring", T=1000, d=640, V=12000, seed=41)
    inp = wl.resplit(inp, [3000, 0, 5000, 4000], order=[3, 1, 0, 2])
    H, Ws, t = to_device(inp)
    dev = H.device
    T, d = inp.T, inp.d
    g = torch.from_numpy(wl.random_grad_loss(T, 41, "random")).to(dev)
    # a small strip so that the backward runs many stage launches and transposes
    prob = vp.problem_for(H, Ws, inp.ignore_index, inp.order, 0, 256 * 512)
    fwd_b, bwd_b = vp.vp_ce_workspace_size(prob)
    ws = torch.empty(max(fwd_b, bwd_b), dtype=torch.uint8, device=dev)
    loss = torch.empty(T, dtype=torch.float32, device=dev)
    lse = torch.empty(T, dtype=torch.float32, device=dev)
    dH = torch.empty(T, d, dtype=torch.float32, device=dev)
    dWs = [torch.empty(w.shape[0], d, dtype=torch.float32, device=dev) for w in Ws]

    def step():
        vp.vp_ce_forward(prob, H, Ws, t, loss, lse, ws)
        vp.vp_ce_backward(prob, H, Ws, t, lse, g, dH, dWs, ws)

    def snapshot():
        torch.cuda.synchronize()
        return [loss.cpu().numpy().copy(), lse.cpu().numpy().copy(), dH.cpu().numpy().copy()] + \
               [w.cpu().numpy().copy() for w in dWs]

    # eager reference (the path is deterministic: the same launches in the same order)
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        step()
    torch.cuda.current_stream().wait_stream(s)
    ref = snapshot()

    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        step()
    for rep in range(3):
        for x in [loss, lse, dH] + dWs:
            x.fill_(float("nan"))  # the replay must rewrite every output
        graph.replay()
        got = snapshot()
        for a, b in zip(got, ref):
            assert np.array_equal(a, b, equal_nan=True), f"replay {rep} differs from the eager run"
        # eager work of the same library between replays, with a different batch
        other = wl.make_inputs("longctx_bf16_T32768_d2880_V201088_P8_ring", T=77, d=640, V=12000,
                               seed=50 + rep)
        H2, W2, t2 = to_device(other)
        vp.forward(H2, W2, t2)
        torch.cuda.synchronize()
    assert vp.vp_ce_check(ws) == 0
