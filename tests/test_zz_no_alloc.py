"""vp_ce_forward_noalloc: the forward with the library's own device workspace.

For callers that cannot allocate, the forward can run on a 16 MiB device buffer
that the library holds per device.  It runs the same kernels as vp_ce_forward,
so its loss and lse must equal vp_ce_forward's bit for bit on the same inputs.
Two calls in a row, the second with a smaller problem (the buffer keeps the first
call's contents), each compared with vp_ce_forward through the C ABI."""
import numpy as np
import pytest

import workloads as wl

pytestmark = pytest.mark.gpu


def _forward_both(inp):
    import torch

    import paper_2609_14306_amd as vp
    from helpers import to_device

    H, Ws, t = to_device(inp)
    prob = vp.problem_for(H, Ws, inp.ignore_index, inp.order)
    fwd_b, _ = vp.vp_ce_workspace_size(prob)
    assert fwd_b <= 16 << 20
    ws = torch.empty(fwd_b, dtype=torch.uint8, device=H.device)
    loss = torch.empty(inp.T, dtype=torch.float32, device=H.device)
    lse = torch.empty(inp.T, dtype=torch.float32, device=H.device)
    vp.vp_ce_forward(prob, H, Ws, t, loss, lse, ws)
    loss2 = torch.full((inp.T,), float("nan"), dtype=torch.float32, device=H.device)
    lse2 = torch.full((inp.T,), float("nan"), dtype=torch.float32, device=H.device)
    vp.vp_ce_forward_noalloc(prob, H, Ws, t, loss2, lse2)
    torch.cuda.synchronize()
    return loss.cpu().numpy(), lse.cpu().numpy(), loss2.cpu().numpy(), lse2.cpu().numpy()


def test_noalloc_forward_equals_forward_twice():
    big = wl.make_inputs("longctx_bf16_T32768_d2880_V201088_P8_ring", T=3000, d=640, V=12000,
                         seed=71)
    big = wl.resplit(big, [3000, 0, 5000, 4000], order=[3, 1, 0, 2])
    small = wl.make_inputs("tiny_f32_T256_d256_V2048_P8", T=333, d=96, V=1100, P=3, seed=72)
    small.targets[5] = 1100  # out of range: NaN loss on both paths
    for inp in (big, small):
        loss, lse, loss2, lse2 = _forward_both(inp)
        assert np.array_equal(loss, loss2, equal_nan=True), f"{inp.dtype} T={inp.T}: loss differs"
        assert np.array_equal(lse, lse2), f"{inp.dtype} T={inp.T}: lse differs"
        assert np.all(np.isfinite(lse2))
        print(f"noalloc {inp.dtype} T={inp.T}: bit-identical to vp_ce_forward", flush=True)
    assert np.isnan(loss2[5])
