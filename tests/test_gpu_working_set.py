"""The working set of the fused path is bounded by its fixed buffers, whatever V is.

Sec. 3.2 bounds the logit memory of one meeting by a strip (Eq. (2)), and the
appendix tables report each path's peak allocation above the resident weight and
input ("increment over resident").  Here the only memory the library touches
besides its inputs and outputs is the caller's workspace, whose size
vp_ce_workspace_size gives without looking at V.  A sweep of V at fixed T and d
(T = 4096, d = 2880, V in 8 shards from 32768 to 262144 ids) checks on the GPU
that the declared workspace is the same for every V and that one forward +
backward raises torch's peak allocation above the resident tensors (H, W, targets,
upstream gradient, loss, lse, dH, dW) by at most that workspace plus 1 MiB.
Inputs are seeded draws of the workloads' laws (H ~ N(0, 1), W ~ N(0, 1/d),
uniform targets), made on the GPU with a seeded generator.
"""
import math

import pytest

pytestmark = pytest.mark.gpu

T, D, P = 4096, 2880, 8
VS = (32768, 65536, 131072, 201088, 262144)


def test_workspace_and_peak_flat_in_V():
    import torch

    import paper_2609_14306_amd as vp

    dev = torch.device("cuda")
    rows_seen = []
    results = []
    for V in VS:
        torch.cuda.synchronize()
        torch.cuda.empty_cache()
        gen = torch.Generator(device=dev).manual_seed(V)
        rows = [V // P] * (P - 1) + [V - (P - 1) * (V // P)]
        H = torch.randn(T, D, generator=gen, device=dev).to(torch.bfloat16)
        Ws = [(torch.randn(r, D, generator=gen, device=dev) / math.sqrt(D)).to(torch.bfloat16)
              for r in rows]
        tg = torch.randint(0, V, (T,), generator=gen, device=dev, dtype=torch.int64)
        g = torch.full((T,), 1.0 / T, dtype=torch.float32, device=dev)
        loss = torch.empty(T, dtype=torch.float32, device=dev)
        lse = torch.empty(T, dtype=torch.float32, device=dev)
        dH = torch.empty(T, D, dtype=torch.float32, device=dev)
        dWs = [torch.empty(r, D, dtype=torch.float32, device=dev) for r in rows]
        prob = vp.problem_for(H, Ws)
        fwd_b, bwd_b = vp.vp_ce_workspace_size(prob)
        ws_bytes = max(fwd_b, bwd_b)
        torch.cuda.synchronize()
        base = torch.cuda.memory_allocated()
        torch.cuda.reset_peak_memory_stats()
        ws = torch.empty(ws_bytes, dtype=torch.uint8, device=dev)
        e = [torch.cuda.Event(enable_timing=True) for _ in range(3)]
        e[0].record()
        vp.vp_ce_forward(prob, H, Ws, tg, loss, lse, ws)
        e[1].record()
        vp.vp_ce_backward(prob, H, Ws, tg, lse, g, dH, dWs, ws)
        e[2].record()
        torch.cuda.synchronize()
        rise = torch.cuda.max_memory_allocated() - base
        resident = sum(x.numel() * x.element_size() for x in [H, tg, g, loss, lse, dH] + Ws + dWs)
        assert vp.vp_ce_check(ws) == 0
        assert bool(torch.isfinite(loss).all()) and bool(torch.isfinite(dH).all())
        # rows of the residual sum to zero, so the rows of dW do (bf16 residual: ~1e-3)
        col = sum(w.double().sum(0) for w in dWs)
        fro = math.sqrt(sum(float((w.double() ** 2).sum()) for w in dWs))
        assert float(col.norm()) <= 1e-2 * fro
        results.append((V, ws_bytes, rise, resident, e[0].elapsed_time(e[1]), e[1].elapsed_time(e[2])))
        rows_seen.append(rows)
        print(f"V={V}: workspace {ws_bytes / 2**20:.1f} MiB, peak rise {rise / 2**20:.1f} MiB "
              f"over {resident / 2**20:.0f} MiB resident; forward {e[0].elapsed_time(e[1]):.2f} ms, "
              f"backward {e[1].elapsed_time(e[2]):.2f} ms", flush=True)
        assert rise <= ws_bytes + (1 << 20), (V, rise, ws_bytes)
        del H, Ws, tg, g, loss, lse, dH, dWs, ws
    assert len({r[1] for r in results}) == 1, "the declared workspace depends on V"
