"""Shared test helpers: move generated inputs to the GPU, run the HIP path through
the C ABI, run the oracle on the same bits, and compare at the stated tolerances.

Tolerances (fixed by the benchmark spec of the parity bar):
* float32 inputs: per token |d loss| and |d lse| <= 1e-5 * max(1, |ref|);
  relative Frobenius error of dH and of dW <= 1e-5;
* bfloat16 inputs: per token |d loss| <= 2e-3 and |d lse| <= 2e-3 (absolute);
  relative Frobenius error of dH and of dW (all shards together) <= 1e-2.
"""
from __future__ import annotations

import numpy as np

import workloads as wl

TOL = {
    "f32": {"loss_rel": 1e-5, "grad_fro": 1e-5},
    "bf16": {"loss_abs": 2e-3, "grad_fro": 1e-2},
}


def to_device(inp: wl.Inputs, device="cuda"):
    import torch

    def dev(x):
        if inp.dtype == "bf16":
            return torch.from_numpy(np.ascontiguousarray(x).view(np.int16)).to(device).view(torch.bfloat16)
        return torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).to(device)

    H = dev(inp.H)
    Ws = [dev(w) for w in inp.W_shards]
    t = torch.from_numpy(inp.targets).to(device)
    return H, Ws, t


def oracle_inputs(inp: wl.Inputs):
    """Exact float64 widening of the bits the GPU receives."""
    H = wl.to_f64(inp.H, inp.dtype)
    Ws = [wl.to_f64(w, inp.dtype) for w in inp.W_shards]
    return H, Ws


def rel_fro(a, b) -> float:
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    den = np.linalg.norm(b)
    num = np.linalg.norm(a - b)
    if den == 0.0:
        return float(num)
    return float(num / den)


def assert_loss_close(dtype: str, got, ref, what: str) -> None:
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    assert got.shape == ref.shape
    assert np.array_equal(np.isnan(got), np.isnan(ref)), f"{what}: NaN pattern differs"
    ok = ~np.isnan(ref)
    err = np.abs(got[ok] - ref[ok])
    if dtype == "f32":
        bound = TOL["f32"]["loss_rel"] * np.maximum(1.0, np.abs(ref[ok]))
    else:
        bound = np.full(err.shape, TOL["bf16"]["loss_abs"])
    if err.size:
        worst = int(np.argmax(err - bound))
        assert np.all(err <= bound), (f"{what}: max err {err.max():.3e} at {worst} "
                                      f"(got {got[ok][worst]!r}, ref {ref[ok][worst]!r})")


def assert_grad_close(dtype: str, got, ref, what: str) -> float:
    e = rel_fro(got, ref)
    assert e <= TOL[dtype]["grad_fro"], f"{what}: relative Frobenius error {e:.3e}"
    return e


def run_gpu(inp: wl.Inputs, g: np.ndarray, strip_elems: int = 0, order=None, check_targets=True):
    """Forward and backward through the C ABI; returns numpy results."""
    import torch

    import paper_2609_14306_amd as vp

    H, Ws, t = to_device(inp)
    order = inp.order if order is None else order
    prob = vp.problem_for(H, Ws, inp.ignore_index, order, 0, strip_elems)
    fwd_b, bwd_b = vp.vp_ce_workspace_size(prob)
    ws = torch.empty(max(fwd_b, bwd_b), dtype=torch.uint8, device=H.device)
    loss = torch.empty(inp.T, dtype=torch.float32, device=H.device)
    lse = torch.empty(inp.T, dtype=torch.float32, device=H.device)
    vp.vp_ce_forward(prob, H, Ws, t, loss, lse, ws)
    bad_fwd = vp.vp_ce_check(ws)
    gd = torch.from_numpy(np.ascontiguousarray(g, dtype=np.float32)).to(H.device)
    dH = torch.empty(inp.T, inp.d, dtype=torch.float32, device=H.device)
    dWs = [torch.empty(w.shape[0], inp.d, dtype=torch.float32, device=H.device) for w in Ws]
    vp.vp_ce_backward(prob, H, Ws, t, lse, gd, dH, dWs, ws)
    bad_bwd = vp.vp_ce_check(ws)
    torch.cuda.synchronize()
    return {
        "loss": loss.cpu().numpy(), "lse": lse.cpu().numpy(), "dH": dH.cpu().numpy(),
        "dW_shards": [x.cpu().numpy() for x in dWs], "bad_fwd": bad_fwd, "bad_bwd": bad_bwd,
        "ws_bytes": (fwd_b, bwd_b),
    }


def run_oracle(inp: wl.Inputs, g: np.ndarray):
    import oracle

    H, Ws = oracle_inputs(inp)
    return oracle.forward_backward(H, Ws, inp.targets, g, inp.ignore_index)


def compare_all(inp: wl.Inputs, got, ref, label: str = "") -> dict:
    dt = inp.dtype
    assert_loss_close(dt, got["loss"], ref["loss"], f"{label} loss")
    assert_loss_close(dt, got["lse"], ref["lse"], f"{label} lse")
    ign = inp.targets == inp.ignore_index
    assert np.all(got["loss"][ign] == 0.0), f"{label}: ignored tokens must have loss exactly 0"
    assert np.all(got["dH"][ign] == 0.0), f"{label}: ignored tokens must have zero dH rows"
    e_dh = assert_grad_close(dt, got["dH"], ref["dH"], f"{label} dH")
    gw = np.concatenate([w.reshape(-1, inp.d) for w in got["dW_shards"]], axis=0)
    rw = np.concatenate([w.reshape(-1, inp.d) for w in ref["dW_shards"]], axis=0)
    e_dw = assert_grad_close(dt, gw, rw, f"{label} dW")
    return {"dH_rel_fro": e_dh, "dW_rel_fro": e_dw}


def strip_layout(T: int, shard_rows, order, Tc: int, Vc: int, tile: int = 256):
    """The backward's cut of the T x V residual as vp_ce_plan_info describes it: token
    chunks of Tc, and each non-empty shard (in visiting order) cut into balanced
    vocabulary chunks of at most Vc rows, tile-aligned.  Returns (token chunks, vocabulary
    chunks) as lists of half-open [lo, hi) ranges; vocabulary ranges are global ids."""
    tok = [(t0, min(T, t0 + Tc)) for t0 in range(0, T, Tc)]
    offs = np.cumsum([0] + list(shard_rows))
    voc = []
    for q in order:
        Vq = int(shard_rows[q])
        if Vq == 0:
            continue
        n = -(-Vq // Vc)
        vc = min(Vc, -(-(-(-Vq // n)) // tile) * tile)
        for v0 in range(0, Vq, vc):
            voc.append((int(offs[q]) + v0, int(offs[q]) + min(Vq, v0 + vc)))
    return tok, voc


def stratified_rows(chunks, per_chunk: int, seed: int) -> np.ndarray:
    """Each chunk's first and last index plus `per_chunk` seeded indices inside it."""
    rng = np.random.default_rng(seed + 15485863)
    out = set()
    for lo, hi in chunks:
        out.update({lo, hi - 1})
        out.update(rng.integers(lo, hi, size=min(per_chunk, hi - lo)).tolist())
    return np.array(sorted(out), dtype=np.int64)
