#!/usr/bin/env python3
"""Benchmark of the fused vocabulary-projection cross-entropy (forward + backward) on one MI355X.

A step is one pass of the whole path over one batch: the fused forward (logits
tiles folded into the online log-sum-exp, target gather, split combine) and the
backward (logits recompute, softmax residual, dH and dW contractions), through
the C ABI on torch's current stream, inputs resident in HBM.

Prints ONE JSON line: tokens/s of the whole job (value), ms per step, achieved
TFLOP/s counted as 8*T*V*d per step (2TVd forward, 6TVd backward with recompute)
against the dense bf16 MFMA peak, the working set, a roofline entry for the
backward stage kernel (the dominant one) and one for the fused forward kernel,
both timed with HIP events on the launch stream, and the CPU oracle timed on a
bounded row sample of the same workload.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2516.6  # MI355X dense bf16 MFMA: 256 CU x 2.4 GHz x 4096 flop/clk
PEAK_F32_TFLOPS = 157.3    # MI355X fp32 (MFMA/vector)
PEAK_HBM_GBS = 8000.0
DEFAULT_WORKLOAD = "longctx_bf16_T32768_d2880_V201088_P8_ring"


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default=DEFAULT_WORKLOAD)
    ap.add_argument("--cpu-sample-rows", type=int, default=4096,
                    help="token rows of the workload the CPU oracle is timed on (at most; fewer "
                         "when V * d is large, so that the sample stays near 20 s of host work)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--strip-elems", type=int, default=0)
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="BYTES",
                    help="only run one device-to-device copy of BYTES (for scaling HBM counters)")
    ap.add_argument("--standard", action="store_true",
                    help="instead of the bench line, compare the fused path with the dense standard "
                         "(full logits, float32 log-softmax cross-entropy, autograd) on the same "
                         "workload: time and peak memory above the resident tensors")
    ap.add_argument("--gemm-reference", action="store_true",
                    help="instead of the bench line, time the fused forward against the library "
                         "GEMM (torch.matmul, i.e. hipBLASLt) of the same logits, alternately, "
                         "on the same operands")
    return ap.parse_args()


def gemm_reference(inp, H, Ws, tg, steps: int, warmup: int):
    """The fused forward against a plain library GEMM of the same operands.  The reference
    computes every shard's logits W_q H^T with torch.matmul (hipBLASLt), written out in the
    input dtype and not folded; the fused forward computes the same products and folds them
    into the online log-sum-exp instead of writing them.  The two alternate, `steps` times
    each after `warmup` rounds, in one process on the same resident operands, and both are
    counted at 2 T V d flops.  The reference is plain torch beside the product, not part of
    it."""
    import numpy as np
    import torch

    import paper_2609_14306_amd as vp

    torch.backends.cuda.matmul.allow_tf32 = False  # float32 products stay float32
    T, d, V = inp.T, inp.d, inp.V
    Ht = H.t()
    C = torch.empty(max(w.shape[0] for w in Ws), T, dtype=H.dtype, device=H.device)
    prob = vp.problem_for(H, Ws, inp.ignore_index, inp.order)
    ws = torch.empty(vp.vp_ce_workspace_size(prob)[0], dtype=torch.uint8, device=H.device)
    loss = torch.empty(T, dtype=torch.float32, device=H.device)
    lse = torch.empty_like(loss)

    def gemm():
        for w in Ws:
            torch.matmul(w, Ht, out=C[: w.shape[0]])

    def fused():
        vp.vp_ce_forward(prob, H, Ws, tg, loss, lse, ws)

    times = {"gemm": [], "fused_forward": []}
    for k in range(warmup + steps):
        for name, fn in (("gemm", gemm), ("fused_forward", fused)):
            e0 = torch.cuda.Event(enable_timing=True)
            e1 = torch.cuda.Event(enable_timing=True)
            e0.record()
            fn()
            e1.record()
            torch.cuda.synchronize()
            if k >= warmup:
                times[name].append(e0.elapsed_time(e1))
    flops = 2.0 * T * V * d
    out = {}
    for name, xs in times.items():
        out[name] = {"median_ms": float(np.median(xs)), "min_ms": float(np.min(xs)),
                     "tflops_at_median": flops / (float(np.median(xs)) * 1e-3) / 1e12}
    out["fused_over_gemm_rate"] = out["gemm"]["median_ms"] / out["fused_forward"]["median_ms"]
    out["gemm_what"] = (f"torch.matmul(W_q, H.t()) for each of the {len(Ws)} shards, "
                        f"{inp.dtype} output")
    return out


def standard_vs_fused(inp, H, Ws, tg, steps: int, warmup: int, keep_outputs: bool = False):
    """The paper's comparison (its standard vs Ring-DTP table of peak memory and latency) on
    one GPU: the dense standard materialises the [T, V] logits (in the input dtype, as torch
    computes the product: bfloat16, or float32 with full float32 products), takes a float32
    log-softmax cross-entropy and backpropagates with autograd; the fused path is this
    library's forward + backward.  Both start from the same resident H, W and targets; memory
    is the peak allocation above them during a step.  The dense path is plain torch, a
    baseline beside the product, not part of it.  Both take the mean of the per-token losses
    over the non-ignored tokens.  With keep_outputs, the result also holds each path's
    per-token loss, dH and dW from its last step (key "outputs", CPU tensors)."""
    import torch
    import torch.nn.functional as F

    import paper_2609_14306_amd as vp

    torch.backends.cuda.matmul.allow_tf32 = False  # float32 products stay float32

    dev = H.device
    T, d, V = inp.T, inp.d, inp.V
    W = torch.cat(Ws, dim=0)  # vocabulary-id order
    n_valid = int((inp.targets != inp.ignore_index).sum())
    out = {}

    def timed(step, pre=None):
        for _ in range(warmup):
            step()
        torch.cuda.synchronize()
        if pre is not None:
            pre()
        base = torch.cuda.memory_allocated()
        torch.cuda.reset_peak_memory_stats()
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(steps):
            step()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / steps, (torch.cuda.max_memory_allocated() - base) / 2**20

    # dense standard; its H / W gradients are allocated by autograd inside the step
    Hs = H.detach().clone().requires_grad_(True)
    Wsd = W.detach().clone().requires_grad_(True)

    dense_last = {}

    def dense_step():
        Hs.grad = None
        Wsd.grad = None
        logits = Hs @ Wsd.t()
        per_tok = F.cross_entropy(logits.float(), tg, ignore_index=inp.ignore_index,
                                  reduction="none")
        (per_tok.sum() / max(n_valid, 1)).backward()
        dense_last["loss"] = per_tok.detach()

    ms, mib = timed(dense_step, pre=lambda: (setattr(Hs, "grad", None), setattr(Wsd, "grad", None)))
    kept = {}
    if keep_outputs:
        kept["standard"] = {"loss": dense_last["loss"].cpu(), "dH": Hs.grad.float().cpu(),
                            "dW": Wsd.grad.float().cpu()}
    dense_last.clear()
    out["standard"] = {"ms_per_step": ms, "peak_above_resident_mib": mib,
                       "what": f"logits = H W^T ({inp.dtype}, [T, V] materialised), "
                               "cross_entropy(logits.float()), autograd backward; includes the dH / dW "
                               "outputs"}
    del Hs, Wsd
    torch.cuda.empty_cache()

    # fused path; dH / dW outputs allocated inside the step like the dense one's gradients
    prob = vp.problem_for(H, Ws, inp.ignore_index, inp.order)
    fwd_b, bwd_b = vp.vp_ce_workspace_size(prob)
    g = torch.full((T,), 1.0 / max(n_valid, 1), dtype=torch.float32, device=dev)

    fused_last = {}

    def fused_step(keep=False):
        ws = torch.empty(max(fwd_b, bwd_b), dtype=torch.uint8, device=dev)
        loss = torch.empty(T, dtype=torch.float32, device=dev)
        lse = torch.empty(T, dtype=torch.float32, device=dev)
        vp.vp_ce_forward(prob, H, Ws, tg, loss, lse, ws)
        dH = torch.empty(T, d, dtype=torch.float32, device=dev)
        dWs = [torch.empty(x.shape[0], d, dtype=torch.float32, device=dev) for x in Ws]
        vp.vp_ce_backward(prob, H, Ws, tg, lse, g, dH, dWs, ws)
        if keep:
            fused_last.update(loss=loss, dH=dH, dW=dWs)

    ms, mib = timed(fused_step)
    if keep_outputs:  # one more step, untimed, whose outputs are kept
        fused_step(keep=True)
        torch.cuda.synchronize()
        kept["fused"] = {"loss": fused_last["loss"].cpu(), "dH": fused_last["dH"].cpu(),
                         "dW": torch.cat(fused_last["dW"], dim=0).cpu()}
        out["outputs"] = kept
    fused_last.clear()
    out["fused"] = {"ms_per_step": ms, "peak_above_resident_mib": mib,
                    "what": "vp_ce_forward + vp_ce_backward; workspace, loss / lse and the dH / dW "
                            "outputs allocated inside the step"}
    out["outputs_mib"] = (T * d * 4 + V * d * 4) / 2**20
    out["dense_logits_fp32_mib"] = T * V * 4 / 2**20
    return out


KERNEL_SOURCE = os.path.join(ROOT, "paper_2609_14306_amd", "csrc", "vpce_kernels.hip")
TRAFFIC_PROFILE = os.path.join(ROOT, "profiles", "hbm_traffic_longctx_T32768_d2880_V201088.md")
MFMA_PROFILE = os.path.join(ROOT, "profiles", "mfma_util_longctx_T32768_d2880_V201088.md")


def kernel_source_sha256() -> str:
    import hashlib
    with open(KERNEL_SOURCE, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()


def profile_values(path: str, workload: str) -> dict:
    """The "- key: `value`" lines of a committed profile summary, or {} when the file is
    missing, covers another workload, or the kernels changed since it was taken."""
    try:
        lines = open(path).read().splitlines()
    except OSError:
        return {}
    vals = {}
    for ln in lines:
        if ln.startswith("- ") and ":" in ln:
            k, v = ln[2:].split(":", 1)
            vals[k.strip()] = v.strip().strip("`")
    if vals.get("workload") != workload or vals.get("kernel_source_sha256") != kernel_source_sha256():
        return {}
    return vals


def measured_traffic(kernel: str, workload: str):
    """HBM bytes per launch of `kernel` from the committed counter profile, or None."""
    v = profile_values(TRAFFIC_PROFILE, workload).get(f"{kernel}_hbm_bytes_per_launch")
    return float(v) if v is not None else None


def measured_clock(kernel: str, workload: str):
    """Clock and MFMA occupancy of `kernel` from the committed counter profile, or None.

    The nameplate MFMA peak assumes 2.4 GHz; `peak_at_clock` is the same peak at the clock the
    counters saw the kernel hold (GRBM_GUI_ACTIVE per XCD over the dispatch duration)."""
    vals = profile_values(MFMA_PROFILE, workload)
    try:
        ghz = float(vals[f"{kernel}_clock_ghz"])
        busy = float(vals[f"{kernel}_mfma_busy"])
    except (KeyError, ValueError):
        return None
    return {"clock_ghz": ghz, "mfma_busy": busy, "peak_at_clock": PEAK_BF16_TFLOPS * ghz / 2.4,
            "source": os.path.relpath(MFMA_PROFILE, ROOT)}


def add_frac_at_clock(roof: dict, dtype: str) -> None:
    """The achieved rate against the MFMA peak at the clock the counters saw (bf16 only: the
    counter profile covers the bf16 long-context workload)."""
    c = roof.get("counters")
    if c is not None and dtype == "bf16":
        c["frac_at_clock"] = roof["achieved"] / c["peak_at_clock"]


def cpu_baseline(inp, rows: int):
    """The oracle as it stands, on the first `rows` tokens (full V and d): its cost is linear in T."""
    import numpy as np

    import oracle
    import workloads as wl

    try:
        from threadpoolctl import threadpool_info
        cores = max([p.get("num_threads", 1) for p in threadpool_info()] or [1])
    except Exception:  # noqa: BLE001
        cores = os.cpu_count() or 1
    # about 1.6e13 float64 operations (6 T V d for the forward and backward products)
    cap = max(256, int(1.6e13 / (6.0 * inp.V * inp.d)) // 256 * 256)
    rows = min(rows, cap, inp.T)
    H = wl.to_f64(inp.H[:rows], inp.dtype)
    Ws = [wl.to_f64(w, inp.dtype) for w in inp.W_shards]
    g = wl.random_grad_loss(rows, 0, "sum")
    t0 = time.perf_counter()
    oracle.forward_backward(H, Ws, inp.targets[:rows], g, inp.ignore_index)
    dt = time.perf_counter() - t0
    cpu_model = None
    try:
        with open("/proc/cpuinfo") as f:
            for ln in f:
                if ln.startswith("model name"):
                    cpu_model = ln.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    return {"value": rows / dt, "unit": "tokens/s", "cores": int(cores), "kind": "oracle",
            "sample": f"first {rows} of {inp.T} tokens at full V={inp.V}, d={inp.d} "
                      f"(float64 forward+backward, {dt:.2f} s)",
            "seconds": dt, "nproc": os.cpu_count(), "cpu_model": cpu_model,
            # the oracle's three products (logits, dH, dW): 6 rows V d float64 operations
            "gflops": 6.0 * rows * inp.V * inp.d / dt / 1e9}


def main():
    args = parse()
    if args.gpus != 1:
        print(json.dumps({"error": "the benchmark runs on exactly one GPU (one device's share of "
                                   "the ring); --gpus must be 1", "n_gpus": args.gpus}))
        sys.exit(2)

    import numpy as np
    import torch

    import paper_2609_14306_amd as vp
    import workloads as wl

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    if args.copy_calibration:
        n = args.copy_calibration // 4
        src = torch.ones(n, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_bytes": n * 4}), flush=True)
        return
    w = wl.WORKLOADS[args.workload]
    t_gen = time.perf_counter()
    inp = wl.make_inputs(w)
    t_gen = time.perf_counter() - t_gen

    def to_dev(x):
        if inp.dtype == "bf16":
            return torch.from_numpy(np.ascontiguousarray(x).view(np.int16)).to(dev).view(torch.bfloat16)
        return torch.from_numpy(np.ascontiguousarray(x)).to(dev)

    H = to_dev(inp.H)
    Ws = [to_dev(x) for x in inp.W_shards]
    tg = torch.from_numpy(inp.targets).to(dev)
    T, d, V = inp.T, inp.d, inp.V
    if args.standard or args.gemm_reference:
        if args.standard:
            res = standard_vs_fused(inp, H, Ws, tg, args.steps, args.warmup)
        else:
            res = gemm_reference(inp, H, Ws, tg, args.steps, args.warmup)
        res.update({"mode": "standard_vs_fused" if args.standard else "gemm_reference",
                    "workload": w.name, "T": T, "d": d, "V": V, "steps": args.steps,
                    "warmup": args.warmup})
        print(json.dumps(res), flush=True)
        return
    n_valid = int((inp.targets != inp.ignore_index).sum())
    g = torch.full((T,), 1.0 / max(n_valid, 1), dtype=torch.float32, device=dev)
    prob = vp.problem_for(H, Ws, inp.ignore_index, inp.order, 0, args.strip_elems)
    fwd_b, bwd_b = vp.vp_ce_workspace_size(prob)
    plan = vp.vp_ce_plan_info(prob)
    ws = torch.empty(max(fwd_b, bwd_b), dtype=torch.uint8, device=dev)
    loss = torch.empty(T, dtype=torch.float32, device=dev)
    lse = torch.empty(T, dtype=torch.float32, device=dev)
    dH = torch.empty(T, d, dtype=torch.float32, device=dev)
    dWs = [torch.empty(x.shape[0], d, dtype=torch.float32, device=dev) for x in Ws]
    stream = torch.cuda.current_stream()

    def step(ev=None):
        if ev is not None:
            ev[0].record(stream)
        vp.vp_ce_forward(prob, H, Ws, tg, loss, lse, ws)
        if ev is not None:
            ev[1].record(stream)
        vp.vp_ce_backward(prob, H, Ws, tg, lse, g, dH, dWs, ws)
        if ev is not None:
            ev[2].record(stream)

    torch.cuda.synchronize()
    base_alloc = torch.cuda.memory_allocated()
    torch.cuda.reset_peak_memory_stats()
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    bad = vp.vp_ce_check(ws)
    extra_alloc = torch.cuda.max_memory_allocated() - base_alloc

    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for k in range(args.steps):
        step(evs[k])
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    fwd_ms = [e[0].elapsed_time(e[1]) for e in evs]
    bwd_ms = [e[1].elapsed_time(e[2]) for e in evs]
    step_ev_ms = [e[0].elapsed_time(e[2]) for e in evs]

    def stats(xs):
        return {"mean": float(np.mean(xs)), "median": float(np.median(xs)), "min": float(np.min(xs)),
                "max": float(np.max(xs))}
    gpu_ms = evs[0][0].elapsed_time(evs[-1][2]) / args.steps
    ms_per_step = max(wall * 1e3 / args.steps, gpu_ms)
    flops = 8.0 * T * V * d
    tflops = flops / (ms_per_step * 1e-3) / 1e12
    peak = PEAK_BF16_TFLOPS if inp.dtype == "bf16" else PEAK_F32_TFLOPS
    fwd_avg = float(np.mean(fwd_ms))
    bwd_avg = float(np.mean(bwd_ms))
    fwd_tflops = 2.0 * T * V * d / (fwd_avg * 1e-3) / 1e12
    bwd_tflops = 6.0 * T * V * d / (bwd_avg * 1e-3) / 1e12
    bwd_traffic = measured_traffic("bwd_stage_kernel", w.name)
    fwd_traffic = measured_traffic("fwd_kernel", w.name)
    out = {
        "metric": "vocab-proj CE fwd+bwd tokens/s; % bf16 MFMA peak; peak working set MiB",
        "value": T / (ms_per_step * 1e-3),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": inp.dtype,
        "data": "synthetic",
        "config": {"workload": w.name, "T": T, "d": d, "V": V, "P": len(Ws), "order": inp.order,
                   "target_law": w.target_law, "ignore_frac": w.ignore_frac,
                   "parallelism": "single GPU (one rank's share of the ring)"},
        "tflops": tflops,
        "pct_peak": 100.0 * tflops / peak,
        "fwd_ms": fwd_avg,
        "bwd_ms": bwd_avg,
        # per-step HIP-event times on the launch stream (forward call, backward call, both)
        "timing_ms": {"fwd": stats(fwd_ms), "bwd": stats(bwd_ms), "fwd_bwd": stats(step_ev_ms)},
        "working_set_mib": {"workspace_fwd": fwd_b / 2**20, "workspace_bwd": bwd_b / 2**20,
                            "allocated_during_steps": extra_alloc / 2**20,
                            "peak_over_resident": (max(fwd_b, bwd_b) + extra_alloc) / 2**20},
        # The dominant kernel by time: the backward stage kernel (recompute + residual,
        # dH and dW tiles), launched once per strip plus once.  Its average launch
        # carries 6TVd / launches flops; its average duration is taken as the backward
        # call's event time over the launch count (the call also holds the H and W
        # transposes, about 0.5% of it, so achieved is slightly understated).
        "roofline": {"kernel": "bwd_stage_kernel (logits recompute + residual + dH + dW MFMA tiles)",
                     "bound": "mfma", "achieved": bwd_tflops, "peak": peak, "unit": "TFLOP/s",
                     "frac": bwd_tflops / peak, "traffic": bwd_traffic,
                     "launches_per_step": plan["stage_launches"],
                     "flops_per_launch": 6.0 * T * V * d / max(plan["stage_launches"], 1),
                     "avg_launch_ms": bwd_avg / max(plan["stage_launches"], 1),
                     "strip": {"Tc": plan["Tc"], "Vc": plan["Vc"], "strips": plan["strips"]},
                     "counters": measured_clock("bwd_stage_kernel", w.name)},
        "roofline_fwd": {"kernel": "fwd_kernel (fused logits tiles + online LSE fold)",
                         "bound": "mfma", "achieved": fwd_tflops, "peak": peak, "unit": "TFLOP/s",
                         "frac": fwd_tflops / peak, "traffic": fwd_traffic, "launches_per_step": 1,
                         "flops_per_launch": 2.0 * T * V * d, "avg_launch_ms": fwd_avg,
                         "counters": measured_clock("fwd_kernel", w.name)},
        "bad_targets": bad,
        "input_gen_s": t_gen,
        # The paper's own figures for this path (context, not a target: other hardware, FP32,
        # eight GPUs): peak allocation of the projection forward + backward per rank, standard
        # dense projection against Ring-DTP (Sec. 3.2 results table, App. C peak table).
        "paper_context": {"hardware": "one node of 8x NVIDIA H200, FP32",
                          "shape": "N=16384 tokens per rank, H=7168, V=200000, P=8",
                          "projection_peak_gib": {"standard": 42.462, "ring_dtp": 7.322},
                          "increment_over_resident_gib": {"standard": 36.6212, "ring_dtp": 6.1545},
                          "latency_ms": {"standard": 1001.2, "ring_dtp": 1052.2}},
    }
    for key in ("roofline", "roofline_fwd"):  # HBM rate of the counted traffic
        r = out[key]
        r["traffic_gb_per_s"] = (r["traffic"] / (r["avg_launch_ms"] * 1e-3) / 1e9
                                 if r["traffic"] is not None else None)
        add_frac_at_clock(r, inp.dtype)
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(inp, args.cpu_sample_rows)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
