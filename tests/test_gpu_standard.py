"""The dense "standard" baseline beside the fused path (bench.py --standard), on the GPU.

The paper compares Ring-DTP with a standard projection that materialises the full
logits and log-softmax (Sec. 3.2 results table; App. C peak and latency tables).
bench.py's --standard mode runs that dense path with plain torch ops next to this
library's forward + backward on the same resident inputs.  Here both legs' per-token
loss, dH and dW are compared with the float64 oracle on small bf16 and float32
workloads, and the mode's JSON line is checked for the fields it reports.

Bars: the fused leg meets the library's parity bar (bf16: |d loss| <= 2e-3,
relative Frobenius <= 1e-2 on dH and dW; float32: 1e-5).  The dense bf16 leg
rounds its [T, V] logits to bfloat16 (torch's bf16 product), so its loss carries
that rounding: |d loss| <= 2^-8 (1 + max_v |y_tv|) per token (the log-sum-exp and
the target logit each move by at most the largest logit rounding, 2^-9 |y|);
its gradients, like the fused leg's, go through a bfloat16 residual (<= 1e-2).
The dense float32 leg meets the float32 bar.

The --gemm-reference mode (the fused forward alternating with torch.matmul of the same
logits) is checked for the fields it reports.
"""
import json
import os
import subprocess
import sys

import numpy as np
import pytest

import workloads as wl
from helpers import assert_grad_close, assert_loss_close, oracle_inputs, to_device

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.mark.parametrize("name,kw", [
    ("bf16_T4096_d2880_V201088_P8", dict(T=300, d=320, V=5000, P=4, seed=61)),
    ("tiny_f32_T256_d256_V2048_P8", dict(seed=0)),
])
def test_standard_and_fused_legs_against_oracle(name, kw):
    import torch

    import bench
    import oracle

    inp = wl.make_inputs(name, **kw)
    H, Ws, t = to_device(inp)
    res = bench.standard_vs_fused(inp, H, Ws, t, steps=2, warmup=1, keep_outputs=True)
    n_valid = int((inp.targets != inp.ignore_index).sum())
    g = np.full(inp.T, 1.0 / max(n_valid, 1))
    H64, W64 = oracle_inputs(inp)
    ref = oracle.forward_backward(H64, W64, inp.targets, g, inp.ignore_index)
    Wcat = np.concatenate(W64, axis=0)
    ymax = np.abs(H64 @ Wcat.T).max(axis=1)
    for leg in ("standard", "fused"):
        o = res["outputs"][leg]
        loss = o["loss"].numpy().astype(np.float64)
        if leg == "standard" and inp.dtype == "bf16":
            err = np.abs(loss - ref["loss"])
            bound = 2.0 ** -8 * (1.0 + ymax)
            assert np.all(err <= bound), f"standard loss: worst {err.max():.2e}"
        else:
            assert_loss_close(inp.dtype, loss, ref["loss"], f"{leg} loss")
        e_h = assert_grad_close(inp.dtype, o["dH"].numpy(), ref["dH"], f"{leg} dH")
        e_w = assert_grad_close(inp.dtype, o["dW"].numpy(), ref["dW"], f"{leg} dW")
        print(f"{name} {leg}: dH {e_h:.2e} dW {e_w:.2e}, {res[leg]['ms_per_step']:.3f} ms, "
              f"{res[leg]['peak_above_resident_mib']:.1f} MiB", flush=True)
        assert res[leg]["ms_per_step"] > 0 and res[leg]["peak_above_resident_mib"] > 0
    # (at these small shapes the fused leg's workspace, sized by the strip budget and not by
    # T or V, exceeds the dense logits; the memory comparison at full size is bench.py's)
    torch.cuda.synchronize()


def test_standard_mode_json_line():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--standard", "--workload",
                        "tiny_f32_T256_d256_V2048_P8", "--steps", "2", "--warmup", "1"],
                       capture_output=True, text=True, timeout=300, cwd=ROOT)
    assert r.returncode == 0, r.stderr[-2000:]
    d = json.loads([ln for ln in r.stdout.splitlines() if ln.startswith("{")][-1])
    assert d["mode"] == "standard_vs_fused" and d["workload"] == "tiny_f32_T256_d256_V2048_P8"
    for leg in ("standard", "fused"):
        assert d[leg]["ms_per_step"] > 0 and d[leg]["peak_above_resident_mib"] > 0
    assert d["dense_logits_fp32_mib"] == 256 * 2048 * 4 / 2**20
    assert "outputs" not in d


def test_gemm_reference_mode_json_line():
    # bench.py --gemm-reference: the fused forward alternating with torch.matmul of the same
    # logits; both timed, both counted at 2 T V d.
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gemm-reference",
                        "--workload", "tiny_f32_T256_d256_V2048_P8", "--steps", "2", "--warmup", "1"],
                       capture_output=True, text=True, timeout=300, cwd=ROOT)
    assert r.returncode == 0, r.stderr[-2000:]
    d = json.loads([ln for ln in r.stdout.splitlines() if ln.startswith("{")][-1])
    assert d["mode"] == "gemm_reference" and d["workload"] == "tiny_f32_T256_d256_V2048_P8"
    for leg in ("gemm", "fused_forward"):
        assert 0 < d[leg]["min_ms"] <= d[leg]["median_ms"]
        assert d[leg]["tflops_at_median"] > 0
    assert d["fused_over_gemm_rate"] > 0
