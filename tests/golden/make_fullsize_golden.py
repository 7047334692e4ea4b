"""Writes the oracle's per-token loss and lse for the four bf16 workloads at full size.

Expected values for the full-size GPU parity tests (tests/test_gpu_fullsize.py):
the float64 oracle's forward (Sec. 3.2: lse = log sum_v e^y, loss = lse - y_target)
over every token of each workload, and the largest |logit| it met (the stress
workload's logit scale is checked against it), stored with the SHA-256 of the
generated inputs so that a test can confirm it draws the same bits.  Calls only
the oracle and the input generator.  Takes about half an hour on eight cores.

    python tests/golden/make_fullsize_golden.py [workload ...]
"""
import os
import sys
import time

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
sys.path.insert(0, ROOT)

import oracle  # noqa: E402
import workloads as wl  # noqa: E402


def golden_path(name: str) -> str:
    return os.path.join(HERE, f"fullsize_{name}.npz")


def make(name: str) -> None:
    t0 = time.time()
    inp = wl.make_inputs(name)
    sha = inp.sha256()
    H = wl.to_f64(inp.H, inp.dtype)
    W = np.concatenate([wl.to_f64(w, inp.dtype) for w in inp.W_shards], axis=0)
    loss, lse, max_abs = oracle.forward(H, W, inp.targets, inp.ignore_index, return_max_abs=True)
    np.savez_compressed(golden_path(name), loss=loss, lse=lse, sha256=np.array(sha),
                        T=inp.T, d=inp.d, V=inp.V, max_abs_logit=max_abs)
    print(f"{name}: T={inp.T} d={inp.d} V={inp.V} in {time.time() - t0:.0f} s, "
          f"max lse {lse.max():.3f}, max |logit| {max_abs:.3f}", flush=True)


if __name__ == "__main__":
    names = sys.argv[1:] or [w.name for w in wl.WORKLOAD_LIST if w.dtype == "bf16"]
    for n in names:
        make(n)
