"""GPU parity at the size limits the C ABI accepts: the largest hidden width
(d = 2^22) and the largest token count (T = 2^23 - 256).  These are the shapes
where the kernels' 32-bit per-lane load offsets, the k-blocked workspaces and the
launch grids are tightest; both cases also carry an empty shard and a permuted
visiting order.  Compared with the float64 oracle at the bf16 tolerances.

Host memory: about 10 GB (d test) and 25 GB (T test) for the float64 oracle and
the comparison; GPU memory about 6 GB and 5 GB.
"""
import numpy as np
import pytest

import workloads as wl
from helpers import compare_all, run_gpu, run_oracle

pytestmark = pytest.mark.gpu

MAX_D = 1 << 22          # the ABI's largest hidden width
MAX_T = (1 << 23) - 256  # the ABI's largest token count


def test_max_hidden_width():
    inp = wl.make_inputs("bf16_T4096_d2880_V201088_P8", T=40, d=MAX_D, V=48, P=1, seed=31)
    inp = wl.resplit(inp, [16, 0, 32], order=[2, 0, 1])
    g = wl.random_grad_loss(inp.T, 31, "random")
    # A 256 x 256 residual strip keeps the backward workspace (H^T and one W^T chunk,
    # each d x 256) near 4 GiB.
    got = run_gpu(inp, g, strip_elems=256 * 256)
    assert got["ws_bytes"][1] < 5 << 30
    ref = run_oracle(inp, g)
    errs = compare_all(inp, got, ref, "d = 2^22")
    print("d = 2^22:", errs, flush=True)


def test_max_token_count():
    inp = wl.make_inputs("bf16_T4096_d2880_V201088_P8", T=MAX_T, d=64, V=20, P=1, seed=37)
    inp = wl.resplit(inp, [7, 0, 13], order=[2, 0, 1])
    g = wl.random_grad_loss(inp.T, 37, "random")
    got = run_gpu(inp, g)
    ref = run_oracle(inp, g)
    errs = compare_all(inp, got, ref, "T = 2^23 - 256")
    print("T = 2^23 - 256:", errs, flush=True)

