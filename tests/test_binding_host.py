"""Host-side tests of the Python binding's tensor checks (no GPU).

The C ABI takes bare pointers, so the binding checks every tensor against the
problem before taking its pointer: dtype, shape (including each shard's width d),
contiguity, and one GPU device for all of them.  Each refusal below is raised on
the host; the library is never called with these tensors."""
import os

import pytest
import torch

import paper_2609_14306_amd as vp

pytestmark = pytest.mark.skipif(not os.path.exists(vp.LIB_PATH),
                                reason="libvpce.so not built (run __graft_entry__.build())")

T, D, ROWS = 6, 16, [5, 0, 7]


def _inputs(dtype=torch.bfloat16):
    H = torch.zeros(T, D, dtype=dtype)
    Ws = [torch.zeros(r, D, dtype=dtype) for r in ROWS]
    t = torch.zeros(T, dtype=torch.int64)
    return H, Ws, t


def _prob(dtype=torch.bfloat16):
    return vp.Problem(T, D, ROWS, vp.VP_BF16 if dtype == torch.bfloat16 else vp.VP_F32)


def _fwd_args(**over):
    H, Ws, t = _inputs()
    a = dict(prob=_prob(), H=H, W_shards=Ws, targets=t, loss=torch.zeros(T), lse=torch.zeros(T),
             ws=torch.zeros(vp.vp_ce_workspace_size(_prob())[0], dtype=torch.uint8))
    a.update(over)
    return a


def _bwd_args(**over):
    H, Ws, t = _inputs()
    a = dict(prob=_prob(), H=H, W_shards=Ws, targets=t, lse=torch.zeros(T), grad_loss=torch.zeros(T),
             dH=torch.zeros(T, D), dW_shards=[torch.zeros(r, D) for r in ROWS],
             ws=torch.zeros(vp.vp_ce_workspace_size(_prob())[1], dtype=torch.uint8))
    a.update(over)
    return a


def _refused(fn, args, match):
    with pytest.raises(ValueError, match=match):
        fn(**args)


FWD_CASES = {
    "H float32 with bf16 problem": (dict(H=torch.zeros(T, D)), "H: dtype"),
    "H wrong width": (dict(H=torch.zeros(T, D + 8, dtype=torch.bfloat16)), "H: shape"),
    "H not contiguous": (dict(H=torch.zeros(D, T, dtype=torch.bfloat16).t()), "H: must be contiguous"),
    "shard wrong width": (dict(W_shards=[torch.zeros(5, D + 8, dtype=torch.bfloat16),
                                         torch.zeros(0, D, dtype=torch.bfloat16),
                                         torch.zeros(7, D, dtype=torch.bfloat16)]), r"W_shards\[0\]: shape"),
    "shard wrong dtype": (dict(W_shards=[torch.zeros(5, D, dtype=torch.bfloat16),
                                         torch.zeros(0, D, dtype=torch.bfloat16),
                                         torch.zeros(7, D)]), r"W_shards\[2\]: dtype"),
    "shard count": (dict(W_shards=[torch.zeros(5, D, dtype=torch.bfloat16)]), "W_shards: 1 shards"),
    "int32 targets": (dict(targets=torch.zeros(T, dtype=torch.int32)), "targets: dtype"),
    "short targets": (dict(targets=torch.zeros(T - 1, dtype=torch.int64)), "targets: shape"),
    "bf16 loss": (dict(loss=torch.zeros(T, dtype=torch.bfloat16)), "loss: dtype"),
    "strided lse": (dict(lse=torch.zeros(2 * T)[::2]), "lse: must be contiguous"),
    "small workspace": (dict(ws=torch.zeros(8, dtype=torch.uint8)), "ws:"),
    "host tensors": ({}, "must be on a GPU device"),
}


@pytest.mark.parametrize("case", sorted(FWD_CASES))
def test_forward_refuses(case):
    over, match = FWD_CASES[case]
    _refused(vp.vp_ce_forward, _fwd_args(**over), match)


BWD_CASES = {
    "float64 grad_loss": (dict(grad_loss=torch.zeros(T, dtype=torch.float64)), "grad_loss: dtype"),
    "bf16 lse": (dict(lse=torch.zeros(T, dtype=torch.bfloat16)), "lse: dtype"),
    "dH bf16": (dict(dH=torch.zeros(T, D, dtype=torch.bfloat16)), "dH: dtype"),
    "dH transposed": (dict(dH=torch.zeros(D, T).t()), "dH: must be contiguous"),
    "dW bf16": (dict(dW_shards=[torch.zeros(5, D, dtype=torch.bfloat16), torch.zeros(0, D),
                                torch.zeros(7, D)]), r"dW_shards\[0\]: dtype"),
    "dW wrong rows": (dict(dW_shards=[torch.zeros(5, D), torch.zeros(0, D), torch.zeros(6, D)]),
                      r"dW_shards\[2\]: shape"),
    "dW count": (dict(dW_shards=[torch.zeros(5, D)]), "dW_shards: 1 shards"),
    "small workspace": (dict(ws=torch.zeros(64, dtype=torch.uint8)), "ws:"),
    "host tensors": ({}, "must be on a GPU device"),
}


@pytest.mark.parametrize("case", sorted(BWD_CASES))
def test_backward_refuses(case):
    over, match = BWD_CASES[case]
    _refused(vp.vp_ce_backward, _bwd_args(**over), match)


def test_fold_calls_refuse():
    H, Ws, t = _inputs()
    shard = vp.Problem(T, D, [7], vp.VP_BF16)
    ws = torch.zeros(vp.vp_ce_workspace_size(shard)[0], dtype=torch.uint8)
    with pytest.raises(ValueError, match="state: shape"):
        vp.vp_ce_fold_shard(shard, 0, H, Ws[2], t, torch.zeros(T), ws)
    with pytest.raises(ValueError, match="W_shards\\[0\\]: shape"):
        vp.vp_ce_fold_shard(shard, 0, H, Ws[0], t, torch.zeros(3 * T), ws)
    with pytest.raises(ValueError, match="must be on a GPU device"):
        vp.vp_ce_fold_shard(shard, 0, H, Ws[2], t, torch.zeros(3 * T), ws)
    with pytest.raises(ValueError, match="state: dtype"):
        vp.vp_ce_state_init(torch.zeros(3 * T, dtype=torch.float64), T)
    full = vp.Problem(T, D, ROWS, vp.VP_BF16)
    with pytest.raises(ValueError, match="targets: dtype"):
        vp.vp_ce_fold_finalize(full, t.int(), torch.zeros(3 * T), torch.zeros(T), torch.zeros(T),
                               torch.zeros(256, dtype=torch.uint8))
