"""Full-size GPU parity for the four bf16 workloads, in the launch configuration
bench.py times (default strip budget, the workload's visiting order).

Every workload:
* loss and lse of every token against the oracle's values written by
  tests/golden/make_fullsize_golden.py (same input bits, checked by SHA-256);
* ignored tokens have loss exactly 0 and zero dH rows;
* every token's residual row sums to zero over the vocabulary, so the sum of all
  rows of dW is zero: checked on every dW row at once, against 1e-2 of the dW
  Frobenius norm (independent row errors of relative size e add up to about e
  times that norm).

The T = 4096 workload: dH and dW compared whole (every shard concatenated) with the
oracle's forward + backward computed at test time (the contraction of the residual
into both gradients, App. C), relative Frobenius error <= 1e-2.

The long-context, wide and stress workloads (T = 32768 to 65536; the whole oracle
would take 10-20 minutes on the host): dH and dW on samples stratified by the
backward's strip plan, so that every (token chunk x vocabulary chunk) strip
contributes.  dH rows: the first and last token of every token chunk and 8 seeded
tokens inside each; dW rows: the first and last id of every vocabulary chunk of
every shard and 2 seeded ids inside each, plus the most frequent targets.  A dH row
sums over every vocabulary chunk and a dW row over every token chunk, so each strip
enters both samples.  The oracle computes the sampled rows from the full-size inputs.

The stress workload's logit scale is the one its recipe asks for: the largest
|logit| the oracle met (stored with its goldens) lies in [36, 44].

Tolerances as everywhere for bf16: |d loss|, |d lse| <= 2e-3; relative Frobenius
error <= 1e-2 on dH and dW (whole or sampled rows).
"""
import os

import numpy as np
import pytest

import workloads as wl
from helpers import assert_grad_close, assert_loss_close, strip_layout, stratified_rows

pytestmark = pytest.mark.gpu

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")
BF16 = [w.name for w in wl.WORKLOAD_LIST if w.dtype == "bf16"]
FULL = "bf16_T4096_d2880_V201088_P8"


def _run(name):
    import torch

    import paper_2609_14306_amd as vp
    from helpers import to_device

    path = os.path.join(GOLDEN, f"fullsize_{name}.npz")
    if not os.path.exists(path):
        pytest.skip(f"{path} missing: run tests/golden/make_fullsize_golden.py")
    gold = np.load(path, allow_pickle=False)
    inp = wl.make_inputs(name)
    assert inp.sha256() == str(gold["sha256"]), "generated inputs differ from the golden ones"
    n_valid = int((inp.targets != inp.ignore_index).sum())
    g = np.full(inp.T, 1.0 / max(n_valid, 1), dtype=np.float32)
    H, Ws, t = to_device(inp)
    loss, lse = vp.forward(H, Ws, t, inp.ignore_index, inp.order)
    dH, dWs = vp.backward(H, Ws, t, lse, torch.from_numpy(g).cuda(), inp.ignore_index, inp.order)
    torch.cuda.synchronize()
    loss = loss.cpu().numpy()
    lse_gpu = lse.cpu().numpy()
    print(f"{name}: max |dloss| {np.abs(loss - gold['loss']).max():.2e} "
          f"max |dlse| {np.abs(lse_gpu - gold['lse']).max():.2e}", flush=True)
    assert_loss_close("bf16", loss, gold["loss"], f"{name} loss (all tokens)")
    assert_loss_close("bf16", lse_gpu, gold["lse"], f"{name} lse (all tokens)")
    ign = inp.targets == inp.ignore_index
    assert np.all(loss[ign] == 0.0)

    col_sum = torch.zeros(inp.d, dtype=torch.float64, device=dWs[0].device)
    fro2 = 0.0
    for w in dWs:
        w64 = w.double()
        col_sum += w64.sum(0)
        fro2 += float((w64 * w64).sum())
    rel_sum = float(col_sum.norm()) / max(fro2 ** 0.5, 1e-300)
    print(f"{name}: |sum_v dW_v| / |dW|_F = {rel_sum:.2e}", flush=True)
    assert rel_sum <= 1e-2, f"{name}: dW rows do not sum to zero ({rel_sum:.2e})"
    if "max_abs_logit" in gold.files:
        print(f"{name}: oracle max |logit| {float(gold['max_abs_logit']):.3f}", flush=True)
    return inp, gold, g, dH, dWs


def test_fullsize_T4096_whole_gradients():
    import oracle
    from helpers import oracle_inputs

    inp, gold, g, dH, dWs = _run(FULL)
    H64, W64 = oracle_inputs(inp)
    ref = oracle.forward_backward(H64, W64, inp.targets, g.astype(np.float64), inp.ignore_index)
    assert_loss_close("bf16", gold["loss"], ref["loss"], "golden vs oracle loss")
    got_dH = dH.cpu().numpy()
    assert np.all(got_dH[inp.targets == inp.ignore_index] == 0.0)
    e_h = assert_grad_close("bf16", got_dH, ref["dH"], f"{FULL} dH (whole)")
    got_dW = np.concatenate([w.cpu().numpy() for w in dWs], axis=0)
    e_w = assert_grad_close("bf16", got_dW, ref["dW"], f"{FULL} dW (whole)")
    print(f"{FULL}: whole dH rel-Fro {e_h:.2e}, whole dW rel-Fro {e_w:.2e}", flush=True)


@pytest.mark.parametrize("name", [n for n in BF16 if n != FULL])
def test_fullsize_strip_stratified_parity(name):
    import torch

    import oracle
    import paper_2609_14306_amd as vp

    inp, gold, g, dH, dWs = _run(name)
    T, d = inp.T, inp.d
    ign = inp.targets == inp.ignore_index
    plan = vp.vp_ce_plan_info(vp.Problem(T, d, inp.shard_rows, vp.VP_BF16, inp.order))
    tok, voc = strip_layout(T, inp.shard_rows, inp.order, plan["Tc"], plan["Vc"])
    assert len(tok) * len(voc) == plan["strips"]

    H64 = wl.to_f64(inp.H, inp.dtype)
    W64 = np.concatenate([wl.to_f64(w, inp.dtype) for w in inp.W_shards], axis=0)
    rows = stratified_rows(tok, 8, seed=1)
    ref_dH = oracle.backward_rows(H64, W64, inp.targets, gold["lse"][rows], g[rows], rows,
                                  inp.ignore_index)
    got_dH = dH[torch.from_numpy(rows).cuda()].cpu().numpy()
    e = assert_grad_close("bf16", got_dH, ref_dH, f"{name} dH rows")
    assert np.all(got_dH[ign[rows]] == 0.0)

    valid = inp.targets[~ign]
    frequent = np.bincount(valid, minlength=inp.V).argsort()[-4:]
    ids = np.union1d(stratified_rows(voc, 2, seed=2), frequent)
    ref_dW = oracle.dW_rows(H64, W64, inp.targets, gold["lse"], g, ids, inp.ignore_index)
    offs = np.cumsum([0] + inp.shard_rows)
    shard_of = np.searchsorted(offs, ids, side="right") - 1
    got_dW = np.stack([dWs[int(p)][int(v - offs[p])].cpu().numpy() for v, p in zip(ids, shard_of)])
    e2 = assert_grad_close("bf16", got_dW, ref_dW, f"{name} dW rows")
    print(f"{name}: {len(tok)} token x {len(voc)} vocabulary chunks; {rows.size} dH rows "
          f"rel-Fro {e:.2e}, {ids.size} dW rows rel-Fro {e2:.2e}", flush=True)
    if name.startswith("stress"):
        m = float(gold["max_abs_logit"])
        assert 36.0 <= m <= 44.0, f"stress workload max |logit| {m:.2f} outside [36, 44]"
