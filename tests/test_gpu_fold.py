"""GPU parity of the per-shard fold: one meeting of Algorithm 2 at a time, with the
per-token state (m, s, y) carried between calls as it would travel with the
activations on a move-activations ring (Sec. 3.2, Algorithm 2).

Reference: the oracle's fold_shard / fold_finalize on the same bits.  Tolerances as
for the forward: the partial normaliser m + log s and the logits m and y within
|d| <= 2e-3 (bf16) or 1e-5 * max(1, |ref|) (float32); the finalized loss and lse
likewise against the oracle's dense forward.
"""
import numpy as np
import pytest

import workloads as wl
from helpers import assert_loss_close, oracle_inputs, to_device

pytestmark = pytest.mark.gpu


def _offsets(rows):
    return [int(x) for x in np.cumsum([0] + list(rows))]


def _state_np(state, T):
    s = state.cpu().numpy().astype(np.float64)
    return s[:T], s[T:2 * T], s[2 * T:]


def _check_state(dtype, got, ref, targets, met_ids, what):
    m, s, y = got
    mr, zr, yr = ref
    assert_loss_close(dtype, m + np.log(s), mr + np.log(zr), f"{what}: m + log s")
    assert_loss_close(dtype, m, mr, f"{what}: m")
    met = np.isin(targets, met_ids)
    assert_loss_close(dtype, y[met], yr[met], f"{what}: target logits")
    assert np.all(y[~met] == 0.0), f"{what}: y written for a target not met yet"


@pytest.mark.parametrize("name,T", [("tiny_f32_T256_d256_V2048_P8", 256),
                                    ("longctx_bf16_T32768_d2880_V201088_P8_ring", 300)])
def test_fold_meetings_track_the_oracle(name, T):
    import oracle
    import paper_2609_14306_amd as vp

    inp = wl.make_inputs(name, T=T)
    H, Ws, t = to_device(inp)
    H64, W64 = oracle_inputs(inp)
    offs = _offsets(inp.shard_rows)
    state = vp.new_state(inp.T, H.device)
    ref = oracle.fold_init(inp.T)
    met = []
    for q in inp.order:
        vp.fold_shard(H, Ws[q], offs[q], t, state)
        ref = oracle.fold_shard(ref, H64, W64[q], offs[q], inp.targets)
        met.extend(range(offs[q], offs[q + 1]))
        _check_state(inp.dtype, _state_np(state, inp.T), ref, inp.targets, np.array(met),
                     f"{name} after shard {q}")
    loss, lse = vp.fold_finalize(t, state, inp.shard_rows, inp.ignore_index)
    W_all = np.concatenate(W64, axis=0)
    rl, rlse = oracle.forward(H64, W_all, inp.targets, inp.ignore_index)
    assert_loss_close(inp.dtype, loss.cpu().numpy(), rl, f"{name} fold loss")
    assert_loss_close(inp.dtype, lse.cpu().numpy(), rlse, f"{name} fold lse")
    # and the one-call forward over the same shards agrees to rounding
    fl, flse = vp.forward(H, Ws, t, inp.ignore_index, inp.order)
    assert_loss_close(inp.dtype, loss.cpu().numpy(), fl.cpu().numpy().astype(np.float64),
                      f"{name} fold vs forward")


def test_fold_state_serialises_and_moves():
    import torch

    import paper_2609_14306_amd as vp

    inp = wl.make_inputs("bf16_T4096_d2880_V201088_P8", T=513, d=512, V=9000, P=5, seed=11)
    H, Ws, t = to_device(inp)
    offs = _offsets(inp.shard_rows)
    order = [3, 1, 4, 0, 2]
    straight = vp.new_state(inp.T, H.device)
    for q in order:
        vp.fold_shard(H, Ws[q], offs[q], t, straight)
    moved = vp.new_state(inp.T, H.device)
    for q in order[:2]:
        vp.fold_shard(H, Ws[q], offs[q], t, moved)
    blob = moved.cpu().numpy().tobytes()  # 12 T bytes: the whole state
    assert len(blob) == 12 * inp.T
    resumed = torch.from_numpy(np.frombuffer(blob, dtype=np.float32).copy()).to(H.device)
    for q in order[2:]:
        vp.fold_shard(H, Ws[q], offs[q], t, resumed)
    torch.cuda.synchronize()
    assert torch.equal(resumed, straight), "a state resumed from its bytes must fold identically"


def test_fold_cut_shard_and_empty_shard():
    import torch

    import paper_2609_14306_amd as vp

    inp = wl.make_inputs("bf16_T4096_d2880_V201088_P8", T=200, d=256, V=1500, P=1, seed=12)
    H, Ws, t = to_device(inp)
    W = Ws[0]
    whole = vp.new_state(inp.T, H.device)
    vp.fold_shard(H, W, 0, t, whole)
    cut = vp.new_state(inp.T, H.device)
    vp.fold_shard(H, W[:777].contiguous(), 0, t, cut)  # a cut off the 256-row tile grid
    before = cut.clone()
    vp.fold_shard(H, W[:0], 777, t, cut)  # empty strip: no change at all
    torch.cuda.synchronize()
    assert torch.equal(before, cut)
    vp.fold_shard(H, W[777:].contiguous(), 777, t, cut)
    lw, sw = vp.fold_finalize(t, whole, [1500], inp.ignore_index)
    lc, sc = vp.fold_finalize(t, cut, [1500], inp.ignore_index)
    assert_loss_close("bf16", lc.cpu().numpy(), lw.cpu().numpy().astype(np.float64), "cut shard loss")
    assert_loss_close("bf16", sc.cpu().numpy(), sw.cpu().numpy().astype(np.float64), "cut shard lse")


def test_move_activations_ring_on_one_gpu():
    """P ranks emulated in turn: rank r holds shard r and its own token batch; in round i
    batch b is at rank (b + i) mod P and folds that rank's shard into the state that
    travels with it; after P rounds each batch's state is finalized by its owner."""
    import oracle
    import paper_2609_14306_amd as vp

    inp = wl.make_inputs("tiny_f32_T256_d256_V2048_P8", T=500, seed=13)
    H, Ws, t = to_device(inp)
    H64, W64 = oracle_inputs(inp)
    P = len(Ws)
    offs = _offsets(inp.shard_rows)
    cuts = [0, 37, 37, 101, 106, 234, 235, 325, 500]  # batch 1 is empty
    batches = [(cuts[b], cuts[b + 1]) for b in range(P)]
    states = [vp.new_state(hi - lo, H.device) if hi > lo else None for lo, hi in batches]
    for i in range(P):
        for b, (lo, hi) in enumerate(batches):
            if hi == lo:
                continue
            r = (b + i) % P
            vp.fold_shard(H[lo:hi], Ws[r], offs[r], t[lo:hi], states[b])
    W_all = np.concatenate(W64, axis=0)
    rl, rlse = oracle.forward(H64, W_all, inp.targets, inp.ignore_index)
    for b, (lo, hi) in enumerate(batches):
        if hi == lo:
            continue
        loss, lse = vp.fold_finalize(t[lo:hi], states[b], inp.shard_rows, inp.ignore_index)
        assert_loss_close("f32", loss.cpu().numpy(), rl[lo:hi], f"batch {b} loss")
        assert_loss_close("f32", lse.cpu().numpy(), rlse[lo:hi], f"batch {b} lse")


def test_fold_finalize_reports_bad_targets():
    import torch

    import paper_2609_14306_amd as vp

    inp = wl.make_inputs("bf16_T4096_d2880_V201088_P8", T=64, d=128, V=700, P=2, seed=14)
    inp.targets[5] = 700        # one past the vocabulary
    inp.targets[6] = -7         # negative, not the ignore index
    inp.targets[7] = inp.ignore_index
    H, Ws, t = to_device(inp)
    offs = _offsets(inp.shard_rows)
    state = vp.new_state(inp.T, H.device)
    for q in (1, 0):
        vp.fold_shard(H, Ws[q], offs[q], t, state)
    ws = torch.zeros(256, dtype=torch.uint8, device=H.device)
    loss, lse = vp.fold_finalize(t, state, inp.shard_rows, inp.ignore_index, ws=ws)
    loss = loss.cpu().numpy()
    assert np.isnan(loss[5]) and np.isnan(loss[6]) and loss[7] == 0.0
    assert np.all(np.isfinite(np.delete(loss, [5, 6])))
    assert np.all(np.isfinite(lse.cpu().numpy()))
    assert vp.vp_ce_check(ws) == 2
