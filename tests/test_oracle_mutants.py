"""Planted mistakes in the CPU oracle (on the CPU only): each one must trip at least one pin.

Every mutant is a plausible slip in the oracle's arithmetic: a dropped term, a
wrong sign, a wrong index or offset, a transposed or permuted operand.
"""
import numpy as np
import pytest

import oracle.ce as ce
from oracle_pins import ALL_PINS

_orig_fwd = ce._forward_chunk
_orig_res = ce._residual_chunk


def _res_no_onehot(Y, lse, t, g, ign):
    G = np.exp(Y - lse[:, None]) * np.asarray(g)[:, None]
    G[t == ign] = 0.0
    return G


def _res_flipped_sign(Y, lse, t, g, ign):
    return -_orig_res(Y, lse, t, g, ign)


def _res_no_upstream(Y, lse, t, g, ign):
    return _orig_res(Y, lse, t, np.ones_like(np.asarray(g, dtype=np.float64)), ign)


def _res_ignored_not_zeroed(Y, lse, t, g, ign):
    G = np.exp(Y - lse[:, None])
    ok = (t != ign) & (t >= 0) & (t < Y.shape[1])
    G[np.nonzero(ok)[0], t[ok]] -= 1.0
    return G * np.asarray(g)[:, None]


def _res_rolled_lse(Y, lse, t, g, ign):
    return _orig_res(Y, np.roll(lse, 1), t, g, ign)


def _fwd_no_log(Y, t, ign):
    loss, lse = _orig_fwd(Y, t, ign)
    return loss - lse + np.exp(lse), np.exp(lse)


def _fwd_max_only(Y, t, ign):
    loss, lse = _orig_fwd(Y, t, ign)
    mx = Y.max(axis=1)
    return np.where(t == ign, 0.0, loss - lse + mx), mx


def _fwd_loss_sign(Y, t, ign):
    loss, lse = _orig_fwd(Y, t, ign)
    # loss = lse + y_t instead of lse - y_t
    return np.where(t == ign, 0.0, 2 * lse - loss), lse


def _fwd_target_off_by_one(Y, t, ign):
    V = Y.shape[1]
    t2 = np.where((t == ign) | (t < 0) | (t >= V), t, (t + 1) % V)
    return _orig_fwd(Y, t2, ign)


def _make_fold(variant):
    def fold_shard(state, H, W_q, off_q, targets):
        m, z, y = (np.array(a, dtype=np.float64, copy=True) for a in state)
        W_q = np.asarray(W_q, dtype=np.float64)
        targets = np.asarray(targets, dtype=np.int64)
        if W_q.shape[0] == 0:
            return m, z, y
        Y = np.asarray(H, dtype=np.float64) @ W_q.T
        m_new = np.maximum(m, Y.max(axis=1))
        if variant == "no_rescale":
            z = z + np.exp(Y - m_new[:, None]).sum(axis=1)
        else:
            z = np.exp(m - m_new) * z + np.exp(Y - m_new[:, None]).sum(axis=1)
        lo, hi = off_q, off_q + W_q.shape[0]
        if variant == "interval_open":
            own = (targets > lo) & (targets < hi)
        else:
            own = (targets >= lo) & (targets < hi)
        y[own] = Y[np.nonzero(own)[0], targets[own] - lo]
        return m_new, z, y
    return fold_shard


def _finalize_target_added(state, targets, V, ignore_index=-100):
    m, z, y = state
    lse = m + np.log(z)
    return np.where(np.asarray(targets) == ignore_index, 0.0, lse + y), lse


def _make_backward(variant):
    def backward(H, W, targets, lse, grad_loss, ignore_index=-100, row_chunk=None):
        H = np.asarray(H, dtype=np.float64); W = np.asarray(W, dtype=np.float64)
        Y = H @ W.T
        G = _orig_res(Y, np.asarray(lse, dtype=np.float64), np.asarray(targets), grad_loss,
                      ignore_index)
        if variant == "dW_rows_reversed":
            return G @ W, G.T @ H[::-1]
        if variant == "dH_vocab_reversed":
            return G @ W[::-1], G.T @ H
        raise ValueError(variant)
    return backward


def _fb_from(backward):
    def forward_backward(H, W_shards, targets, grad_loss, ignore_index=-100, row_chunk=None):
        W = ce.concat_shards(W_shards)
        loss, lse = ce.forward(H, W, targets, ignore_index)
        dH, dW = backward(H, W, targets, lse, grad_loss, ignore_index)
        rows = [np.asarray(w).shape[0] for w in W_shards]
        offs = np.cumsum([0] + rows)
        return {"loss": loss, "lse": lse, "dH": dH, "dW": dW, "max_abs_logit": 0.0,
                "dW_shards": [dW[offs[p]:offs[p + 1]] for p in range(len(rows))]}
    return forward_backward


MUTANTS = {
    "residual_without_onehot": {"_residual_chunk": _res_no_onehot},
    "residual_sign_flipped": {"_residual_chunk": _res_flipped_sign},
    "residual_without_upstream_gradient": {"_residual_chunk": _res_no_upstream},
    "residual_ignored_rows_not_zeroed": {"_residual_chunk": _res_ignored_not_zeroed},
    "residual_lse_of_wrong_row": {"_residual_chunk": _res_rolled_lse},
    "lse_missing_log": {"_forward_chunk": _fwd_no_log},
    "lse_is_max_only": {"_forward_chunk": _fwd_max_only},
    "loss_sign_of_target_logit": {"_forward_chunk": _fwd_loss_sign},
    "target_gather_off_by_one": {"_forward_chunk": _fwd_target_off_by_one},
    "fold_without_rescale": {"fold_shard": _make_fold("no_rescale")},
    "fold_interval_excludes_first_id": {"fold_shard": _make_fold("interval_open")},
    "fold_finalize_adds_target_logit": {"fold_finalize": _finalize_target_added},
    "dW_token_rows_permuted": {"backward": _make_backward("dW_rows_reversed"),
                               "forward_backward": _fb_from(_make_backward("dW_rows_reversed"))},
    "dH_vocab_rows_permuted": {"backward": _make_backward("dH_vocab_reversed"),
                               "forward_backward": _fb_from(_make_backward("dH_vocab_reversed"))},
}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutant_is_caught(name, monkeypatch):
    for attr, fn in MUTANTS[name].items():
        monkeypatch.setattr(ce, attr, fn)
    caught = []
    for pin in ALL_PINS:
        try:
            pin(ce)
        except Exception as e:  # noqa: BLE001 - any failure of a pin counts
            caught.append((pin.__name__, type(e).__name__))
    assert caught, f"planted mistake {name!r} passed every pin"
