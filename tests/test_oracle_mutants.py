"""Planted mistakes in the CPU oracle (on the CPU only): each one must trip at least one pin.

Every mutant is a plausible slip in the oracle's arithmetic: a dropped term, a
wrong sign, a wrong index or offset, a transposed or permuted operand.
"""
import numpy as np
import pytest

import oracle.ce as ce
from oracle_pins import ALL_PINS

_orig_fwd = ce._forward_chunk
_orig_forward = ce.forward
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


# Mistakes in the row-chunk loop of the dense functions: they change nothing while the
# whole batch fits one chunk, and every full-size expected value is written by this loop.
def _chunk_bounds(T, rc, variant):
    for a in range(0, T, rc):
        b = min(T, a + rc)
        if variant == "drop_last_row" and b < T:
            b -= 1  # off by one at every inner chunk edge; the last chunk ends at T
        yield a, b


def _make_chunk_forward(variant):
    def forward(H, W, targets, ignore_index=-100, row_chunk=None):
        H = np.asarray(H, dtype=np.float64); W = np.asarray(W, dtype=np.float64)
        targets = np.asarray(targets, dtype=np.int64)
        T = H.shape[0]
        rc = row_chunk or ce._default_chunk(W.shape[0])
        loss, lse = np.zeros(T), np.zeros(T)
        for a, b in _chunk_bounds(T, rc, variant):
            loss[a:b], lse[a:b] = _orig_fwd(H[a:b] @ W.T, targets[a:b], ignore_index)
        return loss, lse
    return forward


def _make_chunk_backward(variant):
    def backward(H, W, targets, lse, grad_loss, ignore_index=-100, row_chunk=None):
        H = np.asarray(H, dtype=np.float64); W = np.asarray(W, dtype=np.float64)
        targets = np.asarray(targets, dtype=np.int64)
        g = np.asarray(grad_loss, dtype=np.float64)
        lse = np.asarray(lse, dtype=np.float64)
        T = H.shape[0]
        rc = row_chunk or ce._default_chunk(W.shape[0])
        dH, dW = np.zeros_like(H), np.zeros_like(W)
        for a, b in _chunk_bounds(T, rc, variant):
            la = lse[0:b - a] if variant == "first_chunk_lse" else lse[a:b]
            G = _orig_res(H[a:b] @ W.T, la, targets[a:b], g[a:b], ignore_index)
            dH[a:b] = G @ W
            if variant == "dW_overwritten":
                dW = G.T @ H[a:b]
            else:
                dW += G.T @ H[a:b]
        return dH, dW
    return backward


def _make_chunk_fb(variant):
    def forward_backward(H, W_shards, targets, grad_loss, ignore_index=-100, row_chunk=None):
        W = ce.concat_shards(W_shards)
        H = np.asarray(H, dtype=np.float64)
        targets = np.asarray(targets, dtype=np.int64)
        g = np.asarray(grad_loss, dtype=np.float64)
        T = H.shape[0]
        rc = row_chunk or ce._default_chunk(W.shape[0])
        loss, lse = np.zeros(T), np.zeros(T)
        dH, dW = np.zeros_like(H), np.zeros_like(W)
        for a, b in _chunk_bounds(T, rc, variant):
            Y = H[a:b] @ W.T
            loss[a:b], lse[a:b] = _orig_fwd(Y, targets[a:b], ignore_index)
            la = lse[0:b - a] if variant == "first_chunk_lse" else lse[a:b]
            G = _orig_res(Y, la, targets[a:b], g[a:b], ignore_index)
            dH[a:b] = G @ W
            if variant == "dW_overwritten":
                dW = G.T @ H[a:b]
            else:
                dW += G.T @ H[a:b]
        rows = [np.asarray(w).shape[0] for w in W_shards]
        offs = np.cumsum([0] + rows)
        return {"loss": loss, "lse": lse, "dH": dH, "dW": dW, "max_abs_logit": 0.0,
                "dW_shards": [dW[offs[p]:offs[p + 1]] for p in range(len(rows))]}
    return forward_backward


def _forward_max_of_last_chunk(H, W, targets, ignore_index=-100, row_chunk=None,
                               return_max_abs=False):
    H = np.asarray(H, dtype=np.float64); W = np.asarray(W, dtype=np.float64)
    targets = np.asarray(targets, dtype=np.int64)
    T = H.shape[0]
    rc = row_chunk or ce._default_chunk(W.shape[0])
    loss, lse = np.zeros(T), np.zeros(T)
    max_abs = 0.0
    for a in range(0, T, rc):
        b = min(T, a + rc)
        Y = H[a:b] @ W.T
        max_abs = float(np.max(np.abs(Y)))  # overwritten per chunk instead of a running max
        loss[a:b], lse[a:b] = _orig_fwd(Y, targets[a:b], ignore_index)
    return (loss, lse, max_abs) if return_max_abs else (loss, lse)


def _forward_max_signed(H, W, targets, ignore_index=-100, row_chunk=None, return_max_abs=False):
    out = _orig_forward(H, W, targets, ignore_index, row_chunk)
    if not return_max_abs:
        return out
    Y = np.asarray(H, dtype=np.float64) @ np.asarray(W, dtype=np.float64).T
    return out[0], out[1], float(Y.max())  # the largest logit, not the largest magnitude


def _chunk_mutant(variant):
    return {"forward": _make_chunk_forward(variant), "backward": _make_chunk_backward(variant),
            "forward_backward": _make_chunk_fb(variant)}


MUTANTS = {
    "max_abs_logit_of_last_chunk_only": {"forward": _forward_max_of_last_chunk},
    "max_abs_logit_signed": {"forward": _forward_max_signed},
    "chunk_loop_dW_overwritten_per_chunk": _chunk_mutant("dW_overwritten"),
    "chunk_loop_drops_last_row_of_chunk": _chunk_mutant("drop_last_row"),
    "chunk_loop_lse_of_first_chunk": _chunk_mutant("first_chunk_lse"),
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
