"""Float64 CPU oracle: softmax cross-entropy over a sharded vocabulary projection.

TEST INFRASTRUCTURE ONLY (see the package docstring): never imported by the
product path.  Plain and slow on purpose; a numpy matrix product is the only
library primitive used, and nothing is blocked, fused or reordered beyond
splitting the token rows into independent chunks (every quantity below is
row-local except dW, which is a plain sum over rows).

Notation (Sec. 3.2): token t has hidden state h_t (row of H [T, d]); vocabulary
id v has projection row w_v (row of W [V, d], the concatenation of the shards in
vocabulary-id order: shard p owns ids [off_p, off_p + V_p)); y_tv = h_t . w_v.
"""
from __future__ import annotations

import math
from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np

# Logits beyond this magnitude would overflow exp() in float64; the plain
# definition is only used where it is exact to float64 rounding.
_EXP_SAFE = 700.0


def concat_shards(W_shards: Sequence[np.ndarray]) -> np.ndarray:
    """W [V, d]: the shards stacked in vocabulary-id order (shard p owns [off_p, off_p+V_p))."""
    return np.concatenate([np.asarray(w, dtype=np.float64) for w in W_shards], axis=0)


def _default_chunk(V: int) -> int:
    return max(1, (1 << 26) // max(V, 1))


def _valid(targets: np.ndarray, V: int, ignore_index: int) -> Tuple[np.ndarray, np.ndarray]:
    ignored = targets == ignore_index
    bad = (~ignored) & ((targets < 0) | (targets >= V))
    return ignored, bad


def _forward_chunk(Y: np.ndarray, t: np.ndarray, ignore_index: int):
    """Definition of Sec. 3.2: lse = log sum_v e^y, loss = lse - y_target (0 if ignored)."""
    V = Y.shape[1]
    if Y.size and np.max(np.abs(Y)) >= _EXP_SAFE:
        raise OverflowError("logit magnitude beyond the float64-exact range of the oracle")
    lse = np.log(np.sum(np.exp(Y), axis=1))
    ignored, bad = _valid(t, V, ignore_index)
    ok = ~(ignored | bad)
    y_t = np.zeros(Y.shape[0])
    y_t[ok] = Y[np.nonzero(ok)[0], t[ok]]
    loss = np.where(ok, lse - y_t, 0.0)
    loss[bad] = np.nan
    return loss, lse


def _residual_chunk(Y: np.ndarray, lse: np.ndarray, t: np.ndarray, g: np.ndarray,
                    ignore_index: int) -> np.ndarray:
    """Softmax residual G = g (softmax(y) - onehot(target)); 0 rows if ignored, NaN rows if invalid."""
    V = Y.shape[1]
    ignored, bad = _valid(t, V, ignore_index)
    ok = ~(ignored | bad)
    G = np.exp(Y - lse[:, None])
    rows = np.nonzero(ok)[0]
    G[rows, t[ok]] -= 1.0
    G *= np.asarray(g, dtype=np.float64)[:, None]
    G[ignored] = 0.0
    G[bad] = np.nan
    return G


def forward(H: np.ndarray, W: np.ndarray, targets: np.ndarray, ignore_index: int = -100,
            row_chunk: Optional[int] = None, return_max_abs: bool = False):
    """Per-token (loss, lse) in float64 from the full logits of each row chunk; with
    return_max_abs, also the largest |y_tv| over every token and vocabulary id."""
    H = np.asarray(H, dtype=np.float64)
    W = np.asarray(W, dtype=np.float64)
    targets = np.asarray(targets, dtype=np.int64)
    T = H.shape[0]
    rc = row_chunk or _default_chunk(W.shape[0])
    loss = np.zeros(T)
    lse = np.zeros(T)
    max_abs = 0.0
    for a in range(0, T, rc):
        b = min(T, a + rc)
        Y = H[a:b] @ W.T
        if Y.size:
            max_abs = max(max_abs, float(np.max(np.abs(Y))))
        loss[a:b], lse[a:b] = _forward_chunk(Y, targets[a:b], ignore_index)
    if return_max_abs:
        return loss, lse, max_abs
    return loss, lse


def backward(H: np.ndarray, W: np.ndarray, targets: np.ndarray, lse: np.ndarray,
             grad_loss: np.ndarray, ignore_index: int = -100,
             row_chunk: Optional[int] = None) -> Tuple[np.ndarray, np.ndarray]:
    """(dH, dW) = (G W, G^T H) with G recomputed per row chunk from the saved lse."""
    H = np.asarray(H, dtype=np.float64)
    W = np.asarray(W, dtype=np.float64)
    targets = np.asarray(targets, dtype=np.int64)
    g = np.asarray(grad_loss, dtype=np.float64)
    T = H.shape[0]
    rc = row_chunk or _default_chunk(W.shape[0])
    dH = np.zeros_like(H)
    dW = np.zeros_like(W)
    for a in range(0, T, rc):
        b = min(T, a + rc)
        Y = H[a:b] @ W.T
        G = _residual_chunk(Y, np.asarray(lse[a:b], dtype=np.float64), targets[a:b], g[a:b],
                            ignore_index)
        dH[a:b] = G @ W
        dW += G.T @ H[a:b]
    return dH, dW


def forward_backward(H: np.ndarray, W_shards: Sequence[np.ndarray], targets: np.ndarray,
                     grad_loss: np.ndarray, ignore_index: int = -100,
                     row_chunk: Optional[int] = None) -> Dict[str, object]:
    """Dense forward and backward in one pass over row chunks (each chunk's logits used twice)."""
    W = concat_shards(W_shards)
    H = np.asarray(H, dtype=np.float64)
    targets = np.asarray(targets, dtype=np.int64)
    g = np.asarray(grad_loss, dtype=np.float64)
    T = H.shape[0]
    rc = row_chunk or _default_chunk(W.shape[0])
    loss = np.zeros(T)
    lse = np.zeros(T)
    dH = np.zeros_like(H)
    dW = np.zeros_like(W)
    max_abs = 0.0
    for a in range(0, T, rc):
        b = min(T, a + rc)
        Y = H[a:b] @ W.T
        if Y.size:
            max_abs = max(max_abs, float(np.max(np.abs(Y))))
        loss[a:b], lse[a:b] = _forward_chunk(Y, targets[a:b], ignore_index)
        G = _residual_chunk(Y, lse[a:b], targets[a:b], g[a:b], ignore_index)
        dH[a:b] = G @ W
        dW += G.T @ H[a:b]
    rows = [np.asarray(w).shape[0] for w in W_shards]
    offs = np.cumsum([0] + rows)
    dW_shards = [dW[offs[p]:offs[p + 1]] for p in range(len(rows))]
    return {"loss": loss, "lse": lse, "dH": dH, "dW_shards": dW_shards, "dW": dW,
            "max_abs_logit": max_abs}


def fold_init(T: int):
    """Algorithm 2's initial per-token state (m, z, y) = (-inf, 0, 0)."""
    return np.full(T, -np.inf), np.zeros(T), np.zeros(T)


def fold_shard(state, H: np.ndarray, W_q: np.ndarray, off_q: int, targets: np.ndarray):
    """One meeting of Algorithm 2: fold the logit strip of one shard into the state.

    The shard owns global ids [off_q, off_q + V_q).  With Y = H W_q^T (the strip of
    this meeting), the online-softmax update of Sec. 3.2 gives
    m' = max(m, max_v Y_v) and z' = e^{m - m'} z + sum_v e^{Y_v - m'}; the target
    logit y is written by the one shard whose interval holds the target.  An empty
    strip leaves the state unchanged (reading for the -inf - -inf case).
    Returns a new state; the input is not modified.
    """
    m, z, y = (np.array(a, dtype=np.float64, copy=True) for a in state)
    W_q = np.asarray(W_q, dtype=np.float64)
    targets = np.asarray(targets, dtype=np.int64)
    V_q = W_q.shape[0]
    if V_q == 0:
        return m, z, y
    Y = np.asarray(H, dtype=np.float64) @ W_q.T
    m_new = np.maximum(m, Y.max(axis=1))
    z = np.exp(m - m_new) * z + np.exp(Y - m_new[:, None]).sum(axis=1)
    own = (targets >= off_q) & (targets < off_q + V_q)
    y[own] = Y[np.nonzero(own)[0], targets[own] - off_q]
    return m_new, z, y


def fold_finalize(state, targets: np.ndarray, V: int, ignore_index: int = -100):
    """(loss, lse) from a state that has met every shard: lse = m + log z, loss = lse - y
    (0 for ignored tokens, NaN for targets outside [0, V))."""
    m, z, y = state
    lse = m + np.log(z)
    ignored, bad = _valid(np.asarray(targets, dtype=np.int64), V, ignore_index)
    loss = np.where(ignored, 0.0, lse - y)
    loss[bad] = np.nan
    return loss, lse


def ring_forward(H: np.ndarray, W_shards: Sequence[np.ndarray], targets: np.ndarray,
                 order: Optional[Sequence[int]] = None, ignore_index: int = -100):
    """Algorithm 2's forward on one rank: fold each shard's logit strip in visiting order
    (fold_shard per meeting), then finalize.  Returns (loss, lse, final state)."""
    H = np.asarray(H, dtype=np.float64)
    targets = np.asarray(targets, dtype=np.int64)
    P = len(W_shards)
    order = list(range(P)) if order is None else list(order)
    if sorted(order) != list(range(P)):
        raise ValueError("order must be a permutation of the shards")
    rows = [np.asarray(w).shape[0] for w in W_shards]
    offs = np.cumsum([0] + rows)
    state = fold_init(H.shape[0])
    for q in order:
        state = fold_shard(state, H, W_shards[q], int(offs[q]), targets)
    loss, lse = fold_finalize(state, targets, int(offs[-1]), ignore_index)
    return loss, lse, state


def scalar_forward_backward(H, W, targets, grad_loss, ignore_index: int = -100):
    """Pure-Python loops over tokens, vocabulary ids and features (tiny shapes only)."""
    H = [[float(x) for x in row] for row in np.asarray(H, dtype=np.float64)]
    W = [[float(x) for x in row] for row in np.asarray(W, dtype=np.float64)]
    T, V = len(H), len(W)
    d = len(H[0]) if T else (len(W[0]) if V else 0)
    loss = [0.0] * T
    lse = [0.0] * T
    dH = [[0.0] * d for _ in range(T)]
    dW = [[0.0] * d for _ in range(V)]
    for t in range(T):
        y = []
        for v in range(V):
            acc = 0.0
            for k in range(d):
                acc += H[t][k] * W[v][k]
            y.append(acc)
        s = 0.0
        for v in range(V):
            s += math.exp(y[v])
        lse[t] = math.log(s)
        tgt = int(targets[t])
        if tgt == ignore_index:
            continue
        loss[t] = lse[t] - y[tgt]
        g = float(grad_loss[t])
        for v in range(V):
            gv = g * (math.exp(y[v] - lse[t]) - (1.0 if v == tgt else 0.0))
            for k in range(d):
                dH[t][k] += gv * W[v][k]
                dW[v][k] += gv * H[t][k]
    return (np.array(loss), np.array(lse), np.array(dH).reshape(T, d),
            np.array(dW).reshape(V, d))


# ---------------------------------------------------------------------------
# Restrictions used where the full oracle would take too long.  Each is the
# same definition evaluated on a subset: rows are independent in loss, lse and
# dH; one vocabulary row of dW needs that row's logits for every token and the
# lse of every token.

def forward_rows(H, W, targets, rows, ignore_index: int = -100, row_chunk: Optional[int] = None):
    """(loss, lse) of the listed token rows only."""
    rows = np.asarray(rows, dtype=np.int64)
    return forward(np.asarray(H)[rows], W, np.asarray(targets)[rows], ignore_index, row_chunk)


def backward_rows(H, W, targets, lse_rows, grad_rows, rows, ignore_index: int = -100,
                  row_chunk: Optional[int] = None) -> np.ndarray:
    """dH of the listed token rows, given their lse and upstream gradients."""
    rows = np.asarray(rows, dtype=np.int64)
    H = np.asarray(H, dtype=np.float64)
    W = np.asarray(W, dtype=np.float64)
    t = np.asarray(targets, dtype=np.int64)[rows]
    rc = row_chunk or _default_chunk(W.shape[0])
    out = np.zeros((rows.size, H.shape[1]))
    for a in range(0, rows.size, rc):
        b = min(rows.size, a + rc)
        Y = H[rows[a:b]] @ W.T
        G = _residual_chunk(Y, np.asarray(lse_rows[a:b], dtype=np.float64), t[a:b],
                            np.asarray(grad_rows[a:b], dtype=np.float64), ignore_index)
        out[a:b] = G @ W
    return out


def dW_rows(H, W, targets, lse, grad_loss, vocab_ids, ignore_index: int = -100,
            row_chunk: int = 16384) -> np.ndarray:
    """dW of the listed vocabulary ids, given the lse and upstream gradient of every token."""
    H = np.asarray(H, dtype=np.float64)
    W = np.asarray(W, dtype=np.float64)
    vocab_ids = np.asarray(vocab_ids, dtype=np.int64)
    targets = np.asarray(targets, dtype=np.int64)
    V = W.shape[0]
    Wv = W[vocab_ids]
    out = np.zeros((vocab_ids.size, H.shape[1]))
    ignored, bad = _valid(targets, V, ignore_index)
    for a in range(0, H.shape[0], row_chunk):
        b = min(H.shape[0], a + row_chunk)
        Y = H[a:b] @ Wv.T  # [rows, |ids|]
        G = np.exp(Y - np.asarray(lse[a:b], dtype=np.float64)[:, None])
        G -= (targets[a:b, None] == vocab_ids[None, :])
        G *= np.asarray(grad_loss[a:b], dtype=np.float64)[:, None]
        G[ignored[a:b]] = 0.0
        G[bad[a:b]] = np.nan
        out += G.T @ H[a:b]
    return out
