"""Pins of the CPU oracle to things other than itself.

Each ``pin_*`` takes the oracle module (``oracle.ce``) and raises AssertionError
if the oracle disagrees with a closed form, an invariant, a brute-force result,
finite differences or a library routine.  The functions take the module as an
argument so that the same pins can be run against copies of the oracle with a
planted mistake (``test_oracle_mutants.py``): every plausible mistake must trip
at least one pin.
"""
from __future__ import annotations

import ast
import math
import os

import numpy as np

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")
IGN = -100


def _rng(seed):
    return np.random.default_rng(seed)


def _problem(seed, T=6, d=5, V=12, rows=(4, 3, 5), ignore=(1,), scale=1.0):
    rng = _rng(seed)
    H = rng.standard_normal((T, d)) * scale
    W = rng.standard_normal((V, d)) / math.sqrt(d)
    t = rng.integers(0, V, size=T).astype(np.int64)
    for i in ignore:
        t[i] = IGN
    g = rng.uniform(0.5, 1.5, size=T)
    assert sum(rows) == V
    offs = np.cumsum([0] + list(rows))
    shards = [W[offs[p]:offs[p + 1]] for p in range(len(rows))]
    return H, W, t, g, shards


def _rel(a, b):
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    den = max(np.linalg.norm(b), 1e-300)
    return float(np.linalg.norm(a - b) / den)


# --- a tiny safe evaluator for the golden fixture's exact expressions -------
_ALLOWED = (ast.Expression, ast.List, ast.BinOp, ast.UnaryOp, ast.Constant, ast.Call, ast.Name,
            ast.Load, ast.Add, ast.Sub, ast.Mult, ast.Div, ast.USub, ast.UAdd)


def _eval(expr: str):
    tree = ast.parse(expr, mode="eval")
    for node in ast.walk(tree):
        if not isinstance(node, _ALLOWED):
            raise ValueError(f"disallowed syntax in golden fixture: {type(node).__name__}")
        if isinstance(node, ast.Name) and node.id != "log":
            raise ValueError(f"unknown name {node.id}")
    return eval(compile(tree, "<golden>", "eval"), {"__builtins__": {}}, {"log": math.log})


def load_golden(name: str):
    vals = {}
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            key, expr = line.split("=", 1)
            vals[key.strip()] = _eval(expr.strip())
    return vals


# ---------------------------------------------------------------------------
def pin_golden_closed_form(ce):
    """Hand-derived 3-token, 4-id example (tests/golden/closed_form_4vocab.txt)."""
    gd = load_golden("closed_form_4vocab.txt")
    H = np.array(gd["H"], dtype=np.float64)
    W = np.array(gd["W"], dtype=np.float64)
    t = np.array(gd["targets"], dtype=np.int64)
    g = np.array(gd["g"], dtype=np.float64)
    rows = gd["shard_rows"]
    shards = [W[:rows[0]], W[rows[0]:]]
    out = ce.forward_backward(H, shards, t, g, ignore_index=IGN)
    np.testing.assert_allclose(out["lse"], gd["lse"], rtol=1e-14, atol=1e-15)
    np.testing.assert_allclose(out["loss"], gd["loss"], rtol=1e-14, atol=1e-15)
    np.testing.assert_allclose(out["dH"], gd["dH"], rtol=1e-13, atol=1e-15)
    np.testing.assert_allclose(np.concatenate(out["dW_shards"]), gd["dW"], rtol=1e-13, atol=1e-15)
    loss, lse = ce.forward(H, W, t, IGN)
    np.testing.assert_allclose(lse, gd["lse"], rtol=1e-14)
    np.testing.assert_allclose(loss, gd["loss"], rtol=1e-14, atol=1e-15)
    rl, rlse, _ = ce.ring_forward(H, shards, t, [1, 0], IGN)
    np.testing.assert_allclose(rlse, gd["lse"], rtol=1e-14)
    np.testing.assert_allclose(rl, gd["loss"], rtol=1e-14, atol=1e-15)


def pin_uniform_logits(ce):
    """W = 0: every logit is 0, so lse = loss = log V; with H = 0 as well, dW = 0."""
    for V, rows in [(7, (3, 4)), (2048, (256,) * 8)]:
        T, d = 5, 4
        H = _rng(1).standard_normal((T, d))
        W = np.zeros((V, d))
        t = np.array([0, V - 1, 3, IGN, 1], dtype=np.int64)
        loss, lse = ce.forward(H, W, t, IGN)
        np.testing.assert_allclose(lse, np.full(T, math.log(V)), rtol=1e-14)
        np.testing.assert_allclose(loss, [math.log(V)] * 3 + [0.0, math.log(V)], rtol=1e-14)
        offs = np.cumsum([0] + list(rows))
        rl, rlse, _ = ce.ring_forward(H, [W[offs[p]:offs[p + 1]] for p in range(len(rows))], t,
                                      None, IGN)
        np.testing.assert_allclose(rlse, np.full(T, math.log(V)), rtol=1e-14)


def pin_zero_hidden_closed_form(ce):
    """H = 0: softmax is uniform, so dH_t = g_t (mean_v w_v - w_target) and dW = 0."""
    rng = _rng(2)
    T, d, V = 4, 3, 9
    H = np.zeros((T, d))
    W = rng.standard_normal((V, d))
    t = np.array([2, IGN, 8, 0], dtype=np.int64)
    g = np.array([1.0, 2.0, 0.5, 3.0])
    loss, lse = ce.forward(H, W, t, IGN)
    dH, dW = ce.backward(H, W, t, lse, g, IGN)
    mean_w = W.mean(axis=0)
    for i in range(T):
        want = np.zeros(d) if t[i] == IGN else g[i] * (mean_w - W[t[i]])
        np.testing.assert_allclose(dH[i], want, rtol=1e-13, atol=1e-15)
    assert np.all(dW == 0.0)


def pin_two_class_logistic(ce):
    """V = 2 reduces to logistic loss: loss = softplus(y_o - y_t), dloss/dy_t = -sigmoid(y_o - y_t)."""
    rng = _rng(3)
    T, d = 8, 4
    H = rng.standard_normal((T, d)) * 2
    W = rng.standard_normal((2, d))
    t = rng.integers(0, 2, size=T).astype(np.int64)
    g = rng.uniform(0.5, 2.0, size=T)
    loss, lse = ce.forward(H, W, t, IGN)
    dH, dW = ce.backward(H, W, t, lse, g, IGN)
    dW_want = np.zeros_like(W)
    for i in range(T):
        yt = float(H[i] @ W[t[i]])
        yo = float(H[i] @ W[1 - t[i]])
        u = yo - yt
        softplus = max(u, 0.0) + math.log1p(math.exp(-abs(u)))
        sig = 1.0 / (1.0 + math.exp(-u))
        assert abs(loss[i] - softplus) <= 1e-13 * max(1.0, softplus)
        # G[i, t] = -g sig, G[i, o] = +g sig
        np.testing.assert_allclose(dH[i], g[i] * sig * (W[1 - t[i]] - W[t[i]]), rtol=1e-12,
                                   atol=1e-14)
        dW_want[t[i]] += -g[i] * sig * H[i]
        dW_want[1 - t[i]] += g[i] * sig * H[i]
    np.testing.assert_allclose(dW, dW_want, rtol=1e-12, atol=1e-14)


def pin_shift_invariance(ce):
    """Adding a constant c to every logit (a ones feature and a c column) shifts lse by c only."""
    H, W, t, g, _ = _problem(4)
    c = 0.7321
    H2 = np.concatenate([H, np.ones((H.shape[0], 1))], axis=1)
    W2 = np.concatenate([W, np.full((W.shape[0], 1), c)], axis=1)
    loss, lse = ce.forward(H, W, t, IGN)
    loss2, lse2 = ce.forward(H2, W2, t, IGN)
    np.testing.assert_allclose(lse2, lse + c, rtol=1e-14)
    np.testing.assert_allclose(loss2, loss, rtol=1e-12, atol=1e-14)
    dH, dW = ce.backward(H, W, t, lse, g, IGN)
    dH2, dW2 = ce.backward(H2, W2, t, lse2, g, IGN)
    np.testing.assert_allclose(dH2[:, :-1], dH, rtol=1e-12, atol=1e-14)
    np.testing.assert_allclose(dW2[:, :-1], dW, rtol=1e-12, atol=1e-14)


def pin_fold_order_invariance(ce):
    """Algorithm 2's fold over any visiting order (and empty shards) equals the dense definition."""
    H, W, t, g, shards = _problem(5, T=9, d=6, V=20, rows=(5, 0, 7, 8), ignore=(2, 6))
    loss, lse = ce.forward(H, W, t, IGN)
    rng = _rng(55)
    for _ in range(6):
        order = list(rng.permutation(len(shards)))
        rl, rlse, (m, z, y) = ce.ring_forward(H, shards, t, order, IGN)
        np.testing.assert_allclose(rlse, lse, rtol=1e-12)
        np.testing.assert_allclose(rl, loss, rtol=1e-12, atol=1e-13)
        Y = H @ W.T
        np.testing.assert_allclose(m, Y.max(axis=1), rtol=0, atol=0)


def pin_fold_state_passing(ce):
    """A state carried from meeting to meeting (one move-activations hop per shard, a shard
    cut in two at an arbitrary id, an empty shard) is, after any subset of meetings, the
    closed form over exactly the ids met so far: m = max of their logits, z = sum of
    e^{logit - m}, y = the target logit if the target was among them; after all of
    them it finalizes to the dense definition."""
    H, W, t, g, shards = _problem(8, T=11, d=5, V=23, rows=(6, 9, 0, 8), ignore=(4,))
    loss, lse = ce.forward(H, W, t, IGN)
    Y = H @ W.T
    # meetings: (global id offset, rows); shard 1 is cut at id 6 + 4
    meets = [(15, W[15:23]), (6, W[6:10]), (23, W[23:23]), (0, W[0:6]), (10, W[10:15])]
    state = ce.fold_init(H.shape[0])
    seen = np.zeros(W.shape[0], dtype=bool)
    for off, Wq in meets:
        state = ce.fold_shard(state, H, Wq, off, t)
        seen[off:off + Wq.shape[0]] = True
        if not seen.any():
            assert np.all(state[0] == -np.inf) and np.all(state[1] == 0.0)
            continue
        m_ref = Y[:, seen].max(axis=1)
        z_ref = np.exp(Y[:, seen] - m_ref[:, None]).sum(axis=1)
        np.testing.assert_allclose(state[0], m_ref, rtol=0, atol=0)
        np.testing.assert_allclose(state[1], z_ref, rtol=1e-13)
        met = (t >= 0) & (t < W.shape[0]) & (t != IGN)
        met[met] = seen[t[met]]
        np.testing.assert_allclose(state[2][met], Y[np.nonzero(met)[0], t[met]], rtol=0, atol=0)
        np.testing.assert_array_equal(state[2][~met], 0.0)
    fl, flse = ce.fold_finalize(state, t, W.shape[0], IGN)
    np.testing.assert_allclose(flse, lse, rtol=1e-12)
    np.testing.assert_allclose(fl, loss, rtol=1e-12, atol=1e-13)


def pin_finite_differences(ce):
    """Central differences of sum_t g_t loss_t in float64 match the analytic dH and dW."""
    H, W, t, g, _ = _problem(6, T=4, d=8, V=16, rows=(16,), ignore=(3,))
    loss, lse = ce.forward(H, W, t, IGN)
    dH, dW = ce.backward(H, W, t, lse, g, IGN)

    def L(Hx, Wx):
        l, _ = ce.forward(Hx, Wx, t, IGN)
        return float(np.dot(g, l))

    eps = 1e-6
    num_H = np.zeros_like(H)
    for idx in np.ndindex(*H.shape):
        Hp = H.copy(); Hp[idx] += eps
        Hm = H.copy(); Hm[idx] -= eps
        num_H[idx] = (L(Hp, W) - L(Hm, W)) / (2 * eps)
    num_W = np.zeros_like(W)
    for idx in np.ndindex(*W.shape):
        Wp = W.copy(); Wp[idx] += eps
        Wm = W.copy(); Wm[idx] -= eps
        num_W[idx] = (L(H, Wp) - L(H, Wm)) / (2 * eps)
    assert _rel(dH, num_H) <= 1e-7, _rel(dH, num_H)
    assert _rel(dW, num_W) <= 1e-7, _rel(dW, num_W)


def pin_ignore_masking(ce):
    """Ignored tokens: loss exactly 0, zero dH rows, and dW equal to dW without those tokens."""
    H, W, t, g, _ = _problem(7, T=10, d=4, V=11, rows=(11,), ignore=(0, 4, 9))
    loss, lse = ce.forward(H, W, t, IGN)
    dH, dW = ce.backward(H, W, t, lse, g, IGN)
    ign = t == IGN
    assert np.all(loss[ign] == 0.0)
    assert np.all(dH[ign] == 0.0)
    assert np.all(np.isfinite(lse))
    keep = ~ign
    loss_k, lse_k = ce.forward(H[keep], W, t[keep], IGN)
    dH_k, dW_k = ce.backward(H[keep], W, t[keep], lse_k, g[keep], IGN)
    np.testing.assert_allclose(dW, dW_k, rtol=1e-13, atol=1e-15)
    np.testing.assert_allclose(dH[keep], dH_k, rtol=1e-13, atol=1e-15)
    np.testing.assert_allclose(lse[keep], lse_k, rtol=1e-14)


def pin_invariants(ce):
    """sum_v dW_v = 0 (rows of G sum to 0); loss >= 0; max_v y <= lse <= max_v y + log V."""
    H, W, t, g, _ = _problem(8, T=12, d=7, V=30, rows=(30,), ignore=(5,), scale=3.0)
    loss, lse = ce.forward(H, W, t, IGN)
    dH, dW = ce.backward(H, W, t, lse, g, IGN)
    assert np.linalg.norm(dW.sum(axis=0)) <= 1e-13 * max(1.0, np.linalg.norm(dW))
    assert np.all(loss >= 0.0)
    Y = H @ W.T
    mx = Y.max(axis=1)
    assert np.all(mx <= lse + 1e-14) and np.all(lse <= mx + math.log(W.shape[0]) + 1e-14)


def pin_scalar_loops(ce):
    """Pure-Python triple loops agree with the numpy form (and both with the fold)."""
    H, W, t, g, shards = _problem(9, T=5, d=6, V=10, rows=(3, 7), ignore=(2,))
    sl, slse, sdH, sdW = ce.scalar_forward_backward(H, W, t, g, IGN)
    out = ce.forward_backward(H, shards, t, g, IGN)
    np.testing.assert_allclose(out["loss"], sl, rtol=1e-12, atol=1e-14)
    np.testing.assert_allclose(out["lse"], slse, rtol=1e-12)
    np.testing.assert_allclose(out["dH"], sdH, rtol=1e-12, atol=1e-14)
    np.testing.assert_allclose(out["dW"], sdW, rtol=1e-12, atol=1e-14)


def pin_torch_cross_entropy(ce):
    """Library cross-check: torch.nn.functional.cross_entropy in float64 on the CPU, with autograd."""
    import torch

    H, W, t, g, shards = _problem(10, T=16, d=12, V=40, rows=(10, 10, 20), ignore=(3, 11))
    Ht = torch.tensor(H, dtype=torch.float64, requires_grad=True)
    Wt = torch.tensor(W, dtype=torch.float64, requires_grad=True)
    tt = torch.tensor(t)
    lt = torch.nn.functional.cross_entropy(Ht @ Wt.T, tt, ignore_index=IGN, reduction="none")
    (lt * torch.tensor(g)).sum().backward()
    out = ce.forward_backward(H, shards, t, g, IGN)
    np.testing.assert_allclose(out["loss"], lt.detach().numpy(), rtol=1e-12, atol=1e-14)
    np.testing.assert_allclose(out["dH"], Ht.grad.numpy(), rtol=1e-12, atol=1e-14)
    np.testing.assert_allclose(out["dW"], Wt.grad.numpy(), rtol=1e-12, atol=1e-14)
    lse_t = torch.logsumexp(Ht.detach() @ Wt.detach().T, dim=1).numpy()
    np.testing.assert_allclose(out["lse"], lse_t, rtol=1e-13)


def pin_restrictions(ce):
    """Row and vocabulary-id restrictions equal the corresponding slices of the full result."""
    H, W, t, g, shards = _problem(11, T=14, d=5, V=25, rows=(25,), ignore=(1, 13))
    out = ce.forward_backward(H, shards, t, g, IGN)
    rows = np.array([0, 3, 7, 13])
    l_r, lse_r = ce.forward_rows(H, W, t, rows, IGN)
    np.testing.assert_allclose(l_r, out["loss"][rows], rtol=1e-14, atol=1e-15)
    np.testing.assert_allclose(lse_r, out["lse"][rows], rtol=1e-14)
    dH_r = ce.backward_rows(H, W, t, lse_r, g[rows], rows, IGN)
    np.testing.assert_allclose(dH_r, out["dH"][rows], rtol=1e-13, atol=1e-15)
    ids = np.array([0, 4, 24, int(t[0])])
    dW_v = ce.dW_rows(H, W, t, out["lse"], g, ids, IGN, row_chunk=5)
    np.testing.assert_allclose(dW_v, out["dW"][ids], rtol=1e-12, atol=1e-14)


def pin_out_of_range_target(ce):
    """A target outside [0, V) that is not ignore_index yields a NaN loss and NaN gradient row."""
    H, W, t, g, _ = _problem(12, T=4, d=3, V=6, rows=(6,), ignore=())
    t = t.copy()
    t[2] = 6
    loss, lse = ce.forward(H, W, t, IGN)
    assert np.isnan(loss[2]) and np.all(np.isfinite(np.delete(loss, 2)))
    dH, _ = ce.backward(H, W, t, lse, g, IGN)
    assert np.all(np.isnan(dH[2])) and np.all(np.isfinite(np.delete(dH, 2, axis=0)))


def pin_max_abs_logit(ce):
    """The largest |logit| both dense functions report equals a pure-Python scan of every
    h_t . w_v (the stress workload's logit scale is read from it)."""
    H, W, t, g, shards = _problem(13, T=7, d=4, V=9, rows=(4, 5), ignore=(2,), scale=2.0)
    # the largest magnitude sits in an interior token row, which is in neither the first
    # nor the last row chunk when the rows are cut into chunks of 1 to 3
    H[3] *= 6.0
    want = 0.0
    for i in range(H.shape[0]):
        for v in range(W.shape[0]):
            want = max(want, abs(sum(float(H[i, k]) * float(W[v, k]) for k in range(H.shape[1]))))
    _, _, got = ce.forward(H, W, t, IGN, return_max_abs=True)
    assert abs(got - want) <= 1e-13 * want, (got, want)
    got_fb = ce.forward_backward(H, shards, t, g, IGN)["max_abs_logit"]
    assert abs(got_fb - want) <= 1e-13 * want, (got_fb, want)


class _RowChunked:
    """The oracle with every row-chunked entry point forced to a given row chunk.

    The dense functions split the token rows into independent chunks (only dW sums
    across them).  The pins above use shapes far below the default chunk, so they run
    one chunk; through this view they run with chunks of 1, 2 and 3 rows, i.e. with
    every token in a chunk of its own, with chunk edges inside the batch and with a
    short last chunk.  Attributes are looked up on the wrapped module at call time, so
    a planted mistake in it is seen through the view."""

    _CHUNKED = ("forward", "backward", "forward_backward", "forward_rows", "backward_rows",
                "dW_rows")

    def __init__(self, ce, rc):
        self._ce = ce
        self._rc = rc

    def __getattr__(self, name):
        fn = getattr(self._ce, name)
        if name not in self._CHUNKED:
            return fn
        rc = self._rc

        def chunked(*args, **kw):
            kw["row_chunk"] = rc
            return fn(*args, **kw)
        return chunked


_CHUNK_PINS = (pin_golden_closed_form, pin_torch_cross_entropy, pin_finite_differences,
               pin_ignore_masking, pin_two_class_logistic, pin_restrictions,
               pin_zero_hidden_closed_form, pin_invariants, pin_scalar_loops, pin_max_abs_logit)


def pin_row_chunk_loop(ce):
    """The closed forms, library routine, finite differences, masking, two-class and
    restriction pins again with the token rows cut into chunks of 1, 2 and 3 rows, through
    every entry point that takes a row chunk (the full-size expected values are written by
    the same loop over many chunks)."""
    for rc in (1, 2, 3):
        view = _RowChunked(ce, rc)
        for pin in _CHUNK_PINS:
            try:
                pin(view)
            except AssertionError as e:
                raise AssertionError(f"{pin.__name__} with row_chunk={rc}: {e}") from e


ALL_PINS = [
    pin_golden_closed_form,
    pin_uniform_logits,
    pin_zero_hidden_closed_form,
    pin_two_class_logistic,
    pin_shift_invariance,
    pin_fold_order_invariance,
    pin_fold_state_passing,
    pin_finite_differences,
    pin_ignore_masking,
    pin_invariants,
    pin_scalar_loops,
    pin_torch_cross_entropy,
    pin_restrictions,
    pin_out_of_range_target,
    pin_max_abs_logit,
    pin_row_chunk_loop,
]
