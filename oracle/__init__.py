"""CPU oracle for the fused vocabulary-projection cross-entropy (test infrastructure).

TEST INFRASTRUCTURE ONLY.  Nothing in the product path may import, call, link or
execute anything in this package: only the tests, the smoke check and the
benchmark's CPU-baseline leg use it.  It shares no code with the HIP path and
imports nothing from the repository.

What it computes (Sec. 3.2 of the paper, and the appendix section on Ring-DTP):

* forward: for every token t with hidden state h_t and every vocabulary row w_v,
  the logit y_tv = h_t . w_v; the per-token normaliser lse_t = log sum_v e^{y_tv};
  the negative log-likelihood loss_t = lse_t - y_{t, target_t}, and 0 for a token
  whose target is ``ignore_index``;
* backward (the paper promises but does not print the formulas; the reading used
  here is the textbook softmax cross-entropy gradient): with upstream per-token
  gradient g_t, G_tv = g_t (e^{y_tv - lse_t} - [v = target_t]) (0 on ignored
  tokens), dH = G W and dW = G^T H, W being the vocabulary projection in
  [V, d] row layout;
* the ring form of the forward: Algorithm 2's Fold applied shard by shard in any
  visiting order, the running state (m, z, y) starting at (-inf, 0, 0); one
  meeting (``fold_shard``) is what a move-activations hop carries the state
  through, and ``fold_finalize`` turns the state into (loss, lse).

Everything is float64.  Inputs arrive as the exact float64 widening of the bits
the GPU path receives.  Every function here is pinned by a test in
``tests/test_oracle_pins.py`` to something other than itself.
"""
from .ce import (  # noqa: F401
    backward,
    backward_rows,
    concat_shards,
    dW_rows,
    fold_finalize,
    fold_init,
    fold_shard,
    forward,
    forward_backward,
    forward_rows,
    ring_forward,
    scalar_forward_backward,
)
