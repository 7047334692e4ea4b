/*
 * vpce.h: fused vocabulary-projection softmax cross-entropy for one GPU's share
 * of a Ring-DTP vocabulary projection (arXiv 2609.14306, Sec. 3.2 and the
 * appendix section on Ring-DTP, Algorithm 2), for AMD Instinct MI355X (gfx950).
 *
 * Problem (Sec. 3.2 notation in brackets):
 *   H        [T, d]   hidden states of the T local tokens          [X_r, N x H]
 *   W_p      [V_p, d] vocabulary shard p, row layout (one row per vocabulary
 *                     id), owning global ids [off_p, off_p + V_p) with
 *                     off_p = V_0 + ... + V_{p-1}                  [W_r^T, V_r]
 *   targets  [T]      int64 target ids, or ignore_index
 *   y_tv = h_t . w_v  logit of token t and vocabulary id v
 *
 * The forward visits the shards in `order` (the ring's visiting order: on rank
 * r of a move-weights ring that is r, r-1, ..., r-P+1 mod P, Algorithm 2) and
 * folds each block of logits into a running per-token state (m, s, y_target)
 * with the online-softmax update of Sec. 3.2; no logits tensor larger than a
 * fixed register tile is ever formed.  The backward recomputes each block of
 * logits from the saved normaliser lse, forms the softmax residual and
 * contracts it into the input and weight gradients (appendix on Ring-DTP),
 * staging the residual through a fixed-size strip buffer.  Every buffer the
 * library uses is allocated by the caller; the workspace size depends on T and
 * the strip budget, never on V.
 *
 * Conventions for every entry point:
 *   - device pointers are HIP device (or managed) memory on the current device;
 *     "host" arrays are ordinary CPU memory read before the call returns;
 *   - dense arrays are row-major and contiguous; H, every W_p and the workspace
 *     must be 16-byte aligned;
 *   - `stream` is a hipStream_t (NULL = the null stream); all work is enqueued
 *     on it and the call returns without synchronising (except vp_ce_check);
 *   - argument, shape, alignment and workspace errors are returned before any
 *     work is enqueued; a failed launch returns VP_ERR_HIP;
 *   - the library keeps no pointer after a call returns and has no global
 *     mutable state: calls on different streams with different workspaces may
 *     run concurrently.
 */
#ifndef VPCE_H
#define VPCE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define VPCE_ABI_VERSION 1
#define VP_MAX_SHARDS 64

typedef enum {
  VP_OK = 0,
  VP_ERR_NULL = 1,        /* a required pointer is NULL */
  VP_ERR_SHAPE = 2,       /* T out of [0, 2^23 - 256], d out of [8, 2^22] or d % 8 != 0,
                             P out of [1, VP_MAX_SHARDS], V_p out of [0, 2^30], sum V_p out of
                             [1, 2^31 - 1], strip_elems out of [0, 2^30] */
  VP_ERR_DTYPE = 3,       /* dtype is not VP_F32 / VP_BF16 */
  VP_ERR_ORDER = 4,       /* order is not a permutation of 0..P-1 */
  VP_ERR_ALIGN = 5,       /* a device pointer is not 16-byte aligned (4 for a fold state) */
  VP_ERR_WORKSPACE = 6,   /* workspace pointer NULL or smaller than the size the library asked for */
  VP_ERR_TARGET = 7,      /* (vp_ce_check) some target was outside [0, V) and not ignore_index */
  VP_ERR_HIP = 8,         /* a HIP runtime call or a kernel launch failed */
  VP_ERR_UNSUPPORTED = 9  /* valid request the library does not implement */
} vp_status;

typedef enum {
  VP_F32 = 0,  /* H and W in float32; logits, residual and gradients in float32 */
  VP_BF16 = 1  /* H and W in bfloat16; products accumulated in float32; the residual
                  staged as bfloat16 (round to nearest even); gradients in float32 */
} vp_dtype;

/* flags */
#define VP_ACCUMULATE_DW 1u /* backward adds into dW_p instead of overwriting it: on a
                               move-weights ring the weight gradient travels with the
                               weight shard and collects every rank's contribution */

typedef struct {
  int64_t T;                  /* local tokens, 0..2^23 - 256 (T == 0 is a no-op) */
  int64_t d;                  /* hidden width, 8..2^22 and a multiple of 8 */
  int32_t P;                  /* number of vocabulary shards, 1..VP_MAX_SHARDS */
  int32_t dtype;              /* vp_dtype of H and W */
  const int64_t* shard_rows;  /* host [P]: V_p >= 0 rows of shard p, sum >= 1 */
  const int32_t* order;       /* host [P]: visiting order, a permutation of 0..P-1; NULL = 0..P-1 */
  int64_t ignore_index;       /* target value that marks a token without loss (e.g. -100) */
  uint32_t flags;             /* VP_ACCUMULATE_DW */
  int64_t strip_elems;        /* backward residual-strip budget in elements per layout,
                                 0..2^30; 0 = default (100 Mi) */
} vp_problem;

/* Workspace sizes in bytes for vp_ce_forward (*fwd_bytes) and vp_ce_backward
 * (*bwd_bytes); either output pointer may be NULL.  Host only, needs no device.
 * forward: per-token partial states of the vocabulary splits, O(T);
 * backward: the residual strip in two layouts, twice (one being written while
 * the other is contracted: 4 x strip_elems elements at most), H^T (T x d
 * elements, T rounded up to 256) and W^T of one vocabulary chunk (d x strip
 * columns).  Neither depends on V. */
vp_status vp_ce_workspace_size(const vp_problem* prob, size_t* fwd_bytes, size_t* bwd_bytes);

/* Forward (Sec. 3.2, Eq. of the online-softmax fold; Algorithm 2):
 *   lse[t]  = log sum_{v < V} exp(y_tv)                       (float32, device [T])
 *   loss[t] = lse[t] - y_{t, targets[t]},  0 if targets[t] == ignore_index,
 *             NaN if targets[t] is outside [0, V) (also counted for vp_ce_check)
 * H: device [T, d] of dtype; W_shards: host array of P device pointers, shard p
 * is [V_p, d] of dtype (NULL allowed when V_p == 0); targets: device int64 [T];
 * ws: device workspace of at least the forward size.  lse is the saved
 * normaliser the backward replays from. */
vp_status vp_ce_forward(const vp_problem* prob, const void* H, const void* const* W_shards,
                        const int64_t* targets, float* loss, float* lse, void* ws,
                        size_t ws_bytes, void* stream);

/* The forward for callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid allocation): the same as
 * vp_ce_forward, with the same kernels and results, but its workspace is a
 * library-owned device buffer of 16 MiB per device (held from the first call on a
 * device until the process ends), so the call allocates nothing.  The caller still
 * passes H, the shards, the targets and the outputs.
 *   - Returns VP_ERR_WORKSPACE before any work is enqueued if the problem's forward
 *     workspace (vp_ce_workspace_size) exceeds 16 MiB (about T <= 460000 tokens at the
 *     usual split counts).
 *   - Every call on one device shares that device's buffer: calls that overlap on a
 *     device (different streams or threads) race and give wrong results; calls
 *     ordered on one stream are safe.
 *   - The count of out-of-range targets is kept in that buffer and is not reported
 *     (vp_ce_check needs a caller's workspace); such tokens still get a NaN loss.
 *   - The first call on a device looks up the buffer's device address (no
 *     allocation); VP_ERR_HIP if that fails. */
vp_status vp_ce_forward_noalloc(const vp_problem* prob, const void* H,
                                const void* const* W_shards, const int64_t* targets,
                                float* loss, float* lse, void* stream);

/* Backward (appendix on Ring-DTP: recompute each block of logits from the saved
 * normaliser, form the softmax residual, contract into both gradients):
 *   G[t, v]  = grad_loss[t] * (exp(y_tv - lse[t]) - [v == targets[t]]),
 *              0 on ignored tokens, NaN on out-of-range targets
 *   dH       = G W            device float32 [T, d], overwritten
 *   dW_p     = G[:, shard p]^T H   device float32 [V_p, d] per shard (host array of
 *              P device pointers; NULL allowed when V_p == 0), overwritten, or
 *              added to with VP_ACCUMULATE_DW
 * lse: device float32 [T] from vp_ce_forward on the same inputs; grad_loss:
 * device float32 [T] upstream gradient of each token's loss (1/N_valid for a
 * mean, 1 for a sum). */
vp_status vp_ce_backward(const vp_problem* prob, const void* H, const void* const* W_shards,
                         const int64_t* targets, const float* lse, const float* grad_loss,
                         float* dH, float* const* dW_shards, void* ws, size_t ws_bytes,
                         void* stream);

/* Per-shard fold: one meeting of Algorithm 2 at a time, for a per-token state
 * that travels with the activations (move-activations: the hidden states, the
 * targets and the state visit the ranks that hold the vocabulary shards, and a
 * final hop returns the state to its owner, Sec. 3.2 and Algorithm 2).
 *
 * State: device float32 [3 * T], three planes of T values:
 *   m[t]  = state[t]          running maximum logit over the vocabulary ids folded so
 *                             far (natural units), -inf before the first shard;
 *   s[t]  = state[T + t]      sum over those ids of exp(y_tv - m[t]);
 *   y[t]  = state[2T + t]     the target logit h_t . w_{targets[t]} once the shard
 *                             owning targets[t] has been folded, 0 before.
 * The planes are plain numbers in host byte order: the state is serialised by
 * copying its 12 T bytes, on any device or the host, and folding may resume
 * from such a copy on another device.  Folding is order-free up to rounding
 * (the online-softmax update is associative and commutative). */

/* state <- (-inf, 0, 0) for every token.  state: device float32 [3 * T], 4-byte
 * aligned; T in [0, 2^23 - 256] (VP_ERR_SHAPE otherwise). */
vp_status vp_ce_state_init(float* state, int64_t T, void* stream);

/* Folds one vocabulary shard into the state (the online-softmax update of Sec. 3.2):
 *   m' = max(m, max_v y_tv),  s' = s e^(m - m') + sum_v e^(y_tv - m'),
 *   y' = y_{t, targets[t]} where id_offset <= targets[t] < id_offset + V_q, else y.
 * shard: a vp_problem with P == 1 whose shard_rows[0] = V_q are the shard's rows
 * (T, d, dtype as for vp_ce_forward; order NULL or {0}; ignore_index, flags and
 * strip_elems unused); id_offset: the global vocabulary id of the shard's first
 * row (id_offset + V_q <= 2^31 - 1).  H: device [T, d]; W_shard: device [V_q, d]
 * (NULL allowed when V_q == 0); targets: device int64 [T] of global ids; state as
 * above, updated in place.  ws: the forward workspace of `shard`
 * (vp_ce_workspace_size(shard, &fwd, NULL); it depends on T, d and dtype, never on
 * V_q), 16-byte aligned.  V_q == 0 or T == 0 returns VP_OK before anything else is
 * checked or launched and leaves the state unchanged: ws, H, W_shard, targets and
 * state may then be NULL. */
vp_status vp_ce_fold_shard(const vp_problem* shard, int64_t id_offset, const void* H,
                           const void* W_shard, const int64_t* targets, float* state, void* ws,
                           size_t ws_bytes, void* stream);

/* From a state that has met every shard of the vocabulary described by `prob`
 * (V = sum of its shard_rows; T and ignore_index as for vp_ce_forward):
 *   lse[t]  = m[t] + log s[t],
 *   loss[t] = lse[t] - y[t], 0 if targets[t] == ignore_index, NaN if targets[t] is
 *             outside [0, V) (counted in ws for vp_ce_check).
 * The state is only read.  ws: at least 256 bytes (the forward workspace of any
 * problem is enough), 16-byte aligned. */
vp_status vp_ce_fold_finalize(const vp_problem* prob, const int64_t* targets, const float* state,
                              float* loss, float* lse, void* ws, size_t ws_bytes, void* stream);

/* How vp_ce_backward cuts a problem (host only, needs no device): the residual
 * strip is Tc tokens by at most Vc vocabulary rows; `strips` strips cover the
 * T x V residual (each shard cut into balanced vocabulary chunks, each chunk
 * meeting every token chunk), and the backward makes stage_launches = strips + 1
 * launches of its fused recompute / residual / dH / dW kernel (0 when T == 0). */
typedef struct {
  int64_t Tc;
  int64_t Vc;
  int64_t strips;
  int64_t stage_launches;
} vp_plan_info;
vp_status vp_ce_plan_info(const vp_problem* prob, vp_plan_info* info);

/* Reads the count of out-of-range targets that the last forward or backward on
 * this workspace found (synchronises `stream`).  Returns VP_ERR_TARGET if it is
 * non-zero.  *bad_targets may be NULL. */
vp_status vp_ce_check(const void* ws, void* stream, int64_t* bad_targets);

const char* vp_status_str(vp_status s);
int vp_abi_version(void);

#ifdef __cplusplus
}
#endif
#endif /* VPCE_H */
