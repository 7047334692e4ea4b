// Internal interface between the host API (vpce_api.cpp) and the kernels.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <algorithm>

#include "vpce.h"

namespace vpce {

// Vocabulary shards in visiting order: position i is shard order[i].
struct ShardTable {
  const void* w[VP_MAX_SHARDS];   // device [rows[i], d]
  int64_t off[VP_MAX_SHARDS];     // global id of the shard's first row
  int32_t rows[VP_MAX_SHARDS];    // V_p
  int32_t tile0[VP_MAX_SHARDS + 1];  // first forward tile index of position i (prefix sums)
  int32_t P;
};

struct FwdArgs {
  ShardTable st;
  const void* H;
  const int64_t* targets;
  int64_t T;
  int32_t d;
  int32_t n_tok_blocks, n_splits, n_tiles;
  float* m_part;  // [n_splits][T]
  float* s_part;  // [n_splits][T]
  float* y_tgt;   // [T]
};

struct CombArgs {
  const float* m_part;
  const float* s_part;
  const float* y_tgt;
  const int64_t* targets;
  int64_t T, V, ignore_index;
  int32_t n_splits;
  float* loss;
  float* lse;
  unsigned long long* bad_counter;
};

// Per-token fold state of Algorithm 2 as the ABI exposes it: float32 [3][T],
// planes m (running maximum logit, natural units), s (sum of e^(y - m) over the
// ids folded so far) and y (the target logit once its shard has been folded).
struct FoldArgs {
  const float* m_part;  // [n_splits][T], base-2 domain (max of y log2 e)
  const float* s_part;  // [n_splits][T]
  int64_t T;
  int32_t n_splits;
  float* state;
};

struct FinArgs {
  const float* state;
  const int64_t* targets;
  int64_t T, V, ignore_index;
  float* loss;
  float* lse;
  unsigned long long* bad_counter;
};

struct GradArgs {
  const void* W;   // first row of this vocabulary chunk, [M, d]
  const void* H;   // whole H [T, d]
  const int64_t* targets;
  const float* lse;
  const float* grad;
  // The residual strip in two layouts, Tc tokens by Vc vocabulary rows each,
  // k-blocked in 128-byte blocks of KB elements (64 bfloat16, 32 float32):
  // G [Tc/KB][Vc][KB] (element (v, t) at ((t / KB) Vc + v) KB + t % KB) and
  // G^T [Vc/KB][Tc][KB] (element (t, v) at ((v / KB) Tc + t) KB + v % KB), so that a
  // KB-deep slice of a 256-row tile of either operand is one contiguous 32 KiB block.
  void* strip;
  void* strip_t;
  int64_t Tc, Vc;
  int64_t t0;      // first token of this chunk
  int64_t gid0;    // global id of the chunk's first row
  int64_t V, ignore_index;
  const float* yt;  // [T] target logit h_t . w_{targets[t]} of every token (0 if none)
  int32_t M;       // vocabulary rows in this chunk
  int32_t N;       // tokens in this chunk
  int32_t d;
  int32_t n_vt;    // vocabulary tiles over M
};

// Target logits: yt[t] = h_t . w_{targets[t]} for targets in [0, V), 0 otherwise.  The
// shard table may list the shards in any order.
struct TgtArgs {
  ShardTable st;
  const void* H;
  const int64_t* targets;
  int64_t T, V;
  int32_t d;
  float* yt;
};

// C[M][N] = (beta ? C : 0) + A B^T with A [M][K] (row stride lda) and B [N][K]
// (row stride ldb), both k-contiguous.
struct GemmArgs {
  const void* A;
  int64_t lda;
  const void* B;
  int64_t ldb;
  float* C;
  int64_t ldc;
  int32_t M, N, K;
  int32_t beta;
  // elements between consecutive k-blocks (KB = 64 bfloat16 or 32 float32 wide)
  // of A and of B: KB for a row-major operand, rows * KB for a k-blocked one
  // (whose row pitch is KB)
  int64_t kblka, kblkb;
};

// out[c][r] = in[r][c] for r < R (zero for R <= r < R_pad), c < C.  in is
// row-major with pitch ld_in; out is k-blocked in 128-byte blocks of KB elements
// (64 bfloat16, 32 float32), [R_pad/KB][C][KB] (element (c, r) at
// ((r / KB) C + c) KB + r % KB).  C and ld_in are whole 16-byte vectors, R_pad a
// multiple of KB.
struct TransposeArgs {
  const void* in;
  int64_t ld_in;
  void* out;
  int32_t R, C, R_pad;
};

struct TileShape {
  int fwd_bm, fwd_bn, grad_bm, grad_bn;
  int kalign;  // the dH / dW contractions are launched with K rounded up to this
  int kblock;  // elements of one 128-byte k-block of the backward workspaces
};

TileShape tile_shape(int dtype);

// Bytes of the library-owned device workspace of vp_ce_forward_noalloc.
constexpr size_t kScratchBytes = 16u << 20;
// Device address of that workspace on the current device (looked up on the first
// call per device and kept); false if the lookup fails.
bool scratch_base(void** out);
bool run_ws_init(unsigned long long* counter, hipStream_t s);
bool run_fill_zero(float* p, int64_t n, hipStream_t s);
bool run_fwd(int dtype, const FwdArgs& a, hipStream_t s);
bool run_comb(const CombArgs& a, hipStream_t s);
bool run_state_init(float* state, int64_t T, hipStream_t s);
bool run_fold_merge(const FoldArgs& a, hipStream_t s);
bool run_fold_finalize(const FinArgs& a, hipStream_t s);
bool run_count_bad(const int64_t* targets, int64_t T, int64_t V, int64_t ignore_index,
                   unsigned long long* counter, hipStream_t s);
// Per-XCD tile counts of one backward stage launch (dH, dW, residual tiles).
struct StageSplit {
  int32_t cnt[3][8], first[3][8];
};

// One backward stage: the dH (h) and dW (w) tiles of one strip and the residual
// tiles (g) of the next strip, in one launch.  A kind with M == 0 is absent.
bool run_bwd_stage(int dtype, const GemmArgs& h, const GemmArgs& w, const GradArgs& g,
                   hipStream_t s);
bool run_transpose(int dtype, const TransposeArgs& a, hipStream_t s);
bool run_target_logits(int dtype, const TgtArgs& a, hipStream_t s);

}  // namespace vpce
