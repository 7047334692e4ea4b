// Host side of the C ABI declared in include/vpce.h: argument validation,
// workspace planning and launch sequencing.  Every argument, shape, alignment
// and workspace error is detected here before any HIP call is made, so these
// paths run (and are tested) on a machine without a GPU.
#include <hip/hip_runtime.h>
#include <stdint.h>
#include <string.h>

#include <algorithm>
#include <cmath>
#include <vector>

#include "vpce_internal.h"

namespace {

constexpr size_t kHeaderBytes = 256;       // error counter + reserved
constexpr int64_t kDefaultStrip = 100ll << 20;  // residual-strip budget in elements per layout
constexpr int64_t kCUs = 256;                      // compute units of one MI355X
constexpr int64_t kPanelCacheBudget = 160ll << 20;  // of the 256 MiB memory-side cache
constexpr int kMaxSplits = 32;

inline size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }
inline int64_t round_up(int64_t x, int64_t m) { return (x + m - 1) / m * m; }
inline int64_t round_down(int64_t x, int64_t m) { return x / m * m; }
inline int64_t ceil_div(int64_t x, int64_t m) { return (x + m - 1) / m; }

size_t elem_bytes(int dtype) { return dtype == VP_BF16 ? 2 : 4; }

constexpr int64_t kMaxT = (1ll << 23) - 256;
constexpr int64_t kMaxD = 1ll << 22;

vp_status validate(const vp_problem* p, int64_t* V_out, bool allow_empty_vocab = false) {
  if (!p) return VP_ERR_NULL;
  if (p->dtype != VP_F32 && p->dtype != VP_BF16) return VP_ERR_DTYPE;
  // The bf16 GEMM tiles address a 256-row operand tile with 32-bit byte offsets
  // (256 rows x leading dimension x 2 bytes < 2^32): leading dimensions are d,
  // the padded token count and strip widths, so T and d are capped below 2^23.
  if (p->T < 0 || p->d < 8 || p->d % 8 != 0 || p->d > kMaxD) return VP_ERR_SHAPE;
  if (p->T > kMaxT) return VP_ERR_SHAPE;
  if (p->P < 1 || p->P > VP_MAX_SHARDS) return VP_ERR_SHAPE;
  if (!p->shard_rows) return VP_ERR_NULL;
  if (p->strip_elems < 0 || p->strip_elems > (1ll << 30)) return VP_ERR_SHAPE;
  int64_t V = 0;
  for (int i = 0; i < p->P; ++i) {
    if (p->shard_rows[i] < 0 || p->shard_rows[i] > (1ll << 30)) return VP_ERR_SHAPE;
    V += p->shard_rows[i];
  }
  if (V < (allow_empty_vocab ? 0 : 1) || V > (1ll << 31) - 1) return VP_ERR_SHAPE;
  if (p->order) {
    bool seen[VP_MAX_SHARDS] = {false};
    for (int i = 0; i < p->P; ++i) {
      const int q = p->order[i];
      if (q < 0 || q >= p->P || seen[q]) return VP_ERR_ORDER;
      seen[q] = true;
    }
  }
  if (V_out) *V_out = V;
  return VP_OK;
}

inline bool misaligned(const void* ptr) { return ((uintptr_t)ptr & 15u) != 0; }

// Vocabulary splits of the forward: workgroup (token block, split) folds one token
// block over one contiguous range of the vocabulary tiles, and an XCD runs 32
// consecutive workgroups at a time, i.e. 32 / S token blocks by S splits.  S is the
// smallest power of two (at most 32) that
// - fills the CUs (token blocks x S >= 256);
// - is at least 4, so that those 32 tiles share 12 operand panels in the XCD's L2
//   (8 x 4 or 4 x 8);
// - keeps the H panels of the 256 / S token blocks running at once within 160 MiB,
//   so that they stay in the memory-side cache while every vocabulary tile re-reads
//   them.
int splits_for(const vp_problem* p) {
  const vpce::TileShape ts = vpce::tile_shape(p->dtype);
  const int64_t tok_blocks = std::max<int64_t>(1, ceil_div(p->T, ts.fwd_bn));
  const int64_t panel = (int64_t)ts.fwd_bn * p->d * (int64_t)elem_bytes(p->dtype);
  const int64_t need = std::max<int64_t>(
      4, std::max(ceil_div(kCUs, tok_blocks), ceil_div(kCUs * panel, kPanelCacheBudget)));
  int s = 4;
  while (s < need && s < kMaxSplits) s *= 2;
  return s;
}

size_t fwd_ws_bytes(const vp_problem* p) {
  const size_t T = (size_t)p->T;
  const size_t S = (size_t)splits_for(p);
  return kHeaderBytes + 2 * align256(S * T * 4) + align256(T * 4);
}

// Backward plan.  The softmax residual of a strip of Tc tokens by Vc
// vocabulary rows is staged in both layouts (G [Vc][Tc] and G^T [Tc][Vc]),
// twice: one launch writes the residual of strip c+1 while it contracts strip
// c into dH and dW.  Tc*Vc <= budget; tokens in balanced chunks no larger than
// the square root of the budget (the float32 read-modify-write traffic of dH
// across vocabulary chunks plus that of dW across token chunks is proportional
// to 1/Vc + 1/Tc).  The workspace also holds H^T [d][T_pad] (written once per
// call) and W^T [d][Vc] of the current vocabulary chunk.  Nothing here depends
// on V.
struct StripPlan {
  int64_t Tc, Vc, T_pad;
  size_t off_g[2], off_gt[2], off_ht, off_wt, off_yt, total;
};

StripPlan strip_plan(const vp_problem* p) {
  const vpce::TileShape ts = vpce::tile_shape(p->dtype);
  const int64_t budget = p->strip_elems > 0 ? p->strip_elems : kDefaultStrip;
  const int64_t T = std::max<int64_t>(p->T, 1);
  const int64_t side = std::max<int64_t>(ts.grad_bn, round_down((int64_t)std::sqrt((double)budget), ts.grad_bn));
  StripPlan s;
  s.Tc = std::min<int64_t>(round_up(T, ts.grad_bn), round_up(ceil_div(T, ceil_div(T, side)), ts.grad_bn));
  s.Vc = std::max<int64_t>(ts.grad_bm, std::min<int64_t>(round_down(budget / s.Tc, ts.grad_bm),
                                                        32768));
  s.T_pad = round_up(T, 256);
  const size_t eb = elem_bytes(p->dtype);
  const size_t strip = align256((size_t)s.Vc * s.Tc * eb);
  size_t off = kHeaderBytes;
  for (int b = 0; b < 2; ++b) {
    s.off_g[b] = off;
    s.off_gt[b] = off + strip;
    off += 2 * strip;
  }
  s.off_ht = off;
  s.off_wt = s.off_ht + align256((size_t)p->d * s.T_pad * eb);
  s.off_yt = s.off_wt + align256((size_t)p->d * s.Vc * eb);
  s.total = s.off_yt + align256((size_t)T * 4);
  return s;
}

size_t bwd_ws_bytes(const vp_problem* p) { return strip_plan(p).total; }

void build_table(const vp_problem* p, const void* const* W_shards, int bm, vpce::ShardTable* st,
                 int32_t* n_tiles) {
  int64_t off[VP_MAX_SHARDS];
  int64_t acc = 0;
  for (int q = 0; q < p->P; ++q) {
    off[q] = acc;
    acc += p->shard_rows[q];
  }
  st->P = p->P;
  int32_t tiles = 0;
  for (int i = 0; i < p->P; ++i) {
    const int q = p->order ? p->order[i] : i;
    st->w[i] = W_shards[q];
    st->off[i] = off[q];
    st->rows[i] = (int32_t)p->shard_rows[q];
    st->tile0[i] = tiles;
    tiles += (int32_t)ceil_div(p->shard_rows[q], bm);
  }
  for (int i = p->P; i <= VP_MAX_SHARDS; ++i) st->tile0[i] = tiles;
  for (int i = p->P; i < VP_MAX_SHARDS; ++i) {
    st->w[i] = nullptr;
    st->off[i] = acc;
    st->rows[i] = 0;
  }
  *n_tiles = tiles;
}

vp_status check_shards(const vp_problem* p, const void* const* W_shards) {
  if (!W_shards) return VP_ERR_NULL;
  for (int q = 0; q < p->P; ++q) {
    if (p->shard_rows[q] > 0 && !W_shards[q]) return VP_ERR_NULL;
    if (p->shard_rows[q] > 0 && misaligned(W_shards[q])) return VP_ERR_ALIGN;
  }
  return VP_OK;
}

// The strips of a backward call in visiting order: shards in `order`, each cut
// into balanced, tile-aligned vocabulary chunks (never above Vc), each chunk
// meeting every token chunk.
struct Chunk {
  int q;
  int64_t v0, M, t0, N;
  bool new_vchunk, first_vchunk;
};

std::vector<Chunk> strip_chunks(const vp_problem* prob, const StripPlan& plan) {
  const vpce::TileShape ts = vpce::tile_shape(prob->dtype);
  std::vector<Chunk> chunks;
  bool first = true;
  for (int i = 0; i < prob->P; ++i) {
    const int q = prob->order ? prob->order[i] : i;
    const int64_t Vq = prob->shard_rows[q];
    if (Vq == 0) continue;
    const int64_t vc =
        std::min<int64_t>(plan.Vc, round_up(ceil_div(Vq, ceil_div(Vq, plan.Vc)), ts.grad_bm));
    for (int64_t v0 = 0; v0 < Vq; v0 += vc) {
      for (int64_t t0 = 0; t0 < prob->T; t0 += plan.Tc)
        chunks.push_back({q, v0, std::min<int64_t>(vc, Vq - v0), t0,
                          std::min<int64_t>(plan.Tc, prob->T - t0), t0 == 0, first});
      first = false;
    }
  }
  return chunks;
}

}  // namespace

extern "C" {

int vp_abi_version(void) { return VPCE_ABI_VERSION; }

const char* vp_status_str(vp_status s) {
  switch (s) {
    case VP_OK: return "ok";
    case VP_ERR_NULL: return "a required pointer is NULL";
    case VP_ERR_SHAPE: return "invalid shape (T, d, P or shard rows)";
    case VP_ERR_DTYPE: return "unsupported dtype";
    case VP_ERR_ORDER: return "order is not a permutation of the shards";
    case VP_ERR_ALIGN: return "a device pointer is not 16-byte aligned";
    case VP_ERR_WORKSPACE: return "workspace missing or too small";
    case VP_ERR_TARGET: return "a target is outside [0, V) and not ignore_index";
    case VP_ERR_HIP: return "HIP runtime or kernel launch failure";
    case VP_ERR_UNSUPPORTED: return "unsupported request";
  }
  return "unknown status";
}

vp_status vp_ce_workspace_size(const vp_problem* prob, size_t* fwd_bytes, size_t* bwd_bytes) {
  const vp_status st = validate(prob, nullptr);
  if (st != VP_OK) return st;
  if (fwd_bytes) *fwd_bytes = fwd_ws_bytes(prob);
  if (bwd_bytes) *bwd_bytes = bwd_ws_bytes(prob);
  return VP_OK;
}

}  // extern "C"

namespace {

// Argument checks of the forward shared by vp_ce_forward and vp_ce_forward_noalloc
// (everything except the workspace).
vp_status check_forward(const vp_problem* prob, const void* H, const void* const* W_shards,
                        const int64_t* targets, float* loss, float* lse, int64_t* V) {
  vp_status st = validate(prob, V);
  if (st != VP_OK) return st;
  if ((st = check_shards(prob, W_shards)) != VP_OK) return st;
  if (prob->T > 0) {
    if (!H || !targets || !loss || !lse) return VP_ERR_NULL;
    if (misaligned(H)) return VP_ERR_ALIGN;
  }
  return VP_OK;
}

// The forward on a checked problem, with a workspace of at least fwd_ws_bytes(prob).
vp_status forward_impl(const vp_problem* prob, int64_t V, const void* H,
                       const void* const* W_shards, const int64_t* targets, float* loss,
                       float* lse, void* ws, hipStream_t s) {
  const int64_t T = prob->T;
  unsigned long long* counter = (unsigned long long*)ws;
  if (!vpce::run_ws_init(counter, s)) return VP_ERR_HIP;
  if (T == 0) return VP_OK;

  const vpce::TileShape ts = vpce::tile_shape(prob->dtype);
  const int S = splits_for(prob);
  char* base = (char*)ws + kHeaderBytes;
  vpce::FwdArgs a;
  memset(&a, 0, sizeof(a));
  build_table(prob, W_shards, ts.fwd_bm, &a.st, &a.n_tiles);
  a.H = H;
  a.targets = targets;
  a.T = T;
  a.d = (int32_t)prob->d;
  a.n_tok_blocks = (int32_t)ceil_div(T, ts.fwd_bn);
  a.n_splits = S;
  a.m_part = (float*)base;
  a.s_part = (float*)(base + align256((size_t)S * T * 4));
  a.y_tgt = (float*)(base + 2 * align256((size_t)S * T * 4));
  if (!vpce::run_fwd(prob->dtype, a, s)) return VP_ERR_HIP;

  vpce::CombArgs c;
  c.m_part = a.m_part;
  c.s_part = a.s_part;
  c.y_tgt = a.y_tgt;
  c.targets = targets;
  c.T = T;
  c.V = V;
  c.ignore_index = prob->ignore_index;
  c.n_splits = S;
  c.loss = loss;
  c.lse = lse;
  c.bad_counter = counter;
  if (!vpce::run_comb(c, s)) return VP_ERR_HIP;
  return VP_OK;
}

}  // namespace

extern "C" {

vp_status vp_ce_forward(const vp_problem* prob, const void* H, const void* const* W_shards,
                        const int64_t* targets, float* loss, float* lse, void* ws,
                        size_t ws_bytes, void* stream) {
  int64_t V = 0;
  vp_status st = validate(prob, &V);
  if (st != VP_OK) return st;
  if ((st = check_shards(prob, W_shards)) != VP_OK) return st;
  if (!ws) return VP_ERR_WORKSPACE;
  if (ws_bytes < fwd_ws_bytes(prob)) return VP_ERR_WORKSPACE;
  if (misaligned(ws)) return VP_ERR_ALIGN;
  if ((st = check_forward(prob, H, W_shards, targets, loss, lse, &V)) != VP_OK) return st;
  return forward_impl(prob, V, H, W_shards, targets, loss, lse, ws, (hipStream_t)stream);
}

vp_status vp_ce_forward_noalloc(const vp_problem* prob, const void* H,
                                const void* const* W_shards, const int64_t* targets,
                                float* loss, float* lse, void* stream) {
  int64_t V = 0;
  const vp_status st = check_forward(prob, H, W_shards, targets, loss, lse, &V);
  if (st != VP_OK) return st;
  if (fwd_ws_bytes(prob) > vpce::kScratchBytes) return VP_ERR_WORKSPACE;
  void* ws = nullptr;
  if (!vpce::scratch_base(&ws)) return VP_ERR_HIP;
  return forward_impl(prob, V, H, W_shards, targets, loss, lse, ws, (hipStream_t)stream);
}

vp_status vp_ce_state_init(float* state, int64_t T, void* stream) {
  if (T < 0 || T > kMaxT) return VP_ERR_SHAPE;
  if (T == 0) return VP_OK;
  if (!state) return VP_ERR_NULL;
  if (((uintptr_t)state & 3u) != 0) return VP_ERR_ALIGN;
  return vpce::run_state_init(state, T, (hipStream_t)stream) ? VP_OK : VP_ERR_HIP;
}

vp_status vp_ce_fold_shard(const vp_problem* shard, int64_t id_offset, const void* H,
                           const void* W_shard, const int64_t* targets, float* state, void* ws,
                           size_t ws_bytes, void* stream) {
  int64_t Vq = 0;
  vp_status st = validate(shard, &Vq, /*allow_empty_vocab=*/true);
  if (st != VP_OK) return st;
  if (shard->P != 1) return VP_ERR_SHAPE;
  if (id_offset < 0 || id_offset > (1ll << 31) - 1 - Vq) return VP_ERR_SHAPE;
  const int64_t T = shard->T;
  // an empty strip leaves the state unchanged: nothing is launched, nothing is read
  if (T == 0 || Vq == 0) return VP_OK;
  if (!ws) return VP_ERR_WORKSPACE;
  if (ws_bytes < fwd_ws_bytes(shard)) return VP_ERR_WORKSPACE;
  if (misaligned(ws)) return VP_ERR_ALIGN;
  if (!H || !W_shard || !targets || !state) return VP_ERR_NULL;
  if (misaligned(H) || misaligned(W_shard)) return VP_ERR_ALIGN;
  if (((uintptr_t)state & 3u) != 0) return VP_ERR_ALIGN;
  hipStream_t s = (hipStream_t)stream;

  const vpce::TileShape ts = vpce::tile_shape(shard->dtype);
  const int32_t tiles = (int32_t)ceil_div(Vq, ts.fwd_bm);
  const int S = std::min(splits_for(shard), (int)tiles);
  char* base = (char*)ws + kHeaderBytes;
  vpce::FwdArgs a;
  memset(&a, 0, sizeof(a));
  a.st.P = 1;
  a.st.w[0] = W_shard;
  a.st.off[0] = id_offset;
  a.st.rows[0] = (int32_t)Vq;
  a.st.tile0[0] = 0;
  for (int i = 1; i <= VP_MAX_SHARDS; ++i) a.st.tile0[i] = tiles;
  for (int i = 1; i < VP_MAX_SHARDS; ++i) a.st.off[i] = id_offset + Vq;
  a.n_tiles = tiles;
  a.H = H;
  a.targets = targets;
  a.T = T;
  a.d = (int32_t)shard->d;
  a.n_tok_blocks = (int32_t)ceil_div(T, ts.fwd_bn);
  a.n_splits = S;
  a.m_part = (float*)base;
  a.s_part = (float*)(base + align256((size_t)S * T * 4));
  a.y_tgt = state + 2 * T;  // written only for targets this shard owns
  if (!vpce::run_fwd(shard->dtype, a, s)) return VP_ERR_HIP;

  vpce::FoldArgs f;
  f.m_part = a.m_part;
  f.s_part = a.s_part;
  f.T = T;
  f.n_splits = S;
  f.state = state;
  return vpce::run_fold_merge(f, s) ? VP_OK : VP_ERR_HIP;
}

vp_status vp_ce_fold_finalize(const vp_problem* prob, const int64_t* targets, const float* state,
                              float* loss, float* lse, void* ws, size_t ws_bytes, void* stream) {
  int64_t V = 0;
  vp_status st = validate(prob, &V);
  if (st != VP_OK) return st;
  if (!ws) return VP_ERR_WORKSPACE;
  if (ws_bytes < kHeaderBytes) return VP_ERR_WORKSPACE;
  if (misaligned(ws)) return VP_ERR_ALIGN;
  const int64_t T = prob->T;
  if (T > 0) {
    if (!targets || !state || !loss || !lse) return VP_ERR_NULL;
    if (((uintptr_t)state & 3u) != 0) return VP_ERR_ALIGN;
  }
  hipStream_t s = (hipStream_t)stream;
  unsigned long long* counter = (unsigned long long*)ws;
  if (!vpce::run_ws_init(counter, s)) return VP_ERR_HIP;
  vpce::FinArgs f;
  f.state = state;
  f.targets = targets;
  f.T = T;
  f.V = V;
  f.ignore_index = prob->ignore_index;
  f.loss = loss;
  f.lse = lse;
  f.bad_counter = counter;
  return vpce::run_fold_finalize(f, s) ? VP_OK : VP_ERR_HIP;
}

vp_status vp_ce_plan_info(const vp_problem* prob, vp_plan_info* info) {
  const vp_status st = validate(prob, nullptr);
  if (st != VP_OK) return st;
  if (!info) return VP_ERR_NULL;
  const StripPlan plan = strip_plan(prob);
  const int64_t n = prob->T > 0 ? (int64_t)strip_chunks(prob, plan).size() : 0;
  info->Tc = plan.Tc;
  info->Vc = plan.Vc;
  info->strips = n;
  info->stage_launches = n > 0 ? n + 1 : 0;
  return VP_OK;
}

vp_status vp_ce_backward(const vp_problem* prob, const void* H, const void* const* W_shards,
                         const int64_t* targets, const float* lse, const float* grad_loss,
                         float* dH, float* const* dW_shards, void* ws, size_t ws_bytes,
                         void* stream) {
  int64_t V = 0;
  vp_status st = validate(prob, &V);
  if (st != VP_OK) return st;
  if ((st = check_shards(prob, W_shards)) != VP_OK) return st;
  if (!dW_shards) return VP_ERR_NULL;
  for (int q = 0; q < prob->P; ++q) {
    if (prob->shard_rows[q] > 0 && !dW_shards[q]) return VP_ERR_NULL;
    if (prob->shard_rows[q] > 0 && misaligned(dW_shards[q])) return VP_ERR_ALIGN;
  }
  if (!ws) return VP_ERR_WORKSPACE;
  if (ws_bytes < bwd_ws_bytes(prob)) return VP_ERR_WORKSPACE;
  if (misaligned(ws)) return VP_ERR_ALIGN;
  const int64_t T = prob->T;
  if (T > 0) {
    if (!H || !targets || !lse || !grad_loss || !dH) return VP_ERR_NULL;
    if (misaligned(H) || misaligned(dH)) return VP_ERR_ALIGN;
  }
  hipStream_t s = (hipStream_t)stream;
  unsigned long long* counter = (unsigned long long*)ws;
  if (!vpce::run_ws_init(counter, s)) return VP_ERR_HIP;
  const bool accumulate = (prob->flags & VP_ACCUMULATE_DW) != 0;
  const int64_t d = prob->d;

  if (T == 0) {  // G is empty: dW = 0 (or unchanged when accumulating); dH has no rows
    if (!accumulate)
      for (int q = 0; q < prob->P; ++q)
        if (!vpce::run_fill_zero(dW_shards[q], prob->shard_rows[q] * d, s)) return VP_ERR_HIP;
    return VP_OK;
  }
  if (!vpce::run_count_bad(targets, T, V, prob->ignore_index, counter, s)) return VP_ERR_HIP;

  const vpce::TileShape ts = vpce::tile_shape(prob->dtype);
  const StripPlan plan = strip_plan(prob);
  char* wsb = (char*)ws;
  void* Ht = wsb + plan.off_ht;
  void* Wt = wsb + plan.off_wt;
  const size_t eb = elem_bytes(prob->dtype);
  // The workspaces (the residual strips, H^T and W^T) are k-blocked in 128-byte
  // blocks of KB elements (64 bfloat16, 32 float32): every k-slice of a 256-row
  // tile the dH / dW contractions stream is one contiguous 32 KiB block.
  const int64_t KB = ts.kblock;

  {  // H^T [d][T_pad], k-blocked: [T_pad/KB][d][KB], zero beyond T
    vpce::TransposeArgs tr;
    tr.in = H;
    tr.ld_in = d;
    tr.out = Ht;
    tr.R = (int32_t)T;
    tr.C = (int32_t)d;
    tr.R_pad = (int32_t)plan.T_pad;
    if (!vpce::run_transpose(prob->dtype, tr, s)) return VP_ERR_HIP;
  }

  float* yt = (float*)(wsb + plan.off_yt);
  {  // the target logit of every token, read by the residual tiles for the one-hot term
    vpce::TgtArgs ta;
    memset(&ta, 0, sizeof(ta));
    int32_t n_tiles = 0;
    build_table(prob, W_shards, ts.grad_bm, &ta.st, &n_tiles);
    ta.H = H;
    ta.targets = targets;
    ta.T = T;
    ta.V = V;
    ta.d = (int32_t)d;
    ta.yt = yt;
    if (!vpce::run_target_logits(prob->dtype, ta, s)) return VP_ERR_HIP;
  }

  const std::vector<Chunk> chunks = strip_chunks(prob, plan);
  int64_t off[VP_MAX_SHARDS];
  int64_t acc = 0;
  for (int q = 0; q < prob->P; ++q) {
    off[q] = acc;
    acc += prob->shard_rows[q];
  }
  auto wchunk = [&](const Chunk& c) {
    return (const char*)W_shards[c.q] + (size_t)c.v0 * d * eb;
  };
  // Launch k runs the residual of strip k (into buffer k % 2) and the dH / dW
  // contractions of strip k-1 (from buffer (k-1) % 2).  Stream order gives every
  // dependency: strip k-1 was written by launch k-1; buffer k % 2 was last read
  // by launch k-1; dH rows and dW chunks are only updated by consecutive launches.
  const int64_t n = (int64_t)chunks.size();
  for (int64_t k = 0; k <= n; ++k) {
    vpce::GradArgs g;
    memset(&g, 0, sizeof(g));
    if (k < n) {
      const Chunk& c = chunks[k];
      g.W = wchunk(c);
      g.H = H;
      g.targets = targets;
      g.lse = lse;
      g.grad = grad_loss;
      g.strip = wsb + plan.off_g[k % 2];
      g.strip_t = wsb + plan.off_gt[k % 2];
      g.Tc = plan.Tc;
      g.Vc = plan.Vc;
      g.t0 = c.t0;
      g.gid0 = off[c.q] + c.v0;
      g.V = V;
      g.ignore_index = prob->ignore_index;
      g.yt = yt;
      g.M = (int32_t)c.M;
      g.N = (int32_t)c.N;
      g.d = (int32_t)d;
      g.n_vt = (int32_t)ceil_div(c.M, ts.grad_bm);
    }
    vpce::GemmArgs h, w;
    memset(&h, 0, sizeof(h));
    memset(&w, 0, sizeof(w));
    if (k >= 1) {
      const Chunk& c = chunks[k - 1];
      if (c.new_vchunk) {  // W^T of this vocabulary chunk, k-blocked [Vc/KB][d][KB], zero beyond M
        vpce::TransposeArgs tr;
        tr.in = wchunk(c);
        tr.ld_in = d;
        tr.out = Wt;
        tr.R = (int32_t)c.M;
        tr.C = (int32_t)d;
        tr.R_pad = (int32_t)round_up(c.M, KB);  // >= the K the dH launch reads
        if (!vpce::run_transpose(prob->dtype, tr, s)) return VP_ERR_HIP;
      }
      // dH[t0 : t0+N] (+)= G^T W_chunk = G^T . (W^T)^T
      h.A = wsb + plan.off_gt[(k - 1) % 2];
      h.lda = KB;
      h.kblka = plan.Tc * KB;
      h.B = Wt;
      h.ldb = KB;
      h.kblkb = d * KB;
      h.C = dH + c.t0 * d;
      h.ldc = d;
      h.M = (int32_t)c.N;
      h.N = (int32_t)d;
      h.K = (int32_t)round_up(c.M, ts.kalign);  // G^T and W^T are zero past M
      h.beta = c.first_vchunk ? 0 : 1;
      // dW_chunk (+)= G H[t0 : t0+N] = G . (H^T)^T
      w.A = wsb + plan.off_g[(k - 1) % 2];
      w.lda = KB;
      w.kblka = plan.Vc * KB;
      w.B = (const char*)Ht + (size_t)((c.t0 / KB) * d * KB) * eb;  // t0 is a multiple of Tc
      w.ldb = KB;
      w.kblkb = d * KB;
      w.C = dW_shards[c.q] + c.v0 * d;
      w.ldc = d;
      w.M = (int32_t)c.M;
      w.N = (int32_t)d;
      w.K = (int32_t)round_up(c.N, ts.kalign);  // G is zero past N
      w.beta = (c.t0 > 0 || accumulate) ? 1 : 0;
    }
    if (!vpce::run_bwd_stage(prob->dtype, h, w, g, s)) return VP_ERR_HIP;
  }
  return VP_OK;
}

vp_status vp_ce_check(const void* ws, void* stream, int64_t* bad_targets) {
  if (!ws) return VP_ERR_NULL;
  unsigned long long count = 0;
  hipStream_t s = (hipStream_t)stream;
  if (hipMemcpyAsync(&count, ws, sizeof(count), hipMemcpyDeviceToHost, s) != hipSuccess)
    return VP_ERR_HIP;
  if (hipStreamSynchronize(s) != hipSuccess) return VP_ERR_HIP;
  if (bad_targets) *bad_targets = (int64_t)count;
  return count ? VP_ERR_TARGET : VP_OK;
}

}  // extern "C"
