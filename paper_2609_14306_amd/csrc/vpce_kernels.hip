// HIP kernels for gfx950 (MI355X): fused vocabulary-projection softmax
// cross-entropy, forward with an online log-sum-exp fold and backward with
// logits recompute (arXiv 2609.14306, Sec. 3.2 and the appendix on Ring-DTP).
//
// One MFMA GEMM mainloop serves the four contractions of the path:
//   logits (forward and recompute)  C[v][t] = sum_k W[v][k] H[t][k]   (both K-major)
//   dH                              C[t][n] = sum_v G[v][t] W[v][n]   (both MN-major)
//   dW                              C[v][n] = sum_t G[v][t] H[t][n]   (A K-major, B MN-major)
// The residual strip G is stored vocabulary-row by token-column ([Vc][ldg]).
// Logits are computed transposed (vocabulary rows, token columns) so that in the
// MFMA accumulator layout every lane owns whole token columns: the online
// softmax state of a token lives in one lane's registers and needs no
// cross-lane traffic until the very end of a workgroup's vocabulary range.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "vpce_internal.h"

namespace vpce {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef short s16x4_t __attribute__((ext_vector_type(4)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef short __attribute__((address_space(3))) * lds_s16_ptr;

constexpr int kThreads = 256;  // 4 wavefronts of 64, arranged 2 x 2 over the tile
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

// ---------------------------------------------------------------------------
// Element policies.  BK: k elements staged per LDS pass (128 bytes per row);
// KSTEP: k consumed by one MFMA; VEC: elements per 16-byte global load.
struct Bf16 {
  using storage = uint16_t;
  using frag = bf16x8_t;
  static constexpr int BK = 64, KSTEP = 16, VEC = 8, PADK = 8, PADM = 16;
  __device__ static f32x16_t mma(frag a, frag b, f32x16_t c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
  }
  __device__ static storage from_f32(float x) {  // round to nearest even (NaN stays NaN)
    uint32_t u = __float_as_uint(x);
    u += 0x7FFFu + ((u >> 16) & 1u);
    return (storage)(u >> 16);
  }
};
struct F32 {
  using storage = float;
  using frag = float;
  static constexpr int BK = 32, KSTEP = 2, VEC = 4, PADK = 4, PADM = 4;
  __device__ static f32x16_t mma(frag a, frag b, f32x16_t c) {
    return __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, c, 0, 0, 0);
  }
  __device__ static storage from_f32(float x) { return x; }
};

// ---------------------------------------------------------------------------
// Global -> register -> LDS staging of one operand tile.  ROWS is the extent of
// the operand's non-contracted dimension in the tile.  A K-major operand holds
// element (r, k) at p[r * ld + k]; an MN-major one at p[k * ld + r].
// Rows at or beyond R are clamped (K-major) or zero (MN-major): they only feed
// accumulator rows/columns that are never stored.  k at or beyond K is zero,
// so ragged contractions add nothing.
template <class E, int ROWS, bool KMAJOR>
struct Stage {
  using S = typename E::storage;
  static constexpr int BK = E::BK, VEC = E::VEC;
  static constexpr int CHUNKS = ROWS * BK / VEC;
  static constexpr int PER_THREAD = CHUNKS / kThreads;
  static_assert(CHUNKS % kThreads == 0, "tile must split evenly over the workgroup");
  static constexpr int LD = KMAJOR ? (BK + E::PADK) : (ROWS + E::PADM);
  static constexpr int LDS_ELEMS = KMAJOR ? ROWS * LD : BK * LD;
  uint4 regs[PER_THREAD];

  __device__ __forceinline__ void load(const S* __restrict__ p, int64_t ld, int r0, int R, int k0,
                                       int K, int tid) {
#pragma unroll
    for (int i = 0; i < PER_THREAD; ++i) {
      const int c = tid + i * kThreads;
      if constexpr (KMAJOR) {
        const int r = c / (BK / VEC), kc = (c % (BK / VEC)) * VEC;
        const int rr = min(r0 + r, R - 1);
        const int kk = k0 + kc;
        regs[i] = (kk < K && rr >= 0) ? *(const uint4*)(p + (int64_t)rr * ld + kk)
                                      : make_uint4(0, 0, 0, 0);
      } else {
        const int kr = c / (ROWS / VEC), rc = (c % (ROWS / VEC)) * VEC;
        const int kk = k0 + kr, rr = r0 + rc;
        regs[i] = (kk < K && rr < R) ? *(const uint4*)(p + (int64_t)kk * ld + rr)
                                     : make_uint4(0, 0, 0, 0);
      }
    }
  }
  __device__ __forceinline__ void store(S* lds, int tid) const {
#pragma unroll
    for (int i = 0; i < PER_THREAD; ++i) {
      const int c = tid + i * kThreads;
      int off;
      if constexpr (KMAJOR) {
        off = (c / (BK / VEC)) * LD + (c % (BK / VEC)) * VEC;
      } else {
        off = (c / (ROWS / VEC)) * LD + (c % (ROWS / VEC)) * VEC;
      }
      *(uint4*)(lds + off) = regs[i];
    }
  }
};

// MFMA operand fragment of one 32-wide block (rows row0..row0+31 of the
// operand's non-contracted dimension) at k offset kbase of the staged tile.
// 32x32x16 bf16: lane l takes row l%32 and k = kbase + 8*(l/32) + 0..7.
// 32x32x2 f32:   lane l takes row l%32 and k = kbase + l/32.
template <class E, int LD, bool KMAJOR>
__device__ __forceinline__ typename E::frag read_frag(const typename E::storage* lds, int row0,
                                                      int kbase, int lane) {
  if constexpr (sizeof(typename E::storage) == 2) {
    if constexpr (KMAJOR) {
      return *(const bf16x8_t*)(lds + (row0 + (lane & 31)) * LD + kbase + 8 * (lane >> 5));
    } else {
      // LDS transpose read: within each 16-lane group, lane 4b+c points at k-row b,
      // columns 4c..4c+3; lane j of the group receives column j of the 4 k-rows.
      const int g = lane >> 4, i = lane & 15;
      const int krow = kbase + 8 * (g >> 1) + (i >> 2);
      const int col = row0 + 16 * (g & 1) + 4 * (i & 3);
      const typename E::storage* p0 = lds + krow * LD + col;
      s16x4_t lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((s16x4_t __attribute__((address_space(3)))*)(p0));
      s16x4_t hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
          (s16x4_t __attribute__((address_space(3)))*)(p0 + 4 * LD));
      typedef short s16x8_t __attribute__((ext_vector_type(8)));
      s16x8_t v = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
      return __builtin_bit_cast(bf16x8_t, v);
    }
  } else {
    if constexpr (KMAJOR) {
      return lds[(row0 + (lane & 31)) * LD + kbase + (lane >> 5)];
    } else {
      return lds[(kbase + (lane >> 5)) * LD + row0 + (lane & 31)];
    }
  }
}

// Accumulator layout of a 32x32 MFMA block: lane l, register r holds
// row 8*(r/4) + 4*(l/32) + r%4 and column l%32.
__device__ __forceinline__ int acc_row(int r, int lane) { return 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3); }

// Tile GEMM: acc += A[m0 : m0+BM, 0:K] * B[0:K, n0 : n0+BN] on a 2x2 grid of waves.
template <class E, int BM, int BN, bool AK, bool BKM>
struct Gemm {
  using S = typename E::storage;
  static constexpr int WM = BM / 2, WN = BN / 2, MB = WM / 32, NB = WN / 32;
  using SA = Stage<E, BM, AK>;
  using SB = Stage<E, BN, BKM>;
  static constexpr int LDS_ELEMS = SA::LDS_ELEMS + SB::LDS_ELEMS;

  __device__ __forceinline__ static void run(f32x16_t (&acc)[MB][NB], const S* __restrict__ A,
                                             int64_t lda, int m0, int M, const S* __restrict__ B,
                                             int64_t ldb, int n0, int N, int K, S* smem) {
    S* sA = smem;
    S* sB = smem + SA::LDS_ELEMS;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = (wave >> 1) * WM, wn = (wave & 1) * WN;
    SA la;
    SB lb;
    const int nk = (K + E::BK - 1) / E::BK;
    la.load(A, lda, m0, M, 0, K, tid);
    lb.load(B, ldb, n0, N, 0, K, tid);
    la.store(sA, tid);
    lb.store(sB, tid);
    __syncthreads();
    for (int kt = 0; kt < nk; ++kt) {
      const bool more = kt + 1 < nk;
      if (more) {
        la.load(A, lda, m0, M, (kt + 1) * E::BK, K, tid);
        lb.load(B, ldb, n0, N, (kt + 1) * E::BK, K, tid);
      }
#pragma unroll
      for (int kk = 0; kk < E::BK; kk += E::KSTEP) {
        typename E::frag a[MB], b[NB];
#pragma unroll
        for (int i = 0; i < MB; ++i) a[i] = read_frag<E, SA::LD, AK>(sA, wm + 32 * i, kk, lane);
#pragma unroll
        for (int j = 0; j < NB; ++j) b[j] = read_frag<E, SB::LD, BKM>(sB, wn + 32 * j, kk, lane);
#pragma unroll
        for (int i = 0; i < MB; ++i)
#pragma unroll
          for (int j = 0; j < NB; ++j) acc[i][j] = E::mma(a[i], b[j], acc[i][j]);
      }
      __syncthreads();
      if (more) {
        la.store(sA, tid);
        lb.store(sB, tid);
      }
      __syncthreads();
    }
  }
};

// ---------------------------------------------------------------------------
// Online-softmax state merge in the base-2 domain (m is a running maximum of
// y*log2(e), s = sum 2^(y*log2e - m)).  An empty state is (-inf, 0).
__device__ __forceinline__ void merge_state(float& m, float& s, float mo, float so) {
  const float M = fmaxf(m, mo);
  if (M == -INFINITY) return;
  s = s * __builtin_amdgcn_exp2f(m - M) + so * __builtin_amdgcn_exp2f(mo - M);
  m = M;
}

__global__ void ws_init_kernel(unsigned long long* counter) {
  if (threadIdx.x == 0 && blockIdx.x == 0) *counter = 0ull;
}

__global__ void fill_zero_kernel(float* p, int64_t n) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride) p[i] = 0.f;
}

// Forward: each workgroup owns BN tokens and one contiguous range of the
// vocabulary tiles in visiting order; it folds every logits tile into a
// per-lane online-softmax state, gathers the target logit from the one tile
// whose rows contain it, and writes its partial (m, s) per token.
template <class E, int BM, int BN>
__global__ void __launch_bounds__(kThreads) fwd_kernel(FwdArgs a) {
  using G = Gemm<E, BM, BN, true, true>;
  using S = typename E::storage;
  __shared__ __attribute__((aligned(16))) S smem[G::LDS_ELEMS];
  constexpr int MB = G::MB, NB = G::NB;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = (wave >> 1) * G::WM, wn = (wave & 1) * G::WN;
  const int tb = blockIdx.x % a.n_tok_blocks;
  const int split = blockIdx.x / a.n_tok_blocks;
  const int n0 = tb * BN;
  const int t_begin = (int)((int64_t)split * a.n_tiles / a.n_splits);
  const int t_end = (int)((int64_t)(split + 1) * a.n_tiles / a.n_splits);

  float m_run[NB], s_run[NB];
  int64_t tgt[NB];
#pragma unroll
  for (int j = 0; j < NB; ++j) {
    m_run[j] = -INFINITY;
    s_run[j] = 0.f;
    const int64_t n = n0 + wn + 32 * j + (lane & 31);
    tgt[j] = n < a.T ? a.targets[n] : -1;
  }

  int pos = 0;
  for (int ti = t_begin; ti < t_end; ++ti) {
    while (ti >= a.st.tile0[pos + 1]) ++pos;
    const int r0 = (ti - a.st.tile0[pos]) * BM;
    const int rows = min(BM, a.st.rows[pos] - r0);
    const int64_t gid0 = a.st.off[pos] + r0;
    const S* Wt = (const S*)a.st.w[pos] + (int64_t)r0 * a.d;

    f32x16_t acc[MB][NB];
#pragma unroll
    for (int i = 0; i < MB; ++i)
#pragma unroll
      for (int j = 0; j < NB; ++j) acc[i][j] = f32x16_t{};
    G::run(acc, Wt, a.d, 0, rows, (const S*)a.H, a.d, n0, (int)a.T, a.d, smem);

    const bool full = rows == BM;
#pragma unroll
    for (int j = 0; j < NB; ++j) {
      float tmax = -INFINITY;
#pragma unroll
      for (int i = 0; i < MB; ++i)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const float y2 = acc[i][j][r] * kLog2e;
          const bool ok = full || (wm + 32 * i + acc_row(r, lane) < rows);
          tmax = ok ? fmaxf(tmax, y2) : tmax;
        }
      const float scale = tmax > m_run[j] ? __builtin_amdgcn_exp2f(m_run[j] - tmax) : 1.f;
      m_run[j] = fmaxf(m_run[j], tmax);
      float sum = 0.f;
#pragma unroll
      for (int i = 0; i < MB; ++i)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const bool ok = full || (wm + 32 * i + acc_row(r, lane) < rows);
          const float e = __builtin_amdgcn_exp2f(__builtin_fmaf(acc[i][j][r], kLog2e, -m_run[j]));
          sum += ok ? e : 0.f;
        }
      s_run[j] = s_run[j] * scale + sum;

      // Target gather: exactly one tile in the whole vocabulary holds the target.
      const int64_t rel = tgt[j] - gid0;
      if (rel >= 0 && rel < rows) {
        const int relw = (int)rel - wm;
        if (relw >= 0 && relw < G::WM) {
          const int rib = relw & 31;
          if (((rib >> 2) & 1) == (lane >> 5)) {
            const int want_i = relw >> 5, want_r = (rib >> 3) * 4 + (rib & 3);
            float yv = 0.f;
#pragma unroll
            for (int i = 0; i < MB; ++i)
#pragma unroll
              for (int r = 0; r < 16; ++r) yv = (i == want_i && r == want_r) ? acc[i][j][r] : yv;
            a.y_tgt[n0 + wn + 32 * j + (lane & 31)] = yv;
          }
        }
      }
    }
  }

  // Merge the two lane halves that share a token column, then the two wave rows.
#pragma unroll
  for (int j = 0; j < NB; ++j) {
    const float mo = __shfl_xor(m_run[j], 32);
    const float so = __shfl_xor(s_run[j], 32);
    merge_state(m_run[j], s_run[j], mo, so);
  }
  __syncthreads();  // smem is free after the last tile
  float* red = (float*)smem;  // [2][BN]
  if ((wave >> 1) == 1 && lane < 32) {
#pragma unroll
    for (int j = 0; j < NB; ++j) {
      red[wn + 32 * j + lane] = m_run[j];
      red[BN + wn + 32 * j + lane] = s_run[j];
    }
  }
  __syncthreads();
  if ((wave >> 1) == 0 && lane < 32) {
#pragma unroll
    for (int j = 0; j < NB; ++j) {
      const int c = wn + 32 * j + lane;
      merge_state(m_run[j], s_run[j], red[c], red[BN + c]);
      const int64_t n = n0 + c;
      if (n < a.T) {
        a.m_part[(int64_t)split * a.T + n] = m_run[j];
        a.s_part[(int64_t)split * a.T + n] = s_run[j];
      }
    }
  }
}

// Folds the per-split partial states of each token in split order (the
// visiting order), then finalises lse = m + log z and loss = lse - y_target.
__global__ void __launch_bounds__(256) comb_kernel(CombArgs a) {
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= a.T) return;
  float m = -INFINITY, s = 0.f;
  for (int k = 0; k < a.n_splits; ++k)
    merge_state(m, s, a.m_part[(int64_t)k * a.T + t], a.s_part[(int64_t)k * a.T + t]);
  const float lse = (m + __builtin_amdgcn_logf(s)) * kLn2;
  const int64_t tg = a.targets[t];
  float loss;
  if (tg == a.ignore_index) {
    loss = 0.f;
  } else if (tg < 0 || tg >= a.V) {
    loss = __builtin_nanf("");
    atomicAdd(a.bad_counter, 1ull);
  } else {
    loss = lse - a.y_tgt[t];
  }
  a.lse[t] = lse;
  a.loss[t] = loss;
}

// Backward residual: recompute a logits tile of the (vocabulary chunk, token
// chunk) strip and store G = g (2^(y log2e - lse log2e) - onehot) into the strip.
template <class E, int BM, int BN>
__global__ void __launch_bounds__(kThreads) grad_kernel(GradArgs a) {
  using G = Gemm<E, BM, BN, true, true>;
  using S = typename E::storage;
  __shared__ __attribute__((aligned(16))) S smem[G::LDS_ELEMS];
  constexpr int MB = G::MB, NB = G::NB;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = (wave >> 1) * G::WM, wn = (wave & 1) * G::WN;
  const int vt = blockIdx.x % a.n_vt;
  const int tb = blockIdx.x / a.n_vt;
  const int m0 = vt * BM, n0 = tb * BN;

  f32x16_t acc[MB][NB];
#pragma unroll
  for (int i = 0; i < MB; ++i)
#pragma unroll
    for (int j = 0; j < NB; ++j) acc[i][j] = f32x16_t{};
  G::run(acc, (const S*)a.W, a.d, m0, a.M, (const S*)a.H + a.t0 * a.d, a.d, n0, a.N, a.d, smem);

  S* Gs = (S*)a.strip;
#pragma unroll
  for (int j = 0; j < NB; ++j) {
    const int nl = n0 + wn + 32 * j + (lane & 31);  // token column within the chunk
    float lse2 = 0.f, g = 0.f;
    int64_t tg = a.ignore_index;
    bool live = false, bad = false;
    if (nl < a.N) {
      const int64_t t = a.t0 + nl;
      tg = a.targets[t];
      if (tg != a.ignore_index) {
        bad = tg < 0 || tg >= a.V;
        live = true;
        lse2 = a.lse[t] * kLog2e;
        g = a.grad[t];
      }
    }
    const int64_t rel = tg - a.gid0;  // target row within the chunk (if any)
#pragma unroll
    for (int i = 0; i < MB; ++i)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int ml = m0 + wm + 32 * i + acc_row(r, lane);
        if (ml < a.M) {
          float v = 0.f;
          if (live) {
            const float p = __builtin_amdgcn_exp2f(__builtin_fmaf(acc[i][j][r], kLog2e, -lse2));
            v = g * (p - (rel == (int64_t)ml ? 1.f : 0.f));
            if (bad) v = __builtin_nanf("");
          }
          Gs[(int64_t)ml * a.ldg + nl] = E::from_f32(v);
        }
      }
  }
}

// Counts out-of-range targets of a token range (backward's copy of the check).
__global__ void count_bad_kernel(const int64_t* targets, int64_t T, int64_t V, int64_t ignore_index,
                                 unsigned long long* counter) {
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (t < T) {
    const int64_t tg = targets[t];
    if (tg != ignore_index && (tg < 0 || tg >= V)) atomicAdd(counter, 1ull);
  }
}

// Plain tile GEMM with a float32 output: C = (beta ? C : 0) + A * B.
template <class E, int BM, int BN, bool AK, bool BKM>
__global__ void __launch_bounds__(kThreads) gemm_kernel(GemmArgs a) {
  using G = Gemm<E, BM, BN, AK, BKM>;
  using S = typename E::storage;
  __shared__ __attribute__((aligned(16))) S smem[G::LDS_ELEMS];
  constexpr int MB = G::MB, NB = G::NB;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = (wave >> 1) * G::WM, wn = (wave & 1) * G::WN;
  const int nt = blockIdx.x % a.n_nt;
  const int mt = blockIdx.x / a.n_nt;
  const int m0 = mt * BM, n0 = nt * BN;

  f32x16_t acc[MB][NB];
#pragma unroll
  for (int i = 0; i < MB; ++i)
#pragma unroll
    for (int j = 0; j < NB; ++j) acc[i][j] = f32x16_t{};
  G::run(acc, (const S*)a.A, a.lda, m0, a.M, (const S*)a.B, a.ldb, n0, a.N, a.K, smem);

#pragma unroll
  for (int i = 0; i < MB; ++i)
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int m = m0 + wm + 32 * i + acc_row(r, lane);
      if (m >= a.M) continue;
      float* crow = a.C + (int64_t)m * a.ldc;
#pragma unroll
      for (int j = 0; j < NB; ++j) {
        const int n = n0 + wn + 32 * j + (lane & 31);
        if (n < a.N) crow[n] = a.beta ? crow[n] + acc[i][j][r] : acc[i][j][r];
      }
    }
}

// ---------------------------------------------------------------------------
// Launchers (host side).  Tile shapes are fixed per element type.
template <class E> struct Tiles;
template <> struct Tiles<Bf16> {
  static constexpr int FWD_BM = 128, FWD_BN = 128;
  static constexpr int GRAD_BM = 128, GRAD_BN = 128;
  static constexpr int MM_BM = 128, MM_BN = 128;
};
template <> struct Tiles<F32> {
  static constexpr int FWD_BM = 64, FWD_BN = 64;
  static constexpr int GRAD_BM = 64, GRAD_BN = 64;
  static constexpr int MM_BM = 64, MM_BN = 64;
};

static inline bool launched_ok() { return hipGetLastError() == hipSuccess; }

template <class E>
static bool launch_fwd(const FwdArgs& a, hipStream_t s) {
  constexpr int BM = Tiles<E>::FWD_BM, BN = Tiles<E>::FWD_BN;
  const unsigned grid = (unsigned)(a.n_tok_blocks * a.n_splits);
  hipLaunchKernelGGL((fwd_kernel<E, BM, BN>), dim3(grid), dim3(kThreads), 0, s, a);
  return launched_ok();
}
template <class E>
static bool launch_grad(const GradArgs& a, hipStream_t s) {
  constexpr int BM = Tiles<E>::GRAD_BM, BN = Tiles<E>::GRAD_BN;
  const unsigned grid = (unsigned)(a.n_vt * ((a.N + BN - 1) / BN));
  hipLaunchKernelGGL((grad_kernel<E, BM, BN>), dim3(grid), dim3(kThreads), 0, s, a);
  return launched_ok();
}
template <class E, bool AK, bool BKM>
static bool launch_gemm(GemmArgs a, hipStream_t s) {
  constexpr int BM = Tiles<E>::MM_BM, BN = Tiles<E>::MM_BN;
  a.n_nt = (a.N + BN - 1) / BN;
  const unsigned grid = (unsigned)(a.n_nt * ((a.M + BM - 1) / BM));
  hipLaunchKernelGGL((gemm_kernel<E, BM, BN, AK, BKM>), dim3(grid), dim3(kThreads), 0, s, a);
  return launched_ok();
}

}  // namespace vpce

// ---- entry points used by the host API (vpce_api.cpp) ----
namespace vpce {

TileShape tile_shape(int dtype) {
  TileShape t;
  if (dtype == 1) {
    t.fwd_bm = Tiles<Bf16>::FWD_BM; t.fwd_bn = Tiles<Bf16>::FWD_BN;
    t.grad_bm = Tiles<Bf16>::GRAD_BM; t.grad_bn = Tiles<Bf16>::GRAD_BN;
  } else {
    t.fwd_bm = Tiles<F32>::FWD_BM; t.fwd_bn = Tiles<F32>::FWD_BN;
    t.grad_bm = Tiles<F32>::GRAD_BM; t.grad_bn = Tiles<F32>::GRAD_BN;
  }
  return t;
}

bool run_ws_init(unsigned long long* counter, hipStream_t s) {
  hipLaunchKernelGGL(ws_init_kernel, dim3(1), dim3(64), 0, s, counter);
  return launched_ok();
}
bool run_fill_zero(float* p, int64_t n, hipStream_t s) {
  if (n <= 0) return true;
  const int64_t blocks = std::min<int64_t>((n + 255) / 256, 4096);
  hipLaunchKernelGGL(fill_zero_kernel, dim3((unsigned)blocks), dim3(256), 0, s, p, n);
  return launched_ok();
}
bool run_fwd(int dtype, const FwdArgs& a, hipStream_t s) {
  return dtype == 1 ? launch_fwd<Bf16>(a, s) : launch_fwd<F32>(a, s);
}
bool run_comb(const CombArgs& a, hipStream_t s) {
  const unsigned grid = (unsigned)((a.T + 255) / 256);
  hipLaunchKernelGGL(comb_kernel, dim3(grid), dim3(256), 0, s, a);
  return launched_ok();
}
bool run_grad(int dtype, const GradArgs& a, hipStream_t s) {
  return dtype == 1 ? launch_grad<Bf16>(a, s) : launch_grad<F32>(a, s);
}
bool run_count_bad(const int64_t* targets, int64_t T, int64_t V, int64_t ignore_index,
                   unsigned long long* counter, hipStream_t s) {
  if (T <= 0) return true;
  hipLaunchKernelGGL(count_bad_kernel, dim3((unsigned)((T + 255) / 256)), dim3(256), 0, s, targets,
                     T, V, ignore_index, counter);
  return launched_ok();
}
bool run_dH(int dtype, const GemmArgs& a, hipStream_t s) {
  // C[t][n] = sum_v G[v][t] W[v][n]: A (strip) and B (W) both MN-major.
  return dtype == 1 ? launch_gemm<Bf16, false, false>(a, s) : launch_gemm<F32, false, false>(a, s);
}
bool run_dW(int dtype, const GemmArgs& a, hipStream_t s) {
  // C[v][n] = sum_t G[v][t] H[t][n]: A (strip) K-major, B (H) MN-major.
  return dtype == 1 ? launch_gemm<Bf16, true, false>(a, s) : launch_gemm<F32, true, false>(a, s);
}

}  // namespace vpce
