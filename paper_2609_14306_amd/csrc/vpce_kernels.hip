// HIP kernels for gfx950 (MI355X): fused vocabulary-projection softmax
// cross-entropy, forward with an online log-sum-exp fold and backward with
// logits recompute (arXiv 2609.14306, Sec. 3.2 and the appendix on Ring-DTP).
//
// One MFMA GEMM mainloop, C[m][n] = sum_k A[m][k] B[n][k] with both operands
// k-contiguous, serves the four contractions of the path:
//   logits (forward and recompute)  C[v][t] = sum_k W[v][k]   H[t][k]
//   dH                              C[t][n] = sum_v G^T[t][v] W^T[n][v]
//   dW                              C[v][n] = sum_t G[v][t]   H^T[n][t]
// The backward stores the softmax residual of a (vocabulary chunk, token
// chunk) strip in both layouts (G and G^T) and uses transposed copies of H
// (once per call) and of each vocabulary chunk of W, so that every operand is
// staged k-contiguous and every MFMA fragment is one 16-byte LDS read (an
// operand read through gfx950's LDS transpose read, two 8-byte reads per
// fragment, costs the mainloop about 4% of its rate, more than the second
// layout and the transposes cost).
//
// Logits are computed transposed (vocabulary rows, token columns) so that in the
// MFMA accumulator layout every lane owns whole token columns: the online
// softmax state of a token lives in one lane's registers and needs no
// cross-lane traffic until the very end of a workgroup's vocabulary range.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <mutex>
#include <type_traits>

#include "vpce_internal.h"

namespace vpce {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

// ---------------------------------------------------------------------------
// Element policies.  BK: k elements staged per LDS pass (128 bytes per row);
// KSTEP: k consumed by one MFMA; VEC: elements per 16 bytes.
// KB: elements of one 128-byte k-block of the k-blocked backward workspaces (and of
// one row of a direct-to-LDS slice).  frag16 / mma16: one 16-byte operand fragment
// per lane (8 bfloat16 or 4 float32 k values) and the MFMA work it feeds.
struct Bf16 {
  using storage = uint16_t;
  using frag = bf16x8_t;
  using frag16 = bf16x8_t;
  static constexpr int BK = 64, KSTEP = 16, VEC = 8, PADK = 8, KB = 64;
  __device__ static f32x16_t mma(frag a, frag b, f32x16_t c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
  }
  __device__ static f32x16_t mma16(frag16 a, frag16 b, f32x16_t c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
  }
  // Two float32 values rounded to nearest even, packed low then high (one
  // v_cvt_pk_bf16_f32).
  __device__ static uint32_t pack2(float lo, float hi) {
    typedef float f32x2_t __attribute__((ext_vector_type(2)));
    typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
    const f32x2_t v = {lo, hi};
    return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2_t));
  }
};
typedef float f32x4_t __attribute__((ext_vector_type(4)));
struct F32 {
  using storage = float;
  using frag = float;
  using frag16 = f32x4_t;
  static constexpr int BK = 32, KSTEP = 2, VEC = 4, PADK = 4, KB = 32;
  __device__ static f32x16_t mma(frag a, frag b, f32x16_t c) {
    return __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, c, 0, 0, 0);
  }
  // Lane half h holds k = 4h .. 4h + 3 of an 8-wide k group in both operands; MFMA q
  // takes element q, i.e. k = q (lanes 0-31) and 4 + q (lanes 32-63): the four MFMAs
  // together cover the group (the contraction order within it is a permutation).
  __device__ static f32x16_t mma16(frag16 a, frag16 b, f32x16_t c) {
    c = __builtin_amdgcn_mfma_f32_32x32x2f32(a[0], b[0], c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_32x32x2f32(a[1], b[1], c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_32x32x2f32(a[2], b[2], c, 0, 0, 0);
    return __builtin_amdgcn_mfma_f32_32x32x2f32(a[3], b[3], c, 0, 0, 0);
  }
};

// ---------------------------------------------------------------------------
// Global -> register -> LDS staging of one k-contiguous operand tile of ROWS x
// BK (element (r, k) at p[r * ld + k]), written to LDS as [ROWS][BK + PADK].
// Rows at or beyond R are clamped to R-1 (they only feed accumulator rows or
// columns that are never stored); k at or beyond K reads as zero, so ragged
// contractions add nothing.  K is checked per 16-byte chunk: an operand whose
// K is not a multiple of VEC must hold finite values up to the next multiple.
template <class E, int ROWS, int NT>
struct Stage {
  using S = typename E::storage;
  static constexpr int BK = E::BK, VEC = E::VEC;
  static constexpr int LD = BK + E::PADK;
  static constexpr int LDS_ELEMS = ROWS * LD;
  static constexpr int UNITS = ROWS * BK / VEC;
  static constexpr int PER = (UNITS + NT - 1) / NT;
  uint4 regs[PER];

  __device__ __forceinline__ void load(const S* __restrict__ p, int64_t ld, int r0, int R, int k0,
                                       int K, int tid) {
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int u = tid + i * NT;
      const int r = u / (BK / VEC), kc = (u % (BK / VEC)) * VEC;
      const int rr = min(r0 + r, R - 1);
      const int kk = k0 + kc;
      regs[i] = (u < UNITS && kk < K && rr >= 0) ? *(const uint4*)(p + (int64_t)rr * ld + kk)
                                                 : make_uint4(0, 0, 0, 0);
    }
  }
  __device__ __forceinline__ void store(S* lds, int tid) const {
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int u = tid + i * NT;
      if (u < UNITS) *(uint4*)(lds + (u / (BK / VEC)) * LD + (u % (BK / VEC)) * VEC) = regs[i];
    }
  }
};

// MFMA operand fragment of one 32-wide block (rows row0..row0+31 of the
// operand's non-contracted dimension) at k offset kbase of the staged tile.
// 32x32x16 bf16: lane l takes row l%32 and k = kbase + 8*(l/32) + 0..7.
// 32x32x2 f32:   lane l takes row l%32 and k = kbase + l/32.
template <class E, int LD>
__device__ __forceinline__ typename E::frag read_frag(const typename E::storage* lds, int row0,
                                                      int kbase, int lane) {
  if constexpr (sizeof(typename E::storage) == 2) {
    return *(const bf16x8_t*)(lds + (row0 + (lane & 31)) * LD + kbase + 8 * (lane >> 5));
  } else {
    return lds[(row0 + (lane & 31)) * LD + kbase + (lane >> 5)];
  }
}

// Accumulator layout of a 32x32 MFMA block: lane l, register r holds
// row 8*(r/4) + 4*(l/32) + r%4 and column l%32.
__device__ __forceinline__ int acc_row(int r, int lane) { return 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3); }

// Tile GEMM: acc += A[m0 : m0+BM, 0:K] * B[n0 : n0+BN, 0:K]^T on a WGM x WGN grid of
// wavefronts.  Two LDS buffers: while the waves multiply out of one, the next
// k-slice (already fetched into registers one slice ahead) is written into the
// other, so each k-slice costs a single workgroup barrier.
template <class E, int BM_, int BN_, int WGM_, int WGN_>
struct Gemm {
  using S = typename E::storage;
  static constexpr int BM = BM_, BN = BN_, WGM = WGM_, WGN = WGN_;
  static constexpr int NT = 64 * WGM * WGN;
  static constexpr int OCC = 1;  // workgroups per CU the register budget is sized for
  static constexpr int KDIV = 1;  // any K (ragged k-slices are zero-filled)
  static constexpr int WM = BM / WGM, WN = BN / WGN, MB = WM / 32, NB = WN / 32;
  static_assert(WM % 32 == 0 && WN % 32 == 0, "wave tile must be whole 32x32 blocks");
  using SA = Stage<E, BM, NT>;
  using SB = Stage<E, BN, NT>;
  static constexpr int BUF_ELEMS = SA::LDS_ELEMS + SB::LDS_ELEMS;
  static constexpr int LDS_ELEMS = 2 * BUF_ELEMS;

  __device__ __forceinline__ static int wave_m(int wave) { return (wave / WGN) * WM; }
  __device__ __forceinline__ static int wave_n(int wave) { return (wave % WGN) * WN; }

  // Row-major operands only (the k-block strides are for the direct-load tile).
  // RAGGED is accepted for the interface of GemmDma and changes nothing here.
  template <bool RAGGED = false>
  __device__ __forceinline__ static void run(f32x16_t (&acc)[MB][NB], const S* __restrict__ A,
                                             int64_t lda, int m0, int M, const S* __restrict__ B,
                                             int64_t ldb, int n0, int N, int K, S* smem,
                                             int64_t = 64, int64_t = 64) {
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave_m(wave), wn = wave_n(wave);
    SA la;
    SB lb;
    const int nk = (K + E::BK - 1) / E::BK;
    la.load(A, lda, m0, M, 0, K, tid);
    lb.load(B, ldb, n0, N, 0, K, tid);
    la.store(smem, tid);
    lb.store(smem + SA::LDS_ELEMS, tid);
    __syncthreads();
    for (int kt = 0; kt < nk; ++kt) {
      const bool more = kt + 1 < nk;
      if (more) {
        la.load(A, lda, m0, M, (kt + 1) * E::BK, K, tid);
        lb.load(B, ldb, n0, N, (kt + 1) * E::BK, K, tid);
      }
      const S* sA = smem + (kt & 1) * BUF_ELEMS;
      const S* sB = sA + SA::LDS_ELEMS;
      // Fragments of sub-step kk+1 are read while the MFMAs of sub-step kk run.
      constexpr int NKK = E::BK / E::KSTEP;
      typename E::frag a[2][MB], b[2][NB];
#pragma unroll
      for (int i = 0; i < MB; ++i) a[0][i] = read_frag<E, SA::LD>(sA, wm + 32 * i, 0, lane);
#pragma unroll
      for (int j = 0; j < NB; ++j) b[0][j] = read_frag<E, SB::LD>(sB, wn + 32 * j, 0, lane);
#pragma unroll
      for (int q = 0; q < NKK; ++q) {
        const int cur = q & 1;
        if (q + 1 < NKK) {
#pragma unroll
          for (int i = 0; i < MB; ++i)
            a[cur ^ 1][i] = read_frag<E, SA::LD>(sA, wm + 32 * i, (q + 1) * E::KSTEP, lane);
#pragma unroll
          for (int j = 0; j < NB; ++j)
            b[cur ^ 1][j] = read_frag<E, SB::LD>(sB, wn + 32 * j, (q + 1) * E::KSTEP, lane);
        }
#pragma unroll
        for (int i = 0; i < MB; ++i)
#pragma unroll
          for (int j = 0; j < NB; ++j) acc[i][j] = E::mma(a[cur][i], b[cur][j], acc[i][j]);
      }
      if (more) {
        S* nA = smem + ((kt + 1) & 1) * BUF_ELEMS;
        la.store(nA, tid);
        lb.store(nA + SA::LDS_ELEMS, tid);
      }
      __syncthreads();
    }
  }
};

// ---------------------------------------------------------------------------
// Tile GEMM fed by direct global -> LDS loads (global_load_lds_dwordx4, 16 bytes
// per lane straight into LDS, no staging registers) through a ring of two
// k-slices of 128-byte rows: 64 bfloat16 or 32 float32 k values per row.  A
// 16-byte fragment feeds one 32x32x16 bf16 MFMA or four 32x32x2 f32 MFMAs (see
// the element policies); everything else is the same for both types.  Requires K
// to be a multiple of the slice depth and both operands to hold finite values up
// to that K (the backward's buffers are zero-padded).
//
// LDS slice layout: the A rows then the B rows, 128 bytes (eight 16-byte
// chunks) per row, chunk c of row r stored in slot c ^ ((r >> 1) & 7): the 16
// lanes of one LDS read phase (16 consecutive rows, same chunk) hit 16 distinct
// 4-bank groups, and each load instruction writes 1 KiB contiguously (8 rows).
//
// Schedule of one wave (slice kt lives in ring slot kt & 1; sub-step kk covers
// k = 16 kk .. 16 kk + 15 of the slice):
//   sub-steps 0..2: issue the MFMAs of sub-step kk, each followed by one LDS read
//                   of a fragment of sub-step kk+1 into the spare register set;
//   sub-step 3:     wait for this wave's loads of slice kt+1, barrier, then the
//                   MFMAs of sub-step 3 interleaved with the reads of slice kt+1
//                   sub-step 0.
// The loads of slice kt+2 go out one per two MFMAs, half during sub-step 3 of
// slice kt (into slot kt & 1: every wave finished reading slice kt before the
// barrier) and half during sub-step 0 of slice kt+1.  The MFMAs never wait on an
// LDS read issued in the same sub-step, the only barrier of a slice sits where
// every wave holds a sub-step of fragments in registers, each slice's loads have
// three or four sub-steps of MFMAs to land, and no burst of memory instructions
// ever stands in front of a wave's next MFMA.
// The loads are issued from inline assembly with a scalar base (the tile's
// first row at the slice's k offset) and a 32-bit per-lane byte offset, so that
// the compiler neither drains the loads before each LDS read (it cannot tell
// which ring slot a read touches) nor keeps 64-bit addresses per load.
// Completion is tracked by hand with vmcnt: loads return in issue order and the
// only loads a wave has in flight are its slice loads.
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  // s_waitcnt simm16 on gfx9: vmcnt[3:0] | expcnt[6:4] | lgkmcnt[11:8] | vmcnt[5:4] << 14
  __builtin_amdgcn_s_waitcnt((N & 0xF) | (0x7 << 4) | (0xF << 8) | ((N >> 4) << 14));
}
__device__ __forceinline__ void wait_lgkmcnt0() { __builtin_amdgcn_s_waitcnt(0xC07F); }

// One direct-to-LDS load from a scalar base.  The hazards the compiler's hazard
// recognizer cannot see inside inline assembly are covered here: five wait states
// before the load in case a VALU instruction (v_readlane of a spilled value, a
// carry-out) wrote the base SGPRs just before it, and one after the M0 write,
// which an LDS DMA reads.
__device__ __forceinline__ void lds_dma16x1(const void* sbase, uint32_t o0, uint32_t l0) {
  uint32_t m0v = l0;
  asm volatile("s_nop 4\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %1, %2"
               : "+{m0}"(m0v)
               : "v"(o0), "s"(sbase)
               : "memory");
}

template <int BM_, int BN_, int WGM_, int WGN_, int BK_ = 64, int STAGES_ = 2, class E = Bf16>
struct GemmDma {
  using S = typename E::storage;
  using F16 = typename E::frag16;
  static constexpr int BM = BM_, BN = BN_, WGM = WGM_, WGN = WGN_;
  static constexpr int NT = 64 * WGM * WGN, NWAVES = WGM * WGN;
  // One workgroup per CU (the ring takes 128 to 160 KiB of LDS): 512 threads run
  // two wavefronts per SIMD with 256 registers each.
  static constexpr int OCC = 1;
  static constexpr int WM = BM / WGM, WN = BN / WGN, MB = WM / 32, NB = WN / 32;
  static_assert(WM % 32 == 0 && WN % 32 == 0, "wave tile must be whole 32x32 blocks");
  // BK_ sizes a slice row in bfloat16 units: 64 (128-byte rows) or 32 (64-byte rows)
  static constexpr int STAGES = STAGES_;
  static constexpr int ROW_BYTES = BK_ * 2;
  static constexpr int BK = ROW_BYTES / (int)sizeof(S);  // k values per slice
  static_assert((BK_ == 32 || BK_ == 64) && STAGES >= 2, "slice depth and ring slots");
  static_assert(E::KB % BK == 0, "slices never straddle a k-block of the layout");
  static constexpr int KDIV = BK;                 // K must be a multiple of the slice depth
  static constexpr int NKK = ROW_BYTES / 32;      // sub-steps per slice (two 16-byte chunks each)
  static_assert(NKK % 2 == 0, "register sets alternate per sub-step across slices");
  static constexpr int CPR = ROW_BYTES / 16;      // 16-byte chunks per row
  static constexpr int RPW = 256 / ROW_BYTES;     // rows per 64-bank (256-byte) window
  static constexpr int RPI = 1024 / ROW_BYTES;    // rows per 1 KiB load instruction
  static constexpr int SLICE_BYTES = (BM + BN) * ROW_BYTES;
  static constexpr int A_LOADS = BM / RPI / NWAVES;  // load instructions per wave and slice
  static constexpr int B_LOADS = BN / RPI / NWAVES;
  static_assert(BM % (RPI * NWAVES) == 0 && BN % (RPI * NWAVES) == 0, "whole load groups per wave");
  static constexpr int NLOADS = A_LOADS + B_LOADS;  // per wave and slice
  // the loads of a slice go out in two halves, the larger first
  static constexpr int HALF0 = (NLOADS + 1) / 2, HALF1 = NLOADS - HALF0;
  static constexpr int NM = MB * NB, NR = MB + NB;   // MFMAs and fragment reads per sub-step
  static_assert(NR <= NM && HALF0 <= (NM + 1) / 2, "interleave slots");
  static constexpr int LDS_ELEMS = STAGES * SLICE_BYTES / (int)sizeof(S);
  static_assert(STAGES * SLICE_BYTES <= 160 * 1024, "LDS");

  // Chunk c of slice row r lives in slot c ^ key(r): within one 256-byte window
  // the rows sit at distinct offsets, and key(r) differs for the CPR rows that
  // share a window offset, so a read phase of 16 consecutive rows at one chunk
  // touches 16 distinct 4-bank groups.
  __device__ __forceinline__ static int key(int r) { return (r / RPW) % CPR; }

  __device__ __forceinline__ static int wave_m(int wave) { return (wave / WGN) * WM; }
  __device__ __forceinline__ static int wave_n(int wave) { return (wave % WGN) * WN; }

  __device__ __forceinline__ static uint32_t slot_bytes(int kt) {
    return (uint32_t)((kt % STAGES) * SLICE_BYTES);
  }

  // Load instruction q of a wave covers the RPI slice rows starting at
  // (wave + q * NWAVES) * RPI; A rows come first.  Rows at or beyond M (N) are
  // clamped to the last row: they only feed accumulator rows (columns) that are
  // never stored.
  struct Loads {
    const char* baseA;  // byte address of the tile's first A row (k = 0)
    const char* baseB;
    int64_t kblkA, kblkB;  // elements between consecutive k-blocks (E::KB wide)
    uint32_t offA[A_LOADS], offB[B_LOADS];  // per-lane byte offsets from the bases
  };

  __device__ __forceinline__ static void plan(Loads& L, const S* __restrict__ A, int64_t lda,
                                              int m0, int M, const S* __restrict__ B, int64_t ldb,
                                              int n0, int N, int wave, int lane) {
    const int ma = min(m0, M - 1), nb = min(n0, N - 1);
    L.baseA = (const char*)(A + (int64_t)ma * lda);
    L.baseB = (const char*)(B + (int64_t)nb * ldb);
    const int row_in = lane / CPR;
#pragma unroll
    for (int q = 0; q < A_LOADS; ++q) {
      const int r = (wave + q * NWAVES) * RPI + row_in;
      const int c = (lane % CPR) ^ key(r);
      L.offA[q] = (uint32_t)((min(m0 + r, M - 1) - ma) * lda * (int64_t)sizeof(S)) + 16u * c;
    }
#pragma unroll
    for (int q = 0; q < B_LOADS; ++q) {
      const int r = (wave + (A_LOADS + q) * NWAVES) * RPI + row_in;  // >= BM
      const int c = (lane % CPR) ^ key(r);
      L.offB[q] = (uint32_t)((min(n0 + r - BM, N - 1) - nb) * ldb * (int64_t)sizeof(S)) + 16u * c;
    }
  }

  // Load q (operand A's loads, then B's) of slice kt, into ring slot kt % STAGES:
  // it fills the 1 KiB at (wave + q * NWAVES) KiB of the slot.
  __device__ __forceinline__ static void issue_one(const Loads& L, int kt, int q, uint32_t lds0,
                                                   int wave) {
    constexpr int KB = E::KB;
    const int64_t k0 = (int64_t)kt * BK;
    const uint32_t l = lds0 + slot_bytes(kt) + (uint32_t)(wave * 1024) + q * NWAVES * 1024;
    if (q < A_LOADS)
      lds_dma16x1(L.baseA + ((k0 / KB) * L.kblkA + (k0 % KB)) * (int64_t)sizeof(S), L.offA[q], l);
    else
      lds_dma16x1(L.baseB + ((k0 / KB) * L.kblkB + (k0 % KB)) * (int64_t)sizeof(S), L.offB[q - A_LOADS], l);
  }

  // Fragment idx (the MB A blocks, then the NB B blocks) of sub-step kk at slot
  // byte address `slot`: lane l takes row l % 32 of the block and the 16 bytes of
  // chunk 2 kk + l / 32 (bf16: k = 16 kk + 8 (l / 32) + 0..7).
  __device__ __forceinline__ static F16 read_one(const char* slot, int wm, int wn, int kk, int lane,
                                                 int idx) {
    const int chunk = 2 * kk + (lane >> 5);
    const int row = idx < MB ? wm + 32 * idx + (lane & 31) : BM + wn + 32 * (idx - MB) + (lane & 31);
    return *(const F16*)(slot + row * ROW_BYTES + ((chunk ^ key(row)) << 4));
  }

  // Wait until at most n slices' loads (n in [0, STAGES - 1]) of this wave are in
  // flight; loads return in issue order.
  __device__ __forceinline__ static void wait_slices(int n) {
    if constexpr (STAGES == 2) {
      if (n <= 0) wait_vmcnt<0>(); else wait_vmcnt<NLOADS>();
    } else {
      static_assert(STAGES <= 5, "wait_slices covers up to five slots");
      switch (n) {
        case 0: wait_vmcnt<0>(); break;
        case 1: wait_vmcnt<NLOADS>(); break;
        case 2: wait_vmcnt<2 * NLOADS>(); break;
        case 3: wait_vmcnt<3 * NLOADS>(); break;
        default: wait_vmcnt<4 * NLOADS>(); break;
      }
    }
  }

  // acc += A[m0 : m0+BM, 0:K] B[n0 : n0+BN, 0:K]^T; requires m0 < M and n0 < N.
  // Element (r, k) of A is at A[(k / KB) kblka + r lda + k % KB] with KB = E::KB
  // (row-major: kblka = KB; k-blocked: lda = KB, kblka = rows * KB), likewise for B.
  // RAGGED: the tile reaches past row M of A; each wave skips the MFMAs (and the
  // fragment reads) of its 32-row blocks of A that lie wholly at or past M, whose
  // accumulators stay zero and are never stored.
  // LDS is free again for the caller when run() returns.
  template <bool RAGGED = false>
  __device__ __forceinline__ static void run(f32x16_t (&acc)[MB][NB], const S* __restrict__ A,
                                             int64_t lda, int m0, int M, const S* __restrict__ B,
                                             int64_t ldb, int n0, int N, int K, S* smem,
                                             int64_t kblka = E::KB, int64_t kblkb = E::KB) {
    // The wave index is made scalar so that every branch on it is a scalar branch.
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wm = wave_m(wave), wn = wave_n(wave);
    const int nk = K / BK;
    if (nk <= 0) return;
    // row blocks of A with live rows (wave-uniform); MB unless RAGGED
    const int mb_live = RAGGED ? max(0, min(MB, (M - m0 - wm + 31) / 32)) : MB;
    const uint32_t lds0 = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) S*)smem;
    Loads L;
    plan(L, A, lda, m0, M, B, ldb, n0, N, wave, lane);
    L.kblkA = kblka;
    L.kblkB = kblkb;
    // prologue: the first min(STAGES, nk) slices, whole; wait for slice 0
    const int pro = min(STAGES, nk);
    for (int kt = 0; kt < pro; ++kt)
#pragma unroll
      for (int q = 0; q < NLOADS; ++q) issue_one(L, kt, q, lds0, wave);
    wait_slices(pro - 1);
    __builtin_amdgcn_s_barrier();
    const char* ring = (const char*)smem;
    // A fragments are single-buffered: each is re-read for the next sub-step right
    // after its last MFMA of this one.  B fragments are double-buffered and read
    // during the first MFMAs of the sub-step.  The MFMAs go in snake order (row
    // block i takes its column blocks forwards for even i, backwards for odd i), so
    // that consecutive MFMAs share an operand.
    F16 a[MB], b[2][NB];
#pragma unroll
    for (int idx = 0; idx < NR; ++idx) {
      const F16 f = read_one(ring, wm, wn, 0, lane, idx);
      if (idx < MB)
        a[idx] = f;
      else
        b[0][idx - MB] = f;
    }
    for (int kt = 0; kt < nk; ++kt) {
#pragma unroll
      for (int kk = 0; kk < NKK; ++kk) {
        const int cur = kk & 1;
        // where the fragments of the next sub-step come from
        const char* src;
        int skk;
        if (kk + 1 < NKK) {
          src = ring + slot_bytes(kt);
          skk = kk + 1;
        } else {
          // Slice kt+1 must have landed; slices kt+2 .. kt+STAGES-1 may still be
          // in flight.  Taken on the last slice too (one spare barrier, fragments
          // read from an idle slot and never used): no branch around the LDS
          // reads, so the compiler's count of reads in flight stays exact.
          wait_slices(min(STAGES - 2, nk - 2 - kt));
          wait_lgkmcnt0();  // this wave's reads of slice kt
          __builtin_amdgcn_s_barrier();
          src = ring + slot_bytes(kt + 1);
          skk = 0;
        }
        // The loads of slice kt+STAGES go out in two halves: the first during the
        // last sub-step of slice kt (after the barrier: every wave has finished
        // reading slice kt, whose slot they refill), the second during the first
        // sub-step of slice kt+1 (the prologue issued the first STAGES slices).
        const int dq0 = kk == NKK - 1 ? 0 : HALF0;
        const int dn = kk == NKK - 1 ? HALF0 : HALF1;
        const int dslice = kk == NKK - 1 ? kt + STAGES : kt + STAGES - 1;
        const bool dvalid = (kk == NKK - 1 || (kk == 0 && kt >= 1)) && dslice < nk;
        __builtin_amdgcn_sched_barrier(0);
        // One MFMA, then the fragment reads it frees for the next sub-step, then
        // (every other MFMA) one load: the wave never holds a burst of memory
        // instructions in front of its next MFMA.
#pragma unroll
        for (int idx = 0; idx < NM; ++idx) {
          const int i = idx / NB, jj = idx % NB, j = (i & 1) ? NB - 1 - jj : jj;
          const bool live = !RAGGED || i < mb_live;
          if (live) acc[i][j] = E::mma16(a[i], b[cur][j], acc[i][j]);
          __builtin_amdgcn_sched_barrier(0);
          if (idx < NB) b[cur ^ 1][idx] = read_one(src, wm, wn, skk, lane, MB + idx);
          if (jj == NB - 1 && live) a[i] = read_one(src, wm, wn, skk, lane, i);
          if ((idx & 1) == 0 && idx / 2 < dn && (kk == NKK - 1 || kk == 0) && dvalid)
            issue_one(L, dslice, dq0 + idx / 2, lds0, wave);
          __builtin_amdgcn_sched_barrier(0);
        }
      }
    }
    // no wave may still be reading the ring, nor a load writing it, when the caller
    // reuses LDS
    wait_vmcnt<0>();
    wait_lgkmcnt0();
    __builtin_amdgcn_s_barrier();
  }
};

// ---------------------------------------------------------------------------
// Workgroup -> tile mapping.  Workgroups are dispatched to the 8 XCDs round
// robin (workgroup i on XCD i % 8) and each XCD has its own L2, so consecutive
// logical tile ids are handed to the workgroups of one XCD: the tiles an XCD
// runs at the same time then share operand panels in its L2.
__device__ __forceinline__ int xcd_logical(int bid, int n) {
  constexpr int X = 8;
  const int q = n / X, r = n % X;
  const int xcd = bid % X, local = bid / X;
  return xcd < r ? xcd * (q + 1) + local : r * (q + 1) + (xcd - r) * q + local;
}

// Logical id -> (mt, nt) in column-major groups of GM tile rows, so that a run
// of consecutive ids covers a GM x (run/GM) block of output tiles.
__device__ __forceinline__ void grouped_tile(int logical, int n_m, int n_n, int GM, int& mt,
                                             int& nt) {
  const int per_group = GM * n_n;
  const int group = logical / per_group;
  const int first = group * GM;
  const int gm = min(n_m - first, GM);
  const int in = logical - group * per_group;
  mt = first + in % gm;
  nt = in / gm;
}

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
template <class E, class G>
__global__ void __launch_bounds__(G::NT, G::OCC) fwd_kernel(FwdArgs a) {
  using S = typename E::storage;
  constexpr int BM = G::BM, BN = G::BN, MB = G::MB, NB = G::NB;
  __shared__ __attribute__((aligned(16))) S smem[G::LDS_ELEMS];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = G::wave_m(wave), wn = G::wave_n(wave);
  // split fastest: the workgroups an XCD runs together share token blocks (H panels)
  // across splits and vocabulary tiles (W panels) across token blocks.
  const int logical = xcd_logical(blockIdx.x, gridDim.x);
  const int tb = logical / a.n_splits;
  const int split = logical % a.n_splits;
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

    // Tiles past the end of a shard mask their padded rows; full tiles (all but the
    // last of each shard) take the select-free loops.  Register r of row block i
    // holds tile row wm + 32 i + acc_row(r, lane) = wm + 4 (lane / 32) + (a constant),
    // so the mask compares that constant with one per-lane limit.
    const bool full = rows == BM;
    const int lim = rows - wm - 4 * (lane >> 5);
#pragma unroll
    for (int j = 0; j < NB; ++j) {
      // The maximum is taken on the raw logits and scaled once: scaling by a positive
      // constant is monotone under rounding, so this equals the maximum of the scaled
      // values.
      float tmax = -INFINITY;
      if (full) {
#pragma unroll
        for (int i = 0; i < MB; ++i)
#pragma unroll
          for (int r = 0; r < 16; ++r) tmax = fmaxf(tmax, acc[i][j][r]);
      } else {
#pragma unroll
        for (int i = 0; i < MB; ++i)
#pragma unroll
          for (int r = 0; r < 16; ++r)
            if (32 * i + 8 * (r >> 2) + (r & 3) < lim) tmax = fmaxf(tmax, acc[i][j][r]);
      }
      tmax *= kLog2e;
      const float scale = tmax > m_run[j] ? __builtin_amdgcn_exp2f(m_run[j] - tmax) : 1.f;
      m_run[j] = fmaxf(m_run[j], tmax);
      float sum = 0.f;
      if (full) {
#pragma unroll
        for (int i = 0; i < MB; ++i)
#pragma unroll
          for (int r = 0; r < 16; ++r)
            sum += __builtin_amdgcn_exp2f(__builtin_fmaf(acc[i][j][r], kLog2e, -m_run[j]));
      } else {
#pragma unroll
        for (int i = 0; i < MB; ++i)
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const float e = __builtin_amdgcn_exp2f(__builtin_fmaf(acc[i][j][r], kLog2e, -m_run[j]));
            sum += (32 * i + 8 * (r >> 2) + (r & 3) < lim) ? e : 0.f;
          }
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

  // Merge the two lane halves that share a token column, then the wave rows.
#pragma unroll
  for (int j = 0; j < NB; ++j) {
    const float mo = __shfl_xor(m_run[j], 32);
    const float so = __shfl_xor(s_run[j], 32);
    merge_state(m_run[j], s_run[j], mo, so);
  }
  __syncthreads();  // smem is free after the last tile
  float* red = (float*)smem;  // [WGM][2][BN]
  const int wr = wave / G::WGN;
  if (lane < 32) {
#pragma unroll
    for (int j = 0; j < NB; ++j) {
      red[(wr * 2) * BN + wn + 32 * j + lane] = m_run[j];
      red[(wr * 2 + 1) * BN + wn + 32 * j + lane] = s_run[j];
    }
  }
  __syncthreads();
  if (wr == 0 && lane < 32) {
#pragma unroll
    for (int j = 0; j < NB; ++j) {
      const int c = wn + 32 * j + lane;
      for (int w2 = 1; w2 < G::WGM; ++w2)
        merge_state(m_run[j], s_run[j], red[(w2 * 2) * BN + c], red[(w2 * 2 + 1) * BN + c]);
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

// Per-shard fold (one meeting of Algorithm 2 for a state that travels with the
// activations).  The state's m plane is kept in natural units so that it can be
// exchanged as plain numbers; the kernels work in the base-2 domain.
__global__ void __launch_bounds__(256) state_init_kernel(float* state, int64_t T) {
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= T) return;
  state[t] = -INFINITY;
  state[T + t] = 0.f;
  state[2 * T + t] = 0.f;
}

// state (m, s) <- fold of state and the shard's split partials, in split order.
__global__ void __launch_bounds__(256) fold_merge_kernel(FoldArgs a) {
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= a.T) return;
  const float m_in = a.state[t];
  float m = m_in == -INFINITY ? -INFINITY : m_in * kLog2e;
  float s = a.state[a.T + t];
  for (int k = 0; k < a.n_splits; ++k)
    merge_state(m, s, a.m_part[(int64_t)k * a.T + t], a.s_part[(int64_t)k * a.T + t]);
  a.state[t] = m == -INFINITY ? -INFINITY : m * kLn2;
  a.state[a.T + t] = s;
}

// lse = m + log s and loss = lse - y (0 when ignored, NaN and counted when the
// target is outside [0, V)).
__global__ void __launch_bounds__(256) fold_finalize_kernel(FinArgs a) {
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= a.T) return;
  const float lse = a.state[t] + __builtin_amdgcn_logf(a.state[a.T + t]) * kLn2;
  const int64_t tg = a.targets[t];
  float loss;
  if (tg == a.ignore_index) {
    loss = 0.f;
  } else if (tg < 0 || tg >= a.V) {
    loss = __builtin_nanf("");
    atomicAdd(a.bad_counter, 1ull);
  } else {
    loss = lse - a.state[2 * a.T + t];
  }
  a.lse[t] = lse;
  a.loss[t] = loss;
}

// Byte offset of element (row, col) of a 256 x 256 bfloat16 tile staged in LDS as
// four 64-column blocks of 256 rows x 128 bytes, the 16-byte chunks of each row
// XOR-swizzled by (row / 2) % 8 so that the rows a write or read phase touches
// spread over the banks.  Each block is laid out exactly like the matching
// 32 KiB block of a k-blocked strip.
__device__ __forceinline__ uint32_t tile_lds_byte(int row, int col) {
  return (uint32_t)((col >> 6) * 32768 + row * 128 + ((((col & 63) >> 3) ^ ((row >> 1) & 7)) << 4) +
                    (col & 7) * 2);
}

// Copies the 256 x 256 bfloat16 tile staged in LDS (see tile_lds_byte) to a
// k-blocked strip: block b (columns 64 b .. 64 b + 63) goes to the 32 KiB at
// element ((kb0 + b) * rows_pitch + r0) * 64, one 16-byte chunk per thread and
// step, 1 KiB contiguous per wavefront store.
template <int NT>
__device__ __forceinline__ void store_tile_blocked(const uint16_t* lds, uint16_t* __restrict__ dst,
                                                   uint32_t kb0, uint32_t rows_pitch, uint32_t r0) {
  const int tid = threadIdx.x;
#pragma unroll
  for (int q = 0; q < 8192 / NT; ++q) {
    const int c = q * NT + tid;  // 16-byte chunk of the tile
    const int b = c >> 11, row = (c >> 3) & 255, ch = c & 7;
    const uint4 v = *(const uint4*)((const char*)lds + b * 32768 + row * 128 + ((ch ^ ((row >> 1) & 7)) << 4));
    *(uint4*)(dst + (((kb0 + (uint32_t)b) * rows_pitch + r0 + (uint32_t)row) * 64u + (uint32_t)ch * 8u)) = v;
  }
}

// Backward residual: recompute a logits tile of the (vocabulary chunk, token
// chunk) strip and store G = g (softmax - onehot) into the strip in both layouts:
// G[v][t] (token columns contiguous, for dW) and G^T[t][v] (vocabulary columns
// contiguous, for dH).  Rows and columns of the tile that fall outside the chunk
// are written as zeros so that both contractions can read whole 16-byte chunks
// past a ragged edge.
//
// Every element is first written as g p = sign(g) 2^(y log2e + log2|g| - lse log2e)
// (one multiply-add and one exponential: the upstream gradient is folded into the
// exponent, and an ignored token gets log2|g| = -inf, i.e. zeros); the one element
// of a token column that holds its target is then overwritten, by the one lane that
// owns it, with g (p_t - 1) computed in float32 from the token's target logit yt
// (a separate dot product; it agrees with the tile's own value up to float32
// summation order).  bfloat16 tiles go through LDS (free once the mainloop returns)
// once per layout, so that both layouts leave as whole 16-byte chunks, 1 KiB per
// wavefront store; the target elements are patched in LDS before each store.
template <class E, class G>
__device__ __forceinline__ void grad_tile(const GradArgs& a, int vt, int tb,
                                          typename E::storage* smem) {
  using S = typename E::storage;
  constexpr int BM = G::BM, BN = G::BN, MB = G::MB, NB = G::NB;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = G::wave_m(wave), wn = G::wave_n(wave);
  const int m0 = vt * BM, n0 = tb * BN;

  // The per-token inputs of this lane's token columns are loaded ahead of the
  // mainloop, which drains them with its own loads, so that their latency is not
  // paid after it.  Columns past the chunk read its last token (N >= 1 whenever a
  // residual tile runs) and are masked below.
  int64_t tgv[NB];
  float gv[NB], lsev[NB], ytv[NB];
#pragma unroll
  for (int j = 0; j < NB; ++j) {
    const int64_t t = a.t0 + min(n0 + wn + 32 * j + (lane & 31), a.N - 1);
    tgv[j] = a.targets[t];
    gv[j] = a.grad[t];
    lsev[j] = a.lse[t];
    ytv[j] = a.yt[t];
  }

  f32x16_t acc[MB][NB];
#pragma unroll
  for (int i = 0; i < MB; ++i)
#pragma unroll
    for (int j = 0; j < NB; ++j) acc[i][j] = f32x16_t{};
  G::run(acc, (const S*)a.W, a.d, m0, a.M, (const S*)a.H + a.t0 * a.d, a.d, n0, a.N, a.d, smem);
  // (keeps the compiler from moving arithmetic on the prefetched values, and the wait
  // it needs, in front of the mainloop)
#pragma unroll
  for (int j = 0; j < NB; ++j) asm volatile("" : "+v"(tgv[j]), "+v"(gv[j]), "+v"(lsev[j]), "+v"(ytv[j]));

  // Strip offsets fit in 32 bits (the strip budget is capped below 2^31 elements).
  // Both strips are k-blocked (see GradArgs) with KB = E::KB elements per block.
  constexpr bool kBlocked = sizeof(S) == 2;  // bfloat16 tiles are staged through LDS
  constexpr uint32_t KB = E::KB;
  S* __restrict__ Gs = (S*)a.strip;
  S* __restrict__ Gt = (S*)a.strip_t;
  const uint32_t Tc = (uint32_t)a.Tc, Vc = (uint32_t)a.Vc;
  if constexpr (kBlocked) {
    static_assert(BM == 256 && BN == 256, "the LDS staging holds one 256 x 256 tile");
    static_assert(G::LDS_ELEMS >= BM * BN, "the ring must hold one bfloat16 tile");
  }
  const bool full = m0 + BM <= a.M;  // no padding rows: no row mask
  // row mask of the last tile of a chunk: register group r4 of row block i holds rows
  // m0 + wm + 4 (lane / 32) + 32 i + 8 (r4 / 4) + q
  const int lim = a.M - m0 - wm - 4 * (lane >> 5);
  // Per token column j of this lane: the exponent offset, the sign of g, and the
  // target element this lane owns (tile row, or -1) with its value.
  float cexp[NB], vt_val[NB];
  uint32_t sgn[NB];
  int trow[NB];
#pragma unroll
  for (int j = 0; j < NB; ++j) {
    const int nl = n0 + wn + 32 * j + (lane & 31);  // token column within the chunk
    cexp[j] = -INFINITY;
    sgn[j] = 0u;
    trow[j] = -1;
    vt_val[j] = 0.f;
    if (nl < a.N) {
      const int64_t tg = tgv[j];
      if (tg != a.ignore_index) {
        float g = gv[j];
        if (tg < 0 || tg >= a.V) g = __builtin_nanf("");  // out of range: NaN row
        const float lse2 = lsev[j] * kLog2e;
        const float ag = __builtin_fabsf(g);
        cexp[j] = __builtin_amdgcn_logf(ag) - lse2;  // log2|g| - lse log2e
        sgn[j] = g < 0.f ? 0x80008000u : 0u;
        // the target element: inside the chunk (its padding rows stay zero), in this
        // wave's rows of the tile and in this lane half
        const int64_t rel = tg - a.gid0 - m0 - wm;
        if (tg - a.gid0 < a.M && rel >= 0 && rel < G::WM && (int)((rel >> 2) & 1) == (lane >> 5)) {
          trow[j] = (int)rel + wm;
          const float pt = __builtin_amdgcn_exp2f(__builtin_fmaf(ytv[j], kLog2e, -lse2));
          vt_val[j] = g * (pt - 1.f);
        }
      }
    }
  }
  // G values of this lane, bfloat16 bits packed two per word: packed[j][i][r4/4]
  // holds vocabulary rows ml0 .. ml0 + 3 of token column nl.  Full tiles take the
  // loop without the padding-row mask.
  uint2 packed[NB][MB][4];
  auto residual = [&](auto masked) {
    constexpr bool MASKED = decltype(masked)::value;
#pragma unroll
  for (int j = 0; j < NB; ++j) {
    const int nl = n0 + wn + 32 * j + (lane & 31);
#pragma unroll
    for (int i = 0; i < MB; ++i)
#pragma unroll
      for (int r4 = 0; r4 < 16; r4 += 4) {
        // registers r4..r4+3 hold 4 consecutive vocabulary rows of token column nl
        const int ml0 = m0 + wm + 32 * i + acc_row(r4, lane);
        float v4[4];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const float e = __builtin_amdgcn_exp2f(__builtin_fmaf(acc[i][j][r4 + q], kLog2e, cexp[j]));
          v4[q] = (!MASKED || 32 * i + r4 / 4 * 8 + q < lim) ? e : 0.f;
        }
        if constexpr (kBlocked) {
          packed[j][i][r4 >> 2].x = E::pack2(v4[0], v4[1]) ^ sgn[j];
          packed[j][i][r4 >> 2].y = E::pack2(v4[2], v4[3]) ^ sgn[j];
        } else {
          const float sg = sgn[j] ? -1.f : 1.f;
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            v4[q] *= sg;
            Gs[(((uint32_t)nl / KB) * Vc + (uint32_t)(ml0 + q)) * KB + (uint32_t)nl % KB] = v4[q];
          }
          // 4 consecutive vocabulary rows: one 16-byte store into a 32-wide k-block
          *(float4*)(Gt + (((uint32_t)ml0 / KB) * Tc + (uint32_t)nl) * KB + (uint32_t)ml0 % KB) =
              make_float4(v4[0], v4[1], v4[2], v4[3]);
        }
      }
    if constexpr (!kBlocked) {
      if (trow[j] >= 0) {  // the target element, after this lane's own stores of it
        const uint32_t ml = (uint32_t)(m0 + trow[j]);
        Gs[(((uint32_t)nl / KB) * Vc + ml) * KB + (uint32_t)nl % KB] = vt_val[j];
        Gt[((ml / KB) * Tc + (uint32_t)nl) * KB + ml % KB] = vt_val[j];
      }
    }
  }
  };
  if (full)
    residual(std::false_type{});
  else
    residual(std::true_type{});
  if constexpr (kBlocked) {
    uint16_t* lds = (uint16_t*)smem;
    // G^T: the tile as rows of tokens, columns of vocabulary ids; a lane's 4
    // consecutive ids are one 8-byte write; then the target elements.
#pragma unroll
    for (int j = 0; j < NB; ++j)
#pragma unroll
      for (int i = 0; i < MB; ++i)
#pragma unroll
        for (int r4 = 0; r4 < 16; r4 += 4) {
          const int tl = wn + 32 * j + (lane & 31), vl = wm + 32 * i + acc_row(r4, lane);
          *(uint2*)((char*)lds + tile_lds_byte(tl, vl)) = packed[j][i][r4 >> 2];
        }
    uint16_t tbits[NB];
#pragma unroll
    for (int j = 0; j < NB; ++j) {
      tbits[j] = (uint16_t)(E::pack2(vt_val[j], 0.f) & 0xFFFFu);
      if (trow[j] >= 0)
        *(uint16_t*)((char*)lds + tile_lds_byte(wn + 32 * j + (lane & 31), trow[j])) = tbits[j];
    }
    __syncthreads();
    store_tile_blocked<G::NT>(lds, Gt, (uint32_t)m0 >> 6, Tc, (uint32_t)n0);
    __syncthreads();
    // G: the tile as rows of vocabulary ids, columns of tokens.
#pragma unroll
    for (int j = 0; j < NB; ++j)
#pragma unroll
      for (int i = 0; i < MB; ++i)
#pragma unroll
        for (int r4 = 0; r4 < 16; r4 += 4) {
          const int tl = wn + 32 * j + (lane & 31), vl = wm + 32 * i + acc_row(r4, lane);
          const uint2 p = packed[j][i][r4 >> 2];
          char* base = (char*)lds;
          *(uint16_t*)(base + tile_lds_byte(vl, tl)) = (uint16_t)(p.x & 0xFFFFu);
          *(uint16_t*)(base + tile_lds_byte(vl + 1, tl)) = (uint16_t)(p.x >> 16);
          *(uint16_t*)(base + tile_lds_byte(vl + 2, tl)) = (uint16_t)(p.y & 0xFFFFu);
          *(uint16_t*)(base + tile_lds_byte(vl + 3, tl)) = (uint16_t)(p.y >> 16);
        }
#pragma unroll
    for (int j = 0; j < NB; ++j)
      if (trow[j] >= 0)
        *(uint16_t*)((char*)lds + tile_lds_byte(trow[j], wn + 32 * j + (lane & 31))) = tbits[j];
    __syncthreads();
    store_tile_blocked<G::NT>(lds, Gs, (uint32_t)n0 >> 6, Vc, (uint32_t)m0);
  }
}

// yt[t] = h_t . w_{targets[t]} (float32 sum of the exact products), one wavefront per
// token, 16-byte loads (d is a multiple of 8).  Targets outside [0, V) (ignored or out
// of range) give 0; the residual tiles do not use it for them.
template <class S>
__global__ void __launch_bounds__(256) target_logit_kernel(TgtArgs a) {
  constexpr int VEC = 16 / (int)sizeof(S);
  const int64_t t = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (t >= a.T) return;
  const int64_t tg = a.targets[t];
  float acc = 0.f;
  if (tg >= 0 && tg < a.V) {
    int p = 0;
    while (p + 1 < a.st.P && !(tg >= a.st.off[p] && tg < a.st.off[p] + a.st.rows[p])) ++p;
    const S* w = (const S*)a.st.w[p] + (tg - a.st.off[p]) * (int64_t)a.d;
    const S* h = (const S*)a.H + t * (int64_t)a.d;
    for (int k = lane * VEC; k < a.d; k += 64 * VEC) {
      const uint4 hv = *(const uint4*)(h + k), wv = *(const uint4*)(w + k);
      if constexpr (sizeof(S) == 2) {
        const uint32_t hh[4] = {hv.x, hv.y, hv.z, hv.w}, ww[4] = {wv.x, wv.y, wv.z, wv.w};
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          acc = __builtin_fmaf(__uint_as_float(hh[q] << 16), __uint_as_float(ww[q] << 16), acc);
          acc = __builtin_fmaf(__uint_as_float(hh[q] & 0xFFFF0000u), __uint_as_float(ww[q] & 0xFFFF0000u), acc);
        }
      } else {
        acc = __builtin_fmaf(__uint_as_float(hv.x), __uint_as_float(wv.x), acc);
        acc = __builtin_fmaf(__uint_as_float(hv.y), __uint_as_float(wv.y), acc);
        acc = __builtin_fmaf(__uint_as_float(hv.z), __uint_as_float(wv.z), acc);
        acc = __builtin_fmaf(__uint_as_float(hv.w), __uint_as_float(wv.w), acc);
      }
    }
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) acc += __shfl_xor(acc, o);
  if (lane == 0) a.yt[t] = acc;
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

// One float32 output tile of C = (beta ? C : 0) + A B^T (a dH or a dW tile; N, the
// hidden width, is a multiple of 4).
// Column blocks of a dH / dW contraction, whose N is the hidden width d: BM-wide
// tiles of C^T rows (GM), except that a remainder of at most GW::BM - GM::BM
// columns joins the last full block, which then runs as one GW::BM-wide tile
// instead of leaving a block that is mostly padding (d = 2880: ten 256-wide
// blocks and one 320-wide block, not twelve 256-wide blocks of which the last
// holds 64 live columns).
struct ColBlocks {
  int n;      // column blocks
  bool wide;  // the last block is a GW tile
};
template <class GM, class GW>
__host__ __device__ inline ColBlocks col_blocks(int N) {
  static_assert(GW::BM > GM::BM && GW::BN == GM::BN, "the wide tile only widens C^T rows");
  const int full = N / GM::BM, rem = N % GM::BM;
  if (full >= 1 && rem > 0 && rem <= GW::BM - GM::BM) return ColBlocks{full, true};
  return ColBlocks{(N + GM::BM - 1) / GM::BM, false};
}

// One tile of C (+)= A B^T: rows m0 = mt * BN .. of C, columns n0 .. n0 + BM - 1.
template <class E, class G, bool RAGGED = false>
__device__ __forceinline__ void gemm_tile(const GemmArgs& a, int mt, int n0,
                                          typename E::storage* smem) {
  using S = typename E::storage;
  constexpr int MB = G::MB, NB = G::NB;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = G::wave_m(wave), wn = G::wave_n(wave);
  // The tile is computed transposed, C^T[n][m] = sum_k B[n][k] A[m][k]: accumulator
  // rows run along n, so each lane's group of 4 registers holds 4 consecutive
  // columns of one row of C and the epilogue moves 16 bytes per access.
  const int m0 = mt * G::BN;
  f32x16_t acc[MB][NB];
#pragma unroll
  for (int i = 0; i < MB; ++i)
#pragma unroll
    for (int j = 0; j < NB; ++j) acc[i][j] = f32x16_t{};
  G::template run<RAGGED>(acc, (const S*)a.B, a.ldb, n0, a.N, (const S*)a.A, a.lda, m0, a.M, a.K, smem,
                          a.kblkb, a.kblka);
  // The epilogue takes a lane's row of C a batch of IB row blocks at a time: all
  // old values of the batch (beta = 1) are loaded before the first sum is stored,
  // so the lane waits for memory once per batch rather than once per 16-byte chunk
  // (a store to C ahead of the next load of C would keep the two in order).  Only
  // a RAGGED tile has columns at or past N.
  constexpr int IB = MB <= 4 ? MB : (MB + 1) / 2;
  const bool beta = a.beta != 0;
#pragma unroll
  for (int j = 0; j < NB; ++j) {
    const int m = m0 + wn + 32 * j + (lane & 31);
    if (m >= a.M) continue;
    float* crow = a.C + (int64_t)m * a.ldc;
#pragma unroll
    for (int i0 = 0; i0 < MB; i0 += IB) {
      float4 old[IB][4];
#pragma unroll
      for (int ii = 0; ii < IB; ++ii)
#pragma unroll
        for (int q = 0; q < 4; ++q) old[ii][q] = make_float4(0.f, 0.f, 0.f, 0.f);
      if (beta) {
#pragma unroll
        for (int ii = 0; ii < IB; ++ii)
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            const int i = i0 + ii;
            const int n = n0 + wm + 32 * i + acc_row(4 * q, lane);  // n .. n+3; N % 4 == 0
            if (i < MB && (!RAGGED || n < a.N)) old[ii][q] = *(const float4*)(crow + n);
          }
      }
#pragma unroll
      for (int ii = 0; ii < IB; ++ii)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int i = i0 + ii;
          const int n = n0 + wm + 32 * i + acc_row(4 * q, lane);
          if (i >= MB || (RAGGED && n >= a.N)) continue;
          const float4 c = old[ii][q];
          *(float4*)(crow + n) = make_float4(acc[i][j][4 * q] + c.x, acc[i][j][4 * q + 1] + c.y,
                                             acc[i][j][4 * q + 2] + c.z, acc[i][j][4 * q + 3] + c.w);
        }
    }
  }
}

// One launch of the backward pipeline: the dH and dW tiles of strip c and
// the residual tiles of strip c+1 (which writes the other strip buffer).  XCD x
// runs cnt[0][x] dH tiles, then cnt[1][x] dW tiles, then cnt[2][x] residual
// tiles (numbered from first[.][x]): every XCD gets an even share of each kind,
// consecutive tiles of one kind stay on one XCD's L2, and the longest tiles go
// first so that the partly filled last round is made of the short ones.
template <class E, class GL, class GM, class GW>
__global__ void __launch_bounds__(GM::NT, GM::OCC)
    bwd_stage_kernel(GemmArgs h, GemmArgs w, GradArgs g, StageSplit sp) {
  static_assert(GL::NT == GM::NT && GW::NT == GM::NT, "one workgroup size for every tile kind");
  using S = typename E::storage;
  constexpr int LDS0 = GL::LDS_ELEMS > GM::LDS_ELEMS ? GL::LDS_ELEMS : GM::LDS_ELEMS;
  constexpr int LDS = LDS0 > GW::LDS_ELEMS ? LDS0 : GW::LDS_ELEMS;
  __shared__ __attribute__((aligned(16))) S smem[LDS];
  const int xcd = blockIdx.x % 8;
  int local = blockIdx.x / 8;
  int mt, nt;
  // dH (kind 0) and dW (kind 1) tiles (see col_blocks); a tile that reaches past the
  // hidden width d runs ragged: the waves' row blocks past d do no MFMA work.
#pragma unroll
  for (int k = 0; k < 2; ++k) {
    const GemmArgs& a = k == 0 ? h : w;
    if (local < sp.cnt[k][xcd]) {
      const ColBlocks cb = col_blocks<GM, GW>(a.N);
      const int n_m = (a.M + GM::BN - 1) / GM::BN;
      grouped_tile(sp.first[k][xcd] + local, n_m, cb.n, 4, mt, nt);
      const int n0 = nt * GM::BM;
      if (cb.wide && nt == cb.n - 1) {
        if (n0 + GW::BM > a.N)
          gemm_tile<E, GW, true>(a, mt, n0, smem);
        else
          gemm_tile<E, GW>(a, mt, n0, smem);
      } else if (n0 + GM::BM > a.N) {
        gemm_tile<E, GM, true>(a, mt, n0, smem);
      } else {
        gemm_tile<E, GM>(a, mt, n0, smem);
      }
      return;
    }
    local -= sp.cnt[k][xcd];
  }
  const int n_tb = (g.N + GL::BN - 1) / GL::BN;
  grouped_tile(sp.first[2][xcd] + local, g.n_vt, n_tb, 4, mt, nt);
  grad_tile<E, GL>(g, mt, nt, smem);
}

// out = in^T in the k-blocked layout: in is row-major [R][ld_in]; out is
// [R_pad / KB][C][KB] with KB = 128 / sizeof(S) (element (c, r) at
// ((r / KB) C + c) KB + r % KB), zero for R <= r < R_pad.  One 64 x 64 tile per
// workgroup (one-dimensional grid, row blocks fastest: T / 64 up to 2^17 and
// d / 64 up to 2^16 exceed a grid dimension), staged through LDS with 16-byte
// accesses to global memory on both sides.  A tile row of 64 elements is VPR
// 16-byte vectors; vector v of tile row i sits in slot v ^ ((i / VEC) % VPR), so
// that the column reads of the store side (VEC consecutive rows of one column
// per lane, rows VEC g .. VEC g + VEC - 1 for lane group g) fall in distinct
// banks.  Needs C, ld_in and both base addresses in whole 16-byte vectors and
// R_pad a multiple of KB (checked by run_transpose).
template <class S>
__global__ void __launch_bounds__(256) transpose_kernel(TransposeArgs a) {
  constexpr int VEC = 16 / (int)sizeof(S);  // elements per 16-byte vector
  constexpr int VPR = 64 / VEC;             // vectors per tile row
  constexpr int ROWS = 256 / VPR;           // tile rows (or output rows) per pass
  constexpr int KB = 128 / (int)sizeof(S);
  __shared__ __attribute__((aligned(16))) S tile[64][64];
  const S* in = (const S*)a.in;
  S* out = (S*)a.out;
  const uint32_t n_rb = ((uint32_t)a.R_pad + 63u) / 64u;
  const int r0 = (int)(blockIdx.x % n_rb) * 64, c0 = (int)(blockIdx.x / n_rb) * 64;
  const int v = threadIdx.x % VPR, i0 = threadIdx.x / VPR;
#pragma unroll
  for (int i = i0; i < 64; i += ROWS) {
    const int r = r0 + i, c = c0 + VEC * v;
    uint4 x = make_uint4(0u, 0u, 0u, 0u);
    if (r < a.R && c < a.C) x = *(const uint4*)(in + (int64_t)r * a.ld_in + c);
    *(uint4*)&tile[i][(v ^ ((i / VEC) % VPR)) * VEC] = x;
  }
  __syncthreads();
  // lane group g = v gathers tile rows VEC g .. VEC g + VEC - 1 of one column
#pragma unroll
  for (int cl = i0; cl < 64; cl += ROWS) {
    const int c = c0 + cl, r = r0 + VEC * v;
    if (c < a.C && r < a.R_pad) {
      union {
        uint4 u;
        S e[VEC];
      } y;
#pragma unroll
      for (int j = 0; j < VEC; ++j) y.e[j] = tile[VEC * v + j][((cl / VEC) ^ v) * VEC + cl % VEC];
      *(uint4*)(out + ((int64_t)(r / KB) * a.C + c) * KB + r % KB) = y.u;
    }
  }
}

// ---------------------------------------------------------------------------
// Tile configurations.  Both element types: the direct-to-LDS ring (128-byte
// slice rows: 64 bfloat16 or 32 float32 k values, two slots) with 256 x 256
// tiles; the register-staged tile of the same shape when d is not a multiple of
// the slice depth.
template <class E> struct Cfg;
template <> struct Cfg<Bf16> {
  // 512-thread workgroups (two wavefronts per SIMD), 256 x 256 tiles, 128 x 64 per
  // wave, for every contraction (measured faster inside the backward stage launch
  // than 256 x 192 tiles with 64 x 96 per wave, whose fragment reads per MFMA are
  // higher).  One wavefront per SIMD with 128 x 128 per wave reads a third less LDS
  // per MFMA and runs at a higher clock, but measured 5-17% slower: a lone wave's
  // load waits and barrier waits idle the MFMA pipe.
  using Logits = GemmDma<256, 256, 2, 4>;
  using Mm = Logits;  // the dH / dW contractions
  // the last dH / dW column block when d leaves 1..64 columns past a multiple of
  // 256 (160 x 64 per wave, 0.7 fragment reads per MFMA)
  using MmWide = GemmDma<320, 256, 2, 4>;
  using LogitsReg = Gemm<Bf16, Logits::BM, Logits::BN, Logits::WGM, Logits::WGN>;
  static_assert(64 % Mm::KDIV == 0, "dH / dW launch granularity");
  static constexpr int KALIGN = 64;  // K granularity the dH / dW launches need
};
template <> struct Cfg<F32> {
  // The same direct-to-LDS ring and 256 x 256 tiles: 32 float32 k values per slice,
  // four 32x32x2 f32 MFMAs per fragment pair.  d not a multiple of 32: the
  // register-staged tile of the same shape.
  using Logits = GemmDma<256, 256, 2, 4, 64, 2, F32>;
  using Mm = Logits;  // the dH / dW contractions
  using MmWide = GemmDma<320, 256, 2, 4, 64, 2, F32>;
  using LogitsReg = Gemm<F32, Logits::BM, Logits::BN, Logits::WGM, Logits::WGN>;
  static constexpr int KALIGN = 32;  // K granularity the dH / dW launches need
};

static inline bool launched_ok() { return hipGetLastError() == hipSuccess; }

template <class E, class G>
static bool launch_fwd_g(const FwdArgs& a, hipStream_t s) {
  const unsigned grid = (unsigned)(a.n_tok_blocks * a.n_splits);
  hipLaunchKernelGGL((fwd_kernel<E, G>), dim3(grid), dim3(G::NT), 0, s, a);
  return launched_ok();
}
template <class E>
static bool launch_fwd(const FwdArgs& a, hipStream_t s) {
  if (a.d % Cfg<E>::Logits::KDIV == 0) return launch_fwd_g<E, typename Cfg<E>::Logits>(a, s);
  return launch_fwd_g<E, typename Cfg<E>::LogitsReg>(a, s);
}
// Per-XCD split of n0 + n1 + n2 workgroups (workgroup b runs on XCD b % 8, so
// XCD x receives n/8 of them, one more for x < n%8): kinds 0 and 1 are spread
// as evenly as the capacity allows, kind 2 takes the rest.
static StageSplit split_stage(const int n_kind[3]) {
  StageSplit sp;
  const int n = n_kind[0] + n_kind[1] + n_kind[2];
  int cap[8];
  for (int x = 0; x < 8; ++x) cap[x] = n / 8 + (x < n % 8 ? 1 : 0);
  for (int t = 0; t < 2; ++t) {
    int give = n_kind[t];
    for (int x = 0; x < 8; ++x) {
      const int c = std::min(cap[x], n_kind[t] / 8);
      sp.cnt[t][x] = c;
      cap[x] -= c;
      give -= c;
    }
    for (int x = 0; give > 0; x = (x + 1) % 8)
      if (cap[x] > 0) {
        ++sp.cnt[t][x];
        --cap[x];
        --give;
      }
  }
  for (int x = 0; x < 8; ++x) sp.cnt[2][x] = cap[x];
  for (int t = 0; t < 3; ++t) {
    int f = 0;
    for (int x = 0; x < 8; ++x) {
      sp.first[t][x] = f;
      f += sp.cnt[t][x];
    }
  }
  return sp;
}

template <class E, class GL, class GM, class GW>
static bool launch_stage_g(const GemmArgs& h, const GemmArgs& w, const GradArgs& g, hipStream_t s) {
  auto tiles = [](const GemmArgs& a) {  // C^T tiles: column blocks along N, BN along M
    return a.M > 0 ? ((a.M + GM::BN - 1) / GM::BN) * col_blocks<GM, GW>(a.N).n : 0;
  };
  int n_kind[3];
  n_kind[0] = tiles(h);
  n_kind[1] = tiles(w);
  n_kind[2] = g.M > 0 ? g.n_vt * ((g.N + GL::BN - 1) / GL::BN) : 0;
  const int n = n_kind[0] + n_kind[1] + n_kind[2];
  if (n == 0) return true;
  const StageSplit sp = split_stage(n_kind);
  hipLaunchKernelGGL((bwd_stage_kernel<E, GL, GM, GW>), dim3((unsigned)n), dim3(GM::NT), 0, s, h,
                     w, g, sp);
  return launched_ok();
}
template <class E>
static bool launch_stage(const GemmArgs& h, const GemmArgs& w, const GradArgs& g, hipStream_t s) {
  using Mm = typename Cfg<E>::Mm;
  using Wd = typename Cfg<E>::MmWide;
  if (g.d % Cfg<E>::Logits::KDIV == 0)
    return launch_stage_g<E, typename Cfg<E>::Logits, Mm, Wd>(h, w, g, s);
  return launch_stage_g<E, typename Cfg<E>::LogitsReg, Mm, Wd>(h, w, g, s);
}

// ---------------------------------------------------------------------------
// Library-owned forward workspace for callers that cannot allocate (see
// vp_ce_forward_noalloc).  Each device the library runs on holds its own copy
// from the first use until the process ends.  In host code `scratch` names a
// host-side stand-in, not device memory: its device address is looked up once
// per device with hipGetSymbolAddress, and only that address is ever passed on.
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

namespace {
constexpr int kMaxDevices = 64;
std::mutex scratch_mu;
void* scratch_addr[kMaxDevices] = {};
}  // namespace

bool scratch_base(void** out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return false;
  std::lock_guard<std::mutex> lock(scratch_mu);
  if (!scratch_addr[dev]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return false;
    scratch_addr[dev] = p;
  }
  *out = scratch_addr[dev];
  return true;
}

// ---- entry points used by the host API (vpce_api.cpp) ----
TileShape tile_shape(int dtype) {
  static_assert(Cfg<Bf16>::Logits::BM == Cfg<Bf16>::LogitsReg::BM &&
                    Cfg<Bf16>::Logits::BN == Cfg<Bf16>::LogitsReg::BN,
                "both logits mainloops must share the tile shape");
  static_assert(Cfg<F32>::Logits::BM == Cfg<F32>::LogitsReg::BM &&
                    Cfg<F32>::Logits::BN == Cfg<F32>::LogitsReg::BN,
                "both logits mainloops must share the tile shape");
  static_assert(Cfg<Bf16>::KALIGN == Bf16::KB && Cfg<F32>::KALIGN == F32::KB,
                "dH / dW contractions read whole k-blocks");
  TileShape t;
  if (dtype == 1) {
    t.fwd_bm = t.grad_bm = Cfg<Bf16>::Logits::BM;
    t.fwd_bn = t.grad_bn = Cfg<Bf16>::Logits::BN;
    t.kalign = Cfg<Bf16>::KALIGN;
    t.kblock = Bf16::KB;
  } else {
    t.fwd_bm = t.grad_bm = Cfg<F32>::Logits::BM;
    t.fwd_bn = t.grad_bn = Cfg<F32>::Logits::BN;
    t.kalign = Cfg<F32>::KALIGN;
    t.kblock = F32::KB;
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
bool run_state_init(float* state, int64_t T, hipStream_t s) {
  if (T <= 0) return true;
  hipLaunchKernelGGL(state_init_kernel, dim3((unsigned)((T + 255) / 256)), dim3(256), 0, s, state, T);
  return launched_ok();
}
bool run_fold_merge(const FoldArgs& a, hipStream_t s) {
  if (a.T <= 0) return true;
  hipLaunchKernelGGL(fold_merge_kernel, dim3((unsigned)((a.T + 255) / 256)), dim3(256), 0, s, a);
  return launched_ok();
}
bool run_fold_finalize(const FinArgs& a, hipStream_t s) {
  if (a.T <= 0) return true;
  hipLaunchKernelGGL(fold_finalize_kernel, dim3((unsigned)((a.T + 255) / 256)), dim3(256), 0, s, a);
  return launched_ok();
}
bool run_count_bad(const int64_t* targets, int64_t T, int64_t V, int64_t ignore_index,
                   unsigned long long* counter, hipStream_t s) {
  if (T <= 0) return true;
  hipLaunchKernelGGL(count_bad_kernel, dim3((unsigned)((T + 255) / 256)), dim3(256), 0, s, targets,
                     T, V, ignore_index, counter);
  return launched_ok();
}
bool run_bwd_stage(int dtype, const GemmArgs& h, const GemmArgs& w, const GradArgs& g,
                   hipStream_t s) {
  return dtype == 1 ? launch_stage<Bf16>(h, w, g, s) : launch_stage<F32>(h, w, g, s);
}
bool run_target_logits(int dtype, const TgtArgs& a, hipStream_t s) {
  if (a.T <= 0) return true;
  const dim3 grid((unsigned)((a.T + 3) / 4));
  if (dtype == 1)
    hipLaunchKernelGGL(target_logit_kernel<uint16_t>, grid, dim3(256), 0, s, a);
  else
    hipLaunchKernelGGL(target_logit_kernel<float>, grid, dim3(256), 0, s, a);
  return launched_ok();
}
bool run_transpose(int dtype, const TransposeArgs& a, hipStream_t s) {
  if (a.C <= 0 || a.R_pad <= 0) return true;
  const int esz = dtype == 1 ? 2 : 4, vec = 16 / esz, kb = 128 / esz;
  // the 16-byte accesses of the kernel: whole vectors on both sides, whole k-blocks
  if (a.C % vec != 0 || a.ld_in % vec != 0 || a.R_pad % kb != 0 || a.R < 0 || a.R > a.R_pad ||
      ((uintptr_t)a.in & 15u) != 0 || ((uintptr_t)a.out & 15u) != 0)
    return false;
  const int64_t blocks = (int64_t)((a.R_pad + 63) / 64) * ((a.C + 63) / 64);
  if (blocks > 0x7fffffff) return false;  // beyond any operand that fits in memory
  const dim3 grid((unsigned)blocks);
  if (dtype == 1)
    hipLaunchKernelGGL(transpose_kernel<uint16_t>, grid, dim3(256), 0, s, a);
  else
    hipLaunchKernelGGL(transpose_kernel<float>, grid, dim3(256), 0, s, a);
  return launched_ok();
}

}  // namespace vpce
