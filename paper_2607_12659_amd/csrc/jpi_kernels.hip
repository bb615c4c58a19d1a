// HIP kernels of the action-expert denoiser for gfx950 (CDNA4).
//
// Matrix products run on MFMA: bf16 data uses v_mfma_f32_16x16x32_bf16,
// fp32 data v_mfma_f32_16x16x4_f32, both accumulating in fp32.  One tile loop
// serves both: a lane of a 64-wide wave holds KPL consecutive k values of one
// row of the A operand (row = lane % 16, k group = lane / 16) and the same k
// values of one column of the B operand; the 16x16 result holds
// D[4 * (lane / 16) + i][lane % 16] in element i.
//
// Every reduction (split-K partial sums, attention chunk combine, row norms)
// is summed in a fixed order, so results are bitwise reproducible.
#include <math.h>
#include <stdlib.h>

#include "jpi_device.h"
#include "jpi_internal.h"

namespace jpi {



// ===========================================================================
// GEMM: acc[m][n] = sum_k A[m][k] W[n][k], A and W row-major with leading
// dimension K.  With splitk > 1, blockIdx.z owns the K slice
// [z K/splitk, (z+1) K/splitk) and the epilogue must be EPI_STORE_F32, which
// then writes slice z's partial sums to out_f32 + z*M*N; a separate row kernel
// sums the slices in order (no cross-workgroup signalling inside a GEMM).
// ===========================================================================
// Store that writes through the compute die's L2 (a relaxed device-scope
// atomic store: cache policy sc1).  The split-K slices, read by the row kernel
// on every die, then do not wait in L2 for the end-of-kernel write-back
// (measured on the batch-8 call: 14.71 -> 14.32 ms; the same for the bf16
// z, q, k, v and attention outputs was slower).
__device__ __forceinline__ void store_wt(float* p, float v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

template <typename T, EpiKind EPI>
__device__ __forceinline__ void epilogue_pair(const EpiParams& ep, float* out_f32, int M, int N, int row, int col_lo,
                                              float lo, float hi) {
  if (row >= M) return;
  const int col_hi = col_lo + 16;
  // packed 32-column groups never straddle N (a multiple of 32 for these epilogues)
  if constexpr (EPI != EPI_STORE_F32) {
    if (col_lo >= N) return;
  }
  if constexpr (EPI == EPI_STORE_F32) {
    if (col_lo < N) store_wt(&out_f32[(size_t)row * N + col_lo], lo);
    if (col_hi < N) store_wt(&out_f32[(size_t)row * N + col_hi], hi);
  } else if constexpr (EPI == EPI_GEGLU) {
    // packed group t of 32 columns: [gate f = 16t + c | up f = 16t + c]
    const int f = (col_lo >> 5) * 16 + (col_lo & 15);
    reinterpret_cast<T*>(ep.z)[(size_t)row * ep.mlp_dim + f] = from_f32<T>(gelu_tanh(lo) * hi);
  } else if constexpr (EPI == EPI_QKV) {
    const int Dh = ep.head_dim, half = Dh >> 1, H = ep.horizon;
    const int b = row / H, i = row - b * H;
    const int qcols = ep.n_heads * Dh;
    if (col_lo < qcols + Dh) {
      // q head or k: packed group t of 32 columns holds the RoPE pairs
      // (d, d + Dh/2), d = 16t + c, in columns (32t + c, 32t + 16 + c)
      const int hn = col_lo < qcols ? col_lo / Dh : -1;
      const int within = col_lo < qcols ? col_lo - hn * Dh : col_lo - qcols;
      const int d = (within >> 5) * 16 + (within & 15);
      const float2 cs = ep.rope[((size_t)b * H + i) * half + d];
      const float r_lo = lo * cs.x - hi * cs.y;
      const float r_hi = lo * cs.y + hi * cs.x;
      const size_t kbs = ep.ks_bstride ? (size_t)ep.ks_bstride : (size_t)H * Dh;
      T* dst = hn >= 0 ? reinterpret_cast<T*>(ep.q) + (((size_t)b * ep.n_heads + hn) * H + i) * Dh
                       : reinterpret_cast<T*>(ep.ks) + b * kbs + (size_t)i * Dh;
      dst[d] = from_f32<T>(r_lo);
      dst[d + half] = from_f32<T>(r_hi);
    } else {
      const int within = col_lo - qcols - Dh;  // v: natural order, stored transposed [b][d][i]
      T* dst = reinterpret_cast<T*>(ep.vst) + (size_t)b * Dh * ep.vst_ld + i;
      dst[(size_t)within * ep.vst_ld] = from_f32<T>(lo);
      dst[(size_t)(within + 16) * ep.vst_ld] = from_f32<T>(hi);
    }
  }
}

// Rotation factors of an EPI_QKV result pair (row, col_lo), or (1, 0) where
// none applies (V columns, rows past M).  They do not depend on the product,
// so a kernel can load them before its K loop and pass them to the epilogue.
__device__ __forceinline__ float2 qkv_rope_factor(const EpiParams& ep, int M, int N, int row, int col_lo) {
  const int Dh = ep.head_dim, qcols = ep.n_heads * Dh;
  if (row >= M || col_lo >= N || col_lo >= qcols + Dh) return float2{1.f, 0.f};
  const int hn = col_lo < qcols ? col_lo / Dh : -1;
  const int within = col_lo < qcols ? col_lo - hn * Dh : col_lo - qcols;
  const int d = (within >> 5) * 16 + (within & 15);
  return ep.rope[(size_t)row * (Dh >> 1) + d];  // row = b * H + i
}

// EPI_QKV epilogue with the rotation factors already in hand
template <typename T>
__device__ __forceinline__ void epilogue_qkv_pre(const EpiParams& ep, int M, int N, int row, int col_lo, float lo,
                                                 float hi, float2 cs) {
  if (row >= M || col_lo >= N) return;
  const int Dh = ep.head_dim, half = Dh >> 1, H = ep.horizon;
  const int b = row / H, i = row - b * H;
  const int qcols = ep.n_heads * Dh;
  if (col_lo < qcols + Dh) {
    const int hn = col_lo < qcols ? col_lo / Dh : -1;
    const int within = col_lo < qcols ? col_lo - hn * Dh : col_lo - qcols;
    const int d = (within >> 5) * 16 + (within & 15);
    const float r_lo = lo * cs.x - hi * cs.y;
    const float r_hi = lo * cs.y + hi * cs.x;
    const size_t kbs = ep.ks_bstride ? (size_t)ep.ks_bstride : (size_t)H * Dh;
    T* dst = hn >= 0 ? reinterpret_cast<T*>(ep.q) + (((size_t)b * ep.n_heads + hn) * H + i) * Dh
                     : reinterpret_cast<T*>(ep.ks) + b * kbs + (size_t)i * Dh;
    dst[d] = from_f32<T>(r_lo);
    dst[d + half] = from_f32<T>(r_hi);
  } else {
    const int within = col_lo - qcols - Dh;
    T* dst = reinterpret_cast<T*>(ep.vst) + (size_t)b * Dh * ep.vst_ld + i;
    dst[(size_t)within * ep.vst_ld] = from_f32<T>(lo);
    dst[(size_t)(within + 16) * ep.vst_ld] = from_f32<T>(hi);
  }
}

// ---- tiled GEMM for M > 64: workgroup tile BM x BN, 4 waves in 2 x 2, K
// staged through LDS in BK slices with register double buffering.  An LDS
// row is one 128-byte slice row (8 chunks of 16 bytes); chunk c of row r is
// stored at position c ^ ((r >> 1) & 7), so that the 16 lanes of an LDS
// cycle touch distinct banks both when a slice is written (two rows of 8
// chunks) and when MFMA fragments are read (16 rows, one chunk each) --------
template <typename T, int BM, int BN>
struct GemmShape {
  static constexpr int BK = sizeof(T) == 2 ? 64 : 32;
  static constexpr int VEC = 16 / sizeof(T);      // elements per 16-byte chunk
  static constexpr int LDK = BK;                  // LDS row: 128 bytes, chunks swizzled
  static constexpr int WM = BM / 2, WN = BN / 2;  // wave tile
  static constexpr int TM = WM / 16, TN = WN / 16;
  static constexpr int CPR = BK / VEC;            // 16-byte chunks per tile row
  static constexpr int A_CH = BM * CPR / 256;
  static constexpr int W_CH = BN * CPR / 256;
  static_assert(TN % 2 == 0, "epilogues pair n-subtiles 2t and 2t+1");
  static_assert(A_CH >= 1 && W_CH >= 1, "tile too small for 256 threads");
  static_assert(CPR == 8, "the swizzle permutes 8 chunks per row");
  // element offset of (row r, chunk c) in a tile
  static __device__ __forceinline__ int at(int r, int c) { return r * LDK + ((c ^ ((r >> 1) & 7)) * VEC); }
};

template <typename T, int BM, int BN, EpiKind EPI>
__global__ __launch_bounds__(256) void k_gemm(GemmLaunch g) {
  using S = GemmShape<T, BM, BN>;
  using MF = Mfma<T>;
  __shared__ __attribute__((aligned(16))) T As[2][BM * S::LDK];
  __shared__ __attribute__((aligned(16))) T Ws[2][BN * S::LDK];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int m0 = blockIdx.y * BM, n0 = blockIdx.x * BN;
  const int M = g.M, N = g.N, K = g.K;
  const int kper = K / g.splitk;
  const int kbeg = blockIdx.z * kper;
  const int nkt = kper / S::BK;
  const T* A = reinterpret_cast<const T*>(g.A);
  const T* W = reinterpret_cast<const T*>(g.W);

  uint4 ra[S::A_CH], rw[S::W_CH];
  auto gload = [&](int kt) {
    const int k0 = kbeg + kt * S::BK;
#pragma unroll
    for (int c = 0; c < S::A_CH; ++c) {
      const int e = tid + c * 256, r = e / S::CPR, cc = e - r * S::CPR;
      const int row = m0 + r;
      ra[c] = row < M ? *reinterpret_cast<const uint4*>(A + (size_t)row * K + k0 + cc * S::VEC)
                      : make_uint4(0, 0, 0, 0);
    }
#pragma unroll
    for (int c = 0; c < S::W_CH; ++c) {
      const int e = tid + c * 256, r = e / S::CPR, cc = e - r * S::CPR;
      const int n = n0 + r;
      rw[c] = n < N ? *reinterpret_cast<const uint4*>(W + (size_t)n * K + k0 + cc * S::VEC)
                    : make_uint4(0, 0, 0, 0);
    }
  };
  auto sstore = [&](int buf) {
#pragma unroll
    for (int c = 0; c < S::A_CH; ++c) {
      const int e = tid + c * 256, r = e / S::CPR, cc = e - r * S::CPR;
      *reinterpret_cast<uint4*>(&As[buf][S::at(r, cc)]) = ra[c];
    }
#pragma unroll
    for (int c = 0; c < S::W_CH; ++c) {
      const int e = tid + c * 256, r = e / S::CPR, cc = e - r * S::CPR;
      *reinterpret_cast<uint4*>(&Ws[buf][S::at(r, cc)]) = rw[c];
    }
  };

  f32x4 acc[S::TM][S::TN];
#pragma unroll
  for (int a = 0; a < S::TM; ++a)
#pragma unroll
    for (int b = 0; b < S::TN; ++b) acc[a][b] = f32x4{0.f, 0.f, 0.f, 0.f};

  const int fr = lane & 15, fk = (lane >> 4) * MF::KPL;
  gload(0);
  sstore(0);
  __syncthreads();
  for (int kt = 0; kt < nkt; ++kt) {
    const int buf = kt & 1;
    if (kt + 1 < nkt) gload(kt + 1);
#pragma unroll
    for (int kk = 0; kk < S::BK; kk += MF::KSUB) {
      // lane reads k values kk + fk .. + KPL of its row: one chunk (bf16) or part of one (fp32)
      const int kc = (kk + fk) / S::VEC, ke = (kk + fk) % S::VEC;
      typename MF::frag af[S::TM], bfr[S::TN];
#pragma unroll
      for (int a = 0; a < S::TM; ++a) af[a] = MF::load(As[buf] + S::at(wm * S::WM + a * 16 + fr, kc) + ke);
#pragma unroll
      for (int b = 0; b < S::TN; ++b) bfr[b] = MF::load(Ws[buf] + S::at(wn * S::WN + b * 16 + fr, kc) + ke);
#pragma unroll
      for (int a = 0; a < S::TM; ++a)
#pragma unroll
        for (int b = 0; b < S::TN; ++b) acc[a][b] = MF::run(af[a], bfr[b], acc[a][b]);
    }
    if (kt + 1 < nkt) sstore(buf ^ 1);
    __syncthreads();
  }

  const int rbase = m0 + wm * S::WM + (lane >> 4) * 4;
  const int cbase = n0 + wn * S::WN + fr;
  float* out = g.ep.out_f32 ? g.ep.out_f32 + (size_t)blockIdx.z * M * N : nullptr;
#pragma unroll
  for (int a = 0; a < S::TM; ++a)
#pragma unroll
    for (int b = 0; b < S::TN; b += 2)
#pragma unroll
      for (int i = 0; i < 4; ++i)
        epilogue_pair<T, EPI>(g.ep, out, M, N, rbase + a * 16 + i, cbase + b * 16, acc[a][b][i], acc[a][b + 1][i]);
}

// ---- large bf16 GEMM tiles: 256 x 256 per workgroup, 8 waves in 2 x 4
// (wave tile 128 x 64), the same swizzled 128-byte LDS rows and register
// double buffering as k_gemm.  A K slice moves 64 KB for four times the
// products of a 128 x 128 tile, half the bytes per product. ------------------
template <int BM_, int BN_>
struct BigShape {
  static constexpr int BM = BM_, BN = BN_, BK = 64, VEC = 8, CPR = 8, NT = 512;
  static constexpr int WM = BM / 2, WN = BN / 4, TM = WM / 16, TN = WN / 16;
  static constexpr int A_CH = BM * CPR / NT, W_CH = BN * CPR / NT;  // 16-byte chunks per thread
  static_assert(A_CH >= 1 && W_CH >= 1 && TN % 2 == 0, "tile shape");
  static __device__ __forceinline__ int at(int r, int c) { return r * BK + ((c ^ ((r >> 1) & 7)) * VEC); }
};
typedef BigShape<256, 256> Big256;

template <typename S, EpiKind EPI>
__global__ __launch_bounds__(512) void k_gemm_big(GemmLaunch g) {
  using MF = Mfma<bf16>;
  __shared__ __attribute__((aligned(16))) bf16 As[2][S::BM * S::BK];
  __shared__ __attribute__((aligned(16))) bf16 Ws[2][S::BN * S::BK];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 2, wn = wave & 3;
  const int m0 = blockIdx.y * S::BM, n0 = blockIdx.x * S::BN;
  const int M = g.M, N = g.N, K = g.K;
  const int kper = K / g.splitk, kbeg = blockIdx.z * kper, nkt = kper / S::BK;
  const bf16* A = reinterpret_cast<const bf16*>(g.A);
  const bf16* W = reinterpret_cast<const bf16*>(g.W);
  uint4 ra[S::A_CH], rw[S::W_CH];
  auto gload = [&](int kt) {
    const int k0 = kbeg + kt * S::BK;
#pragma unroll
    for (int c = 0; c < S::A_CH; ++c) {
      const int e = tid + c * S::NT, r = e / S::CPR, cc = e - r * S::CPR, row = m0 + r;
      ra[c] = row < M ? *reinterpret_cast<const uint4*>(A + (size_t)row * K + k0 + cc * S::VEC) : make_uint4(0, 0, 0, 0);
    }
#pragma unroll
    for (int c = 0; c < S::W_CH; ++c) {
      const int e = tid + c * S::NT, r = e / S::CPR, cc = e - r * S::CPR, n = n0 + r;
      rw[c] = n < N ? *reinterpret_cast<const uint4*>(W + (size_t)n * K + k0 + cc * S::VEC) : make_uint4(0, 0, 0, 0);
    }
  };
  auto sstore = [&](int buf) {
#pragma unroll
    for (int c = 0; c < S::A_CH; ++c) {
      const int e = tid + c * S::NT, r = e / S::CPR, cc = e - r * S::CPR;
      *reinterpret_cast<uint4*>(&As[buf][S::at(r, cc)]) = ra[c];
    }
#pragma unroll
    for (int c = 0; c < S::W_CH; ++c) {
      const int e = tid + c * S::NT, r = e / S::CPR, cc = e - r * S::CPR;
      *reinterpret_cast<uint4*>(&Ws[buf][S::at(r, cc)]) = rw[c];
    }
  };
  f32x4 acc[S::TM][S::TN];
#pragma unroll
  for (int a = 0; a < S::TM; ++a)
#pragma unroll
    for (int b = 0; b < S::TN; ++b) acc[a][b] = f32x4{0.f, 0.f, 0.f, 0.f};
  const int fr = lane & 15, fk = (lane >> 4) * MF::KPL;
  gload(0);
  sstore(0);
  __syncthreads();
  for (int kt = 0; kt < nkt; ++kt) {
    const int buf = kt & 1;
    if (kt + 1 < nkt) gload(kt + 1);
#pragma unroll
    for (int kk = 0; kk < S::BK; kk += MF::KSUB) {
      const int kc = (kk + fk) / S::VEC;
      MF::frag af[S::TM], bfr[S::TN];
#pragma unroll
      for (int a = 0; a < S::TM; ++a) af[a] = MF::load(As[buf] + S::at(wm * S::WM + a * 16 + fr, kc));
#pragma unroll
      for (int b = 0; b < S::TN; ++b) bfr[b] = MF::load(Ws[buf] + S::at(wn * S::WN + b * 16 + fr, kc));
#pragma unroll
      for (int a = 0; a < S::TM; ++a)
#pragma unroll
        for (int b = 0; b < S::TN; ++b) acc[a][b] = MF::run(af[a], bfr[b], acc[a][b]);
    }
    if (kt + 1 < nkt) sstore(buf ^ 1);
    __syncthreads();
  }
  const int rbase = m0 + wm * S::WM + (lane >> 4) * 4;
  const int cbase = n0 + wn * S::WN + fr;
  float* out = g.ep.out_f32 ? g.ep.out_f32 + (size_t)blockIdx.z * M * N : nullptr;
#pragma unroll
  for (int a = 0; a < S::TM; ++a)
#pragma unroll
    for (int b = 0; b < S::TN; b += 2)
#pragma unroll
      for (int i = 0; i < 4; ++i)
        epilogue_pair<bf16, EPI>(g.ep, out, M, N, rbase + a * 16 + i, cbase + b * 16, acc[a][b][i], acc[a][b + 1][i]);
}

// ---- bf16 GEMM with a deep load pipeline (M > 64).  Both operand tiles move
// HBM -> LDS by direct-to-LDS buffer loads (no register staging) into a ring
// of NS stages, so that NS - 1 K slices are in flight while one is consumed:
// with one slice in flight a workgroup waits a whole memory round trip per
// slice.  Waits are explicit vmcnt counts and a bare s_barrier (a
// __syncthreads() fence would drain every outstanding load each slice).  A
// direct-to-LDS instruction writes 1 KB of LDS linearly (lane l at 16 l), so
// the bank swizzle is applied through the global addresses: LDS slot s of
// tile row r holds K chunk s ^ f(r).  Rows past M (or N) lie outside the
// buffer range and load as zero. ----------------------------------------------
template <int BM_, int BN_, int NW_, int BK_, int NS_ = 4, int WGM_ = 2>
struct DmaShape {
  static constexpr int BM = BM_, BN = BN_, NW = NW_, BK = BK_, NS = NS_;
  static constexpr int NT = 64 * NW;
  static constexpr int VEC = 8;                       // bf16 per 16-byte chunk
  static constexpr int CPR = BK / VEC;                // chunks per tile row: 8 (BK 64) or 4 (BK 32)
  static constexpr int RPI = 64 / CPR;                // tile rows per 1 KB load instruction
  static constexpr int WGM = WGM_, WGN = NW / WGM;    // wave grid WGM x WGN
  static constexpr int WM = BM / WGM, WN = BN / WGN;
  static constexpr int TM = WM / 16, TN = WN / 16;
  static constexpr int A_INS = BM / RPI, W_INS = BN / RPI;
  static constexpr int INS = (A_INS + W_INS) / NW;    // load instructions per wave per stage
  static constexpr int STAGE = (BM + BN) * BK;        // bf16 elements per stage
  static_assert((A_INS + W_INS) % NW == 0, "load instructions split evenly over the waves");
  static_assert(CPR == 8 || CPR == 4, "swizzle defined for 64- and 32-deep slices");
  static_assert(TN % 2 == 0, "epilogues pair n-subtiles 2t and 2t+1");
  // LDS slot of chunk c in row r (an involution: also the chunk held by slot c)
  static __device__ __forceinline__ int swz(int r, int c) {
    // 64-byte rows (32-deep slices): the row pairs of a 128-byte bank window share the permutation.
    // Measured on the batch-64 GEMMs: c ^ ((r >> 1) & 3) gives no bank conflicts; c ^ ((r >> 2) & 3),
    // c ^ (r & 3) and c ^ ((r >> 3) & 3) give four per LDS instruction (GateUp 67.6 vs 65.6 us).
    return CPR == 8 ? (c ^ ((r >> 1) & 7)) : (c ^ ((r >> 1) & 3));
  }
};

// s_waitcnt with vmcnt = N and the other counters not waited for
template <int N>
__device__ __forceinline__ void wait_vm() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

// wait until at most `later` (<= L) stages of INS loads each are outstanding
template <int INS, int L>
__device__ __forceinline__ void wait_later(int later) {
  if constexpr (L == 0) {
    wait_vm<0>();
  } else {
    if (later >= L) wait_vm<L * INS>();
    else wait_later<INS, L - 1>(later);
  }
}

typedef __attribute__((address_space(3))) char dma_lds_t;
typedef __attribute__((address_space(3))) const bf16x8 dma_lds_frag;

// One 1 KB direct-to-LDS load: 16 bytes per lane from base + byte offset
// `off` (zero past `bytes`) into LDS at dst + 16 * lane.
__device__ __forceinline__ void dma_load_1k(const void* base, unsigned bytes, unsigned off, dma_lds_t* dst) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(
      __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), 0, (int)bytes, 0x00020000), dst, 16, off, 0, 0, 0);
}

// Issue slice kt into its ring stage: this wave's share of the 1 KB
// direct-to-LDS instructions; lane (lr, ls) loads tile row j * RPI + lr, K
// chunk swz(row, ls), into LDS slot ls of that row.
template <typename S>
__device__ __forceinline__ void dma_issue(const GemmLaunch& g, char* ring, int wave, int lr, int ls, int m0, int n0,
                                          int kbeg, int kt) {
  const int K = g.K, k0 = kbeg + kt * S::BK;
  const unsigned a_bytes = (unsigned)((size_t)g.M * K * 2), w_bytes = (unsigned)((size_t)g.N * K * 2);
  dma_lds_t* st = (dma_lds_t*)ring + (kt % S::NS) * (S::STAGE * 2);
#pragma unroll
  for (int i = 0; i < S::INS; ++i) {
    const int j = wave + S::NW * i;  // instruction index within the stage (uniform)
    if (j < S::A_INS) {
      const int r = j * S::RPI + lr;
      dma_load_1k(g.A, a_bytes, (unsigned)(((size_t)(m0 + r) * K + k0 + S::swz(r, ls) * S::VEC) * 2), st + j * 1024);
    } else {
      const int jw = j - S::A_INS, r = jw * S::RPI + lr;
      dma_load_1k(g.W, w_bytes, (unsigned)(((size_t)(n0 + r) * K + k0 + S::swz(r, ls) * S::VEC) * 2),
                  st + S::BM * S::BK * 2 + jw * 1024);
    }
  }
}

template <typename S, EpiKind EPI>
__global__ __launch_bounds__(S::NT) void k_gemm_dma(GemmLaunch g) {
  typedef dma_lds_t lds_t;
  typedef dma_lds_frag lds_frag;
  using MF = Mfma<bf16>;
  __shared__ __attribute__((aligned(1024))) char ring[S::NS * S::STAGE * 2];
  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave / S::WGN, wn = wave % S::WGN;
  const int m0 = blockIdx.y * S::BM, n0 = blockIdx.x * S::BN;
  const int M = g.M, N = g.N, K = g.K;
  const int kper = K / g.splitk, kbeg = blockIdx.z * kper, nkt = kper / S::BK;
  const int lr = lane / S::CPR, ls = lane % S::CPR;
  f32x4 acc[S::TM][S::TN];
#pragma unroll
  for (int a = 0; a < S::TM; ++a)
#pragma unroll
    for (int b = 0; b < S::TN; ++b) acc[a][b] = f32x4{0.f, 0.f, 0.f, 0.f};
  const int fr = lane & 15, fc = lane >> 4;  // fragment row, 16-byte K chunk within a 32-deep step
  const int rbase = m0 + wm * S::WM + (lane >> 4) * 4;
  const int cbase = n0 + wn * S::WN + fr;
  // QKV: the rotation factors of every result pair, loaded before the K loop
  // where they fit in registers beside the accumulators (as many again: up to
  // 16 result tiles per wave at eight waves per workgroup, 8 at sixteen)
  constexpr bool PRE = EPI == EPI_QKV && S::TM * S::TN * S::NW <= 128;
  float2 rope[PRE ? S::TM : 1][PRE ? S::TN / 2 : 1][4];
  if constexpr (PRE) {
#pragma unroll
    for (int a = 0; a < S::TM; ++a)
#pragma unroll
      for (int b = 0; b < S::TN; b += 2)
#pragma unroll
        for (int i = 0; i < 4; ++i) rope[a][b / 2][i] = qkv_rope_factor(g.ep, M, N, rbase + a * 16 + i, cbase + b * 16);
  }

#pragma unroll
  for (int s = 0; s < S::NS - 1; ++s)
    if (s < nkt) dma_issue<S>(g, ring, wave, lr, ls, m0, n0, kbeg, s);
  for (int kt = 0; kt < nkt; ++kt) {
    // slice kt has landed once at most min(NS - 2, nkt - 1 - kt) later slices are pending
    wait_later<S::INS, S::NS - 2>(min(S::NS - 2, nkt - 1 - kt));
    __builtin_amdgcn_s_barrier();  // every wave's part of slice kt; slice kt - 1 fully consumed
    if (kt + S::NS - 1 < nkt) dma_issue<S>(g, ring, wave, lr, ls, m0, n0, kbeg, kt + S::NS - 1);
    const lds_t* As = (const lds_t*)ring + (kt % S::NS) * (S::STAGE * 2);
    const lds_t* Ws = As + S::BM * S::BK * 2;
#pragma unroll
    for (int kk = 0; kk < S::BK; kk += MF::KSUB) {
      const int c = kk / S::VEC + fc;
      MF::frag af[S::TM], bfr[S::TN];
#pragma unroll
      for (int a = 0; a < S::TM; ++a) {
        const int r = wm * S::WM + a * 16 + fr;
        af[a] = *(lds_frag*)(As + (r * S::BK + S::swz(r, c) * S::VEC) * 2);
      }
#pragma unroll
      for (int b = 0; b < S::TN; ++b) {
        const int r = wn * S::WN + b * 16 + fr;
        bfr[b] = *(lds_frag*)(Ws + (r * S::BK + S::swz(r, c) * S::VEC) * 2);
      }
#pragma unroll
      for (int a = 0; a < S::TM; ++a)
#pragma unroll
        for (int b = 0; b < S::TN; ++b) acc[a][b] = MF::run(af[a], bfr[b], acc[a][b]);
    }
  }

  float* out = g.ep.out_f32 ? g.ep.out_f32 + (size_t)blockIdx.z * M * N : nullptr;
#pragma unroll
  for (int a = 0; a < S::TM; ++a)
#pragma unroll
    for (int b = 0; b < S::TN; b += 2)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        if constexpr (PRE)
          epilogue_qkv_pre<bf16>(g.ep, M, N, rbase + a * 16 + i, cbase + b * 16, acc[a][b][i], acc[a][b + 1][i],
                                 rope[a][b / 2][i]);
        else
          epilogue_pair<bf16, EPI>(g.ep, out, M, N, rbase + a * 16 + i, cbase + b * 16, acc[a][b][i],
                                   acc[a][b + 1][i]);
      }
}

// Every ring runs at least two waves per SIMD: with one, a wave's LDS reads and its MFMAs take turns
// (batch 8: four waves on 128 x 128 tiles 14.23 ms per call, eight 13.51 ms; eight waves on 64 x 64 tiles
// 13.18 ms).
typedef DmaShape<128, 128, 8, 64> DmaMid;          // one slice: 32 KB; ring 128 KB; waves 2 x 4 of 64 x 32
typedef DmaShape<64, 64, 8, 64, 4, 4> DmaSmall;    // one slice: 16 KB; ring 64 KB (two workgroups per unit);
                                                   // waves 4 x 2 of 16 x 32
typedef DmaShape<128, 256, 16, 64, 3, 4> DmaWide;  // one slice: 48 KB; ring 144 KB; waves 4 x 4 of 32 x 64
                                                  // (batch 64 48.62 -> 45.89 ms against eight waves on
                                                  // four 32-deep slices)
typedef DmaShape<256, 256, 16, 64, 2, 4> DmaBig;   // one slice: 64 KB; ring 128 KB (double-buffered);
                                                   // waves 4 x 4 of 64 x 64 (batch 64: 48.28 -> 47.31 ms
                                                   // for sixteen waves against eight, 45.74 -> 44.50 ms
                                                   // for two 64-deep stages against four 32-deep ones)

template <typename S>
static hipError_t launch_dma(const GemmLaunch& g, hipStream_t s) {
  dim3 grid((g.N + S::BN - 1) / S::BN, (g.M + S::BM - 1) / S::BM, g.splitk);
  switch (g.epi) {
    case EPI_STORE_F32: JPI_LAUNCH((k_gemm_dma<S, EPI_STORE_F32>), grid, dim3(S::NT), 0, s, g.ev_start, g.ev_stop, g); break;
    case EPI_QKV: JPI_LAUNCH((k_gemm_dma<S, EPI_QKV>), grid, dim3(S::NT), 0, s, g.ev_start, g.ev_stop, g); break;
    case EPI_GEGLU: JPI_LAUNCH((k_gemm_dma<S, EPI_GEGLU>), grid, dim3(S::NT), 0, s, g.ev_start, g.ev_stop, g); break;
  }
  return hipGetLastError();
}

static bool gemm_pipe_enabled() {
  static const int on = [] {
    const char* e = getenv("JPI_GEMM_PIPE");
    return e && e[0] == '0' ? 0 : 1;
  }();
  return on != 0;
}

template <typename S>
static hipError_t launch_big(const GemmLaunch& g, hipStream_t s) {
  dim3 grid((g.N + S::BN - 1) / S::BN, (g.M + S::BM - 1) / S::BM, g.splitk);
  switch (g.epi) {
    case EPI_STORE_F32: JPI_LAUNCH((k_gemm_big<S, EPI_STORE_F32>), grid, dim3(512), 0, s, g.ev_start, g.ev_stop, g); break;
    case EPI_QKV: JPI_LAUNCH((k_gemm_big<S, EPI_QKV>), grid, dim3(512), 0, s, g.ev_start, g.ev_stop, g); break;
    case EPI_GEGLU: JPI_LAUNCH((k_gemm_big<S, EPI_GEGLU>), grid, dim3(512), 0, s, g.ev_start, g.ev_stop, g); break;
  }
  return hipGetLastError();
}

// ---- skinny GEMM for M <= 64 (weight streaming): a workgroup owns 32 output
// columns and one K slice; its 4 waves split the slice four ways.  Each wave
// issues its weight fragments (16 bytes per lane per 16x32 tile) and
// activation fragments straight from memory into registers, BATCH k-steps at
// a time, before the MFMAs.  The four partial tiles are summed in LDS in wave
// order. --------------------------------------------------------------------
template <typename T>
struct SkinnyShape {
  static constexpr int KSUB = Mfma<T>::KSUB;
  static constexpr int WAVES = 8;                        // K split inside the workgroup
  static constexpr int BATCH = sizeof(T) == 2 ? 4 : 16;  // k steps in flight per wave
};

template <typename T, EpiKind EPI>
__global__ __launch_bounds__(512) void k_gemm_skinny(GemmLaunch g) {
  using MF = Mfma<T>;
  using SS = SkinnyShape<T>;
  __shared__ f32x4 red[SS::WAVES][4][2][64];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int M = g.M, N = g.N, K = g.K;
  const int n0 = blockIdx.x * 32;
  const int kper = K / g.splitk;
  const int kw = kper / SS::WAVES;
  const int k0 = blockIdx.z * kper + wave * kw;
  const int nsub = kw / SS::KSUB;
  const T* A = reinterpret_cast<const T*>(g.A);
  const T* W = reinterpret_cast<const T*>(g.W);
  const int fr = lane & 15, fk = (lane >> 4) * MF::KPL;
  const T* wp0 = W + (size_t)min(n0 + fr, N - 1) * K + k0 + fk;
  const T* wp1 = W + (size_t)min(n0 + 16 + fr, N - 1) * K + k0 + fk;

  f32x4 acc[4][2];
#pragma unroll
  for (int a = 0; a < 4; ++a) acc[a][0] = acc[a][1] = f32x4{0.f, 0.f, 0.f, 0.f};

  for (int s0 = 0; s0 < nsub; s0 += SS::BATCH) {
    typename MF::frag wf[SS::BATCH][2], af[SS::BATCH][4];
#pragma unroll
    for (int c = 0; c < SS::BATCH; ++c) {
      if (s0 + c < nsub) {
        wf[c][0] = MF::load(wp0 + (s0 + c) * SS::KSUB);
        wf[c][1] = MF::load(wp1 + (s0 + c) * SS::KSUB);
      } else {
        wf[c][0] = wf[c][1] = typename MF::frag{};
      }
    }
#pragma unroll
    for (int c = 0; c < SS::BATCH; ++c)
#pragma unroll
      for (int a = 0; a < 4; ++a) {
        const int row = a * 16 + fr;
        af[c][a] = (s0 + c < nsub && row < M) ? MF::load(A + (size_t)row * K + k0 + (s0 + c) * SS::KSUB + fk)
                                              : typename MF::frag{};
      }
#pragma unroll
    for (int c = 0; c < SS::BATCH; ++c)
#pragma unroll
      for (int a = 0; a < 4; ++a) {
        acc[a][0] = MF::run(af[c][a], wf[c][0], acc[a][0]);
        acc[a][1] = MF::run(af[c][a], wf[c][1], acc[a][1]);
      }
  }
#pragma unroll
  for (int a = 0; a < 4; ++a) {
    red[wave][a][0][lane] = acc[a][0];
    red[wave][a][1][lane] = acc[a][1];
  }
  __syncthreads();
  if (wave >= 4) return;
  // wave w finishes m-subtile w, summing the K-split waves in order
  const int a = wave;
  f32x4 lo = red[0][a][0][lane], hi = red[0][a][1][lane];
#pragma unroll
  for (int v = 1; v < SS::WAVES; ++v) {
    lo += red[v][a][0][lane];
    hi += red[v][a][1][lane];
  }
  float* out = g.ep.out_f32 ? g.ep.out_f32 + (size_t)blockIdx.z * M * N : nullptr;
  const int rbase = a * 16 + (lane >> 4) * 4;
#pragma unroll
  for (int i = 0; i < 4; ++i) epilogue_pair<T, EPI>(g.ep, out, M, N, rbase + i, n0 + fr, lo[i], hi[i]);
}

static bool use_skinny(int M) { return M <= 64; }

int gemm_k_quantum(jpi_dtype dt, int M) {
  if (use_skinny(M))
    return SkinnyShape<bf16>::WAVES * (dt == JPI_BF16 ? SkinnyShape<bf16>::KSUB : SkinnyShape<float>::KSUB);
  return dt == JPI_BF16 ? GemmShape<bf16, 128, 128>::BK : GemmShape<float, 64, 64>::BK;
}

size_t gemm_tiles(jpi_dtype dt, int M, int N) {
  if (use_skinny(M)) return (size_t)((N + 31) / 32);
  const int BM = dt == JPI_BF16 ? 128 : 64, BN = BM;
  return (size_t)((N + BN - 1) / BN) * ((M + BM - 1) / BM);
}

int gemm_pick_splitk(jpi_dtype dt, int M, int N, int K, int n_cu) {
  const int q = gemm_k_quantum(dt, M);
  const size_t tiles = gemm_tiles(dt, M, N);
  int s = 1;
  while (s < 16 && tiles * s < (size_t)n_cu && K % (2 * s * q) == 0) s *= 2;
  return s;
}

template <typename T, int BM, int BN>
static hipError_t launch_gemm_t(const GemmLaunch& g, hipStream_t s) {
  dim3 grid((g.N + BN - 1) / BN, (g.M + BM - 1) / BM, g.splitk);
  switch (g.epi) {
    case EPI_STORE_F32:
      JPI_LAUNCH((k_gemm<T, BM, BN, EPI_STORE_F32>), grid, dim3(256), 0, s, g.ev_start, g.ev_stop, g);
      break;
    case EPI_QKV: JPI_LAUNCH((k_gemm<T, BM, BN, EPI_QKV>), grid, dim3(256), 0, s, g.ev_start, g.ev_stop, g); break;
    case EPI_GEGLU:
      JPI_LAUNCH((k_gemm<T, BM, BN, EPI_GEGLU>), grid, dim3(256), 0, s, g.ev_start, g.ev_stop, g);
      break;
  }
  return hipGetLastError();
}

template <typename T>
static hipError_t launch_skinny_t(const GemmLaunch& g, hipStream_t s) {
  dim3 grid((g.N + 31) / 32, 1, g.splitk), block(64 * SkinnyShape<T>::WAVES);
  switch (g.epi) {
    case EPI_STORE_F32:
      JPI_LAUNCH((k_gemm_skinny<T, EPI_STORE_F32>), grid, block, 0, s, g.ev_start, g.ev_stop, g);
      break;
    case EPI_QKV: JPI_LAUNCH((k_gemm_skinny<T, EPI_QKV>), grid, block, 0, s, g.ev_start, g.ev_stop, g); break;
    case EPI_GEGLU: JPI_LAUNCH((k_gemm_skinny<T, EPI_GEGLU>), grid, block, 0, s, g.ev_start, g.ev_stop, g); break;
  }
  return hipGetLastError();
}

hipError_t launch_gemm(jpi_dtype dt, const GemmLaunch& g, hipStream_t s) {
  if (g.splitk > 1 && g.epi != EPI_STORE_F32) return hipErrorInvalidValue;
  if (g.K % (g.splitk * gemm_k_quantum(dt, g.M)) != 0) return hipErrorInvalidValue;
  if (use_skinny(g.M)) {
    if (dt == JPI_BF16) return launch_skinny_t<bf16>(g, s);
    return launch_skinny_t<float>(g, s);
  }
  if (dt == JPI_BF16) {
    // 256 x 256 tiles when they alone cover the compute units, else 128 x 128
    // unless that leaves the grid short and the epilogue cannot be split over K
    const int n_cu = g.n_cu > 0 ? g.n_cu : 256;
    auto tiles = [&](int bm, int bn) { return ((g.M + bm - 1) / bm) * ((g.N + bn - 1) / bn) * g.splitk; };
    // the direct-to-LDS pipeline (one 128 KB ring per compute unit) wins where one
    // round of 128 x 128 tiles covers the chip and no more (measured: M = 400
    // GateUp 25.1 -> 19.6 us, Down 16.2 -> 13.4 us); with more tiles the
    // register-staged kernel's two workgroups per unit win, with fewer the
    // smaller tiles below
    if (gemm_pipe_enabled() && g.M <= 512 && tiles(128, 128) >= n_cu && tiles(128, 128) <= n_cu + n_cu / 4 &&
        (g.K / g.splitk) % DmaMid::BK == 0 && (size_t)g.N * g.K * 2 < (1u << 31))
      return launch_dma<DmaMid>(g, s);
    // fewer 128 x 128 tiles than units and no K split (QKV at M = 400: 80 tiles): 64 x 64 tiles on the
    // pipelined kernel, two workgroups per unit (measured 20.0 -> 12.7 us; on split-K shapes no gain)
    if (gemm_pipe_enabled() && g.M <= 512 && tiles(128, 128) < n_cu && g.splitk == 1 && g.K % DmaSmall::BK == 0 &&
        (size_t)g.N * g.K * 2 < (1u << 31))
      return launch_dma<DmaSmall>(g, s);
    // Larger M: 256 x 256 tiles on the direct-to-LDS ring (64-deep slices, double-buffered, sixteen
    // waves) when such tiles alone cover the units (GateUp at M = 3200: 71.5 us on the register-staged
    // k_gemm_big, 68.1 us on the first, eight-wave version of this ring), else one round of 128 x 256 ring
    // tiles (two 64-deep slices in flight, sixteen waves) when they fill at least three quarters of the
    // units (M = 3200, first eight-wave version: QKV 39.6 -> 38.1, split-K O-proj 29.0 -> 25.6 and Down
    // 48.6 -> 42.8 us against two register-staged 128 x 128 workgroups per unit; register-staged 128 x 256
    // tiles were slower than both)
    const bool fits = (size_t)g.N * g.K * 2 < (1u << 31) && (size_t)g.M * g.K * 2 < (1u << 31);
    auto kfits = [&](int bk) { return (g.K / g.splitk) % bk == 0; };
    if (fits && kfits(DmaBig::BK) && tiles(256, 256) >= n_cu) return launch_dma<DmaBig>(g, s);
    if (tiles(256, 256) >= n_cu) return launch_big<Big256>(g, s);
    if (fits && kfits(DmaWide::BK) && tiles(128, 256) <= n_cu && 4 * tiles(128, 256) >= 3 * n_cu)
      return launch_dma<DmaWide>(g, s);
    if (tiles(128, 128) >= n_cu || g.epi == EPI_STORE_F32) return launch_gemm_t<bf16, 128, 128>(g, s);
    // fewer 128 x 128 tiles than units, no K split, yet enough 64 x 64 tiles to fill them (VLM QKV at
    // M = 816, N = 2560: 520 tiles): the ring at two workgroups per unit (prefill 5.52 -> 5.38 ms)
    if (gemm_pipe_enabled() && fits && g.splitk == 1 && kfits(DmaSmall::BK) && tiles(64, 64) >= n_cu)
      return launch_dma<DmaSmall>(g, s);
    if (tiles(128, 64) >= n_cu) return launch_gemm_t<bf16, 128, 64>(g, s);
    return launch_gemm_t<bf16, 64, 64>(g, s);
  }
  return launch_gemm_t<float, 64, 64>(g, s);
}

// fixed-order sum of split-K slices: C[i] = sum_z P[z][i]
__global__ void k_sum_slices(const float* __restrict__ P, float* __restrict__ C, int S, size_t MN) {
  const size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x;
  if (i >= MN) return;
  float v = 0.f;
  for (int z = 0; z < S; ++z) v += P[z * MN + i];
  C[i] = v;
}

hipError_t launch_sum_slices(const float* P, float* C, int S, size_t MN, hipStream_t s) {
  hipLaunchKernelGGL(k_sum_slices, dim3((unsigned)((MN + 255) / 256)), dim3(256), 0, s, P, C, S, MN);
  return hipGetLastError();
}

// ===========================================================================
// Row kernels (one workgroup of 256 threads per activation row m).
//
// Each rollout's sequence is n_lead correction rows followed by `horizon`
// action rows (m = b * (n_lead + horizon) + r); the correction rows carry
// given tokens of the expert's width and produce no velocity.
// k_inproj_norm:  h = x W_in^T + b_in (action rows) or the correction token;
//                 y = adaRMSNorm(h; scale, shift)
// k_resid_norm:   h += gate * sum_z P[z][m];  y = adaRMSNorm(h; scale, shift)
//   FINAL variant (action rows only): v = adaRMSNorm(h; s_f, b_f) W_out^T + b_out
//                  and x[b][i] += dt * v for action rows i >= n_fixed
// adaRMSNorm(h) = h / sqrt(mean(h^2) + eps) * (1 + scale) + shift.
// ===========================================================================
constexpr int ROW_MAX_W = 4096;

__device__ __forceinline__ float row_rstd(const float* hs, int W, float eps, float* red) {
  float ss = 0.f;
  for (int k = threadIdx.x; k < W; k += 256) ss += hs[k] * hs[k];
  ss = block_sum_256(ss, red);
  return 1.0f / sqrtf(ss / (float)W + eps);
}

template <typename T>
__global__ __launch_bounds__(256) void k_inproj_norm(const float* __restrict__ x, const T* __restrict__ w_in,
                                                     const float* __restrict__ b_in, float* __restrict__ h,
                                                     const float* __restrict__ scale, const float* __restrict__ shift,
                                                     T* __restrict__ y, int W, int A, float eps,
                                                     const float* __restrict__ corr, int n_lead, int horizon,
                                                     int n_t0, int64_t t0_delta) {
  __shared__ float hs[ROW_MAX_W];
  __shared__ float xs[256];
  __shared__ float red[4];
  const int m = blockIdx.x, S = n_lead + horizon, b = m / S, i = m % S;
  if (i >= n_lead && i - n_lead < n_t0) {  // a committed row at t = 0: the t = 0 table row
    scale += t0_delta;
    shift += t0_delta;
  }
  if (i < n_lead) {
    const float* cr = corr + ((size_t)b * n_lead + i) * W;
    for (int n = threadIdx.x; n < W; n += 256) {
      const float v = cr[n];
      hs[n] = v;
      h[(size_t)m * W + n] = v;
    }
  } else {
    const float* xr = x + ((size_t)b * horizon + (i - n_lead)) * A;
    for (int a = threadIdx.x; a < A; a += 256) xs[a] = xr[a];
    __syncthreads();
    for (int n = threadIdx.x; n < W; n += 256) {
      float acc = 0.f;
      for (int a = 0; a < A; ++a) acc = fmaf(xs[a], static_cast<float>(w_in[(size_t)n * A + a]), acc);
      const float v = acc + b_in[n];
      hs[n] = v;
      h[(size_t)m * W + n] = v;
    }
  }
  __syncthreads();
  const float r = row_rstd(hs, W, eps, red);
  for (int k = threadIdx.x; k < W; k += 256)
    y[(size_t)m * W + k] = from_f32<T>(hs[k] * r * (1.0f + scale[k]) + shift[k]);
}

constexpr int ROW_MAX_S = 16;
constexpr int ROW_MAX_A = 64;

// four consecutive elements as floats (8- or 16-byte aligned)
__device__ __forceinline__ void load4(const float* p, float (&w)[4]) {
  const f32x4 v = *reinterpret_cast<const f32x4*>(p);
  w[0] = v[0];
  w[1] = v[1];
  w[2] = v[2];
  w[3] = v[3];
}
__device__ __forceinline__ void load4(const bf16* p, float (&w)[4]) {
  const uint2 v = *reinterpret_cast<const uint2*>(p);
  w[0] = __uint_as_float(v.x << 16);
  w[1] = __uint_as_float(v.x & 0xffff0000u);
  w[2] = __uint_as_float(v.y << 16);
  w[3] = __uint_as_float(v.y & 0xffff0000u);
}

template <typename T, bool FINAL>
__global__ __launch_bounds__(256) void k_resid_norm(RowLaunch r) {
  __shared__ float hs[ROW_MAX_W];
  __shared__ float red[4];
  __shared__ float dots[4][ROW_MAX_A];
  const int m = blockIdx.x, W = r.W, S = r.S;
  const size_t MW = (size_t)r.M * W;
  // the last layer's correction rows feed nothing (the next step restarts them)
  if constexpr (FINAL) {
    if (m % (r.n_lead + r.horizon) < r.n_lead) return;
  }
  // committed rows at t = 0 take the gate, scale and shift of the t = 0 table row
  const float *gate = r.gate, *scale = r.scale, *shift = r.shift;
  if (r.n_t0 > 0) {
    const int ia = m % (r.n_lead + r.horizon) - r.n_lead;
    if (ia >= 0 && ia < r.n_t0) {
      gate += r.t0_delta;
      scale += r.t0_delta;
      shift += r.t0_delta;
    }
  }
  float* hr = r.h + (size_t)m * W;
  const float* pr = r.part + (size_t)m * W;
  // four columns per thread per pass; all split-K slices loaded before summing
  for (int k0 = threadIdx.x; k0 < W; k0 += 1024) {
    float v[4][ROW_MAX_S], hv[4], gv[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int k = k0 + 256 * j;
#pragma unroll
      for (int z = 0; z < ROW_MAX_S; ++z) v[j][z] = (z < S && k < W) ? pr[z * MW + k] : 0.f;
      hv[j] = k < W ? hr[k] : 0.f;
      gv[j] = k < W ? gate[k] : 0.f;
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int k = k0 + 256 * j;
      float sum = 0.f;
#pragma unroll
      for (int z = 0; z < ROW_MAX_S; ++z)
        if (z < S) sum += v[j][z];
      if (k < W) {
        const float h2 = hv[j] + gv[j] * sum;
        hr[k] = h2;
        hs[k] = h2;
      }
    }
  }
  __syncthreads();
  const float rs = row_rstd(hs, W, r.eps, red);
  if constexpr (!FINAL) {
    T* yr = reinterpret_cast<T*>(r.y) + (size_t)m * W;
    for (int k = threadIdx.x; k < W; k += 256) yr[k] = from_f32<T>(hs[k] * rs * (1.0f + scale[k]) + shift[k]);
  } else {
    // v[a] = sum_k y[k] W_out[a][k] + b_out[a]; thread t owns columns 4t + 1024 j .. + 3,
    // so each row of W_out is read with one 4-element load per thread, all independent
    constexpr int NJ = ROW_MAX_W / 1024;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const T* wo = reinterpret_cast<const T*>(r.w_out);
    float yk[NJ][4];
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
      const int k = 4 * threadIdx.x + 1024 * j;
#pragma unroll
      for (int e = 0; e < 4; ++e)
        yk[j][e] = k < W ? hs[k + e] * rs * (1.0f + scale[k + e]) + shift[k + e] : 0.f;
    }
    for (int a0 = 0; a0 < r.A; a0 += 8) {
      float p[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        p[u] = 0.f;
#pragma unroll
        for (int j = 0; j < NJ; ++j) {
          const int k = 4 * threadIdx.x + 1024 * j;
          if (a0 + u < r.A && k < W) {
            float w4[4];
            load4(wo + (size_t)(a0 + u) * W + k, w4);
#pragma unroll
            for (int e = 0; e < 4; ++e) p[u] = fmaf(yk[j][e], w4[e], p[u]);
          }
        }
      }
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const float t = wave_sum(p[u]);
        if (lane == 0 && a0 + u < r.A) dots[wave][a0 + u] = t;
      }
    }
    __syncthreads();
    const int seq = r.n_lead + r.horizon, b = m / seq, i = m % seq - r.n_lead;
    if (threadIdx.x < r.A && i >= r.n_fixed) {
      const int a = threadIdx.x;
      const float v = ((dots[0][a] + dots[1][a]) + dots[2][a]) + dots[3][a] + r.b_out[a];
      r.x[((size_t)b * r.horizon + i) * r.A + a] += r.dt * v;
    }
  }
}

// Non-final residual + norm, one workgroup per row: thread t owns columns
// 4t + 1024 j .. + 3; the slices, the residual and the gate, scale and shift
// are all loaded before the row reduction, and the row stays in registers.
template <typename T>
__global__ __launch_bounds__(256) void k_resid_norm_row(RowLaunch r) {
  constexpr int NJ = ROW_MAX_W / 1024;
  __shared__ float red[4];
  const int m = blockIdx.x, W = r.W, S = r.S;
  const size_t MW = (size_t)r.M * W;
  const float *gate = r.gate, *scale = r.scale, *shift = r.shift;
  if (r.n_t0 > 0) {  // committed rows at t = 0: the t = 0 table row
    const int ia = m % (r.n_lead + r.horizon) - r.n_lead;
    if (ia >= 0 && ia < r.n_t0) {
      gate += r.t0_delta;
      scale += r.t0_delta;
      shift += r.t0_delta;
    }
  }
  float* hr = r.h + (size_t)m * W;
  const float* pr = r.part + (size_t)m * W;
  f32x4 hv[NJ], sc[NJ], sh[NJ];
  float ss = 0.f;
#pragma unroll
  for (int j = 0; j < NJ; ++j) {
    const int k = 4 * threadIdx.x + 1024 * j;
    if (k >= W) break;
    f32x4 v[ROW_MAX_S];
#pragma unroll
    for (int z = 0; z < ROW_MAX_S; ++z)
      v[z] = z < S ? *reinterpret_cast<const f32x4*>(pr + z * MW + k) : f32x4{0.f, 0.f, 0.f, 0.f};
    const f32x4 h = *reinterpret_cast<const f32x4*>(hr + k), g4 = *reinterpret_cast<const f32x4*>(gate + k);
    sc[j] = *reinterpret_cast<const f32x4*>(scale + k);
    sh[j] = *reinterpret_cast<const f32x4*>(shift + k);
    f32x4 sum = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int z = 0; z < ROW_MAX_S; ++z)
      if (z < S) sum += v[z];
    const f32x4 h2 = h + g4 * sum;
    *reinterpret_cast<f32x4*>(hr + k) = h2;
    hv[j] = h2;
    ss += h2[0] * h2[0] + h2[1] * h2[1] + h2[2] * h2[2] + h2[3] * h2[3];
  }
  const float rs = 1.0f / sqrtf(block_sum_256(ss, red) / (float)W + r.eps);
  T* yr = reinterpret_cast<T*>(r.y) + (size_t)m * W;
#pragma unroll
  for (int j = 0; j < NJ; ++j) {
    const int k = 4 * threadIdx.x + 1024 * j;
    if (k >= W) break;
#pragma unroll
    for (int e = 0; e < 4; ++e) yr[k + e] = from_f32<T>(hv[j][e] * rs * (1.0f + sc[j][e]) + sh[j][e]);
  }
}

// Non-final residual + norm with one wave per row (four rows per workgroup):
// the row's sum of squares is a wave reduction, so no workgroup barrier.
// Same per-element arithmetic as k_resid_norm (slices summed in order).
template <typename T, int NJ>
__global__ __launch_bounds__(256) void k_resid_norm_wave(RowLaunch r) {
  // A wave per row, W <= 256 NJ.  Every load of the row (up to RW_SLICES
  // split-K slices, the residual and the gate) is issued before any
  // arithmetic or store: written pass by pass, with the slice count and the
  // row end as runtime loop bounds, each 256-column pass waited a memory
  // round trip for the previous one.  y leaves as 4 packed values per lane.
  constexpr int RW_SLICES = 4;
  const int lane = threadIdx.x & 63, m = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (m >= r.M) return;
  const int W = r.W, S = r.S;
  const size_t MW = (size_t)r.M * W;
  const float* __restrict__ gate = r.gate;
  const float* __restrict__ scale = r.scale;
  const float* __restrict__ shift = r.shift;
  if (r.n_t0 > 0) {  // committed rows at t = 0: the t = 0 table row
    const int ia = m % (r.n_lead + r.horizon) - r.n_lead;
    if (ia >= 0 && ia < r.n_t0) {
      gate += r.t0_delta;
      scale += r.t0_delta;
      shift += r.t0_delta;
    }
  }
  float* __restrict__ hr = r.h + (size_t)m * W;
  const float* __restrict__ pr = r.part + (size_t)m * W;
  // columns past W read column 0 (in range) and are then ignored
  int kk[NJ];
#pragma unroll
  for (int j = 0; j < NJ; ++j) kk[j] = 4 * lane + 256 * j < W ? 4 * lane + 256 * j : 0;
  f32x4 pv[RW_SLICES][NJ], hv[NJ], gv[NJ];
#pragma unroll
  for (int z = 0; z < RW_SLICES; ++z)
#pragma unroll
    for (int j = 0; j < NJ; ++j)
      pv[z][j] = z < S ? *reinterpret_cast<const f32x4*>(pr + z * MW + kk[j]) : f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int j = 0; j < NJ; ++j) {
    hv[j] = *reinterpret_cast<const f32x4*>(hr + kk[j]);
    gv[j] = *reinterpret_cast<const f32x4*>(gate + kk[j]);
  }
  float ss = 0.f;
#pragma unroll
  for (int j = 0; j < NJ; ++j) {
    f32x4 sum = pv[0][j];
#pragma unroll
    for (int z = 1; z < RW_SLICES; ++z) sum += pv[z][j];  // zero past S: the same sum in the same order
    for (int z = RW_SLICES; z < S; ++z) sum += *reinterpret_cast<const f32x4*>(pr + z * MW + kk[j]);
    hv[j] += gv[j] * sum;
    if (4 * lane + 256 * j < W) ss += hv[j][0] * hv[j][0] + hv[j][1] * hv[j][1] + hv[j][2] * hv[j][2] + hv[j][3] * hv[j][3];
  }
#pragma unroll
  for (int j = 0; j < NJ; ++j)
    if (4 * lane + 256 * j < W) *reinterpret_cast<f32x4*>(hr + kk[j]) = hv[j];
  const float rs = 1.0f / sqrtf(wave_sum(ss) / (float)W + r.eps);
  T* __restrict__ yr = reinterpret_cast<T*>(r.y) + (size_t)m * W;
#pragma unroll
  for (int j = 0; j < NJ; ++j) {
    if (4 * lane + 256 * j >= W) continue;
    const int k = kk[j];
    const f32x4 sc = *reinterpret_cast<const f32x4*>(scale + k), sh = *reinterpret_cast<const f32x4*>(shift + k);
    T v4[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) v4[e] = from_f32<T>(hv[j][e] * rs * (1.0f + sc[e]) + sh[e]);
    if constexpr (sizeof(T) == 2) {
      typedef T t4 __attribute__((ext_vector_type(4)));
      *reinterpret_cast<t4*>(yr + k) = t4{v4[0], v4[1], v4[2], v4[3]};
    } else {
      *reinterpret_cast<f32x4*>(yr + k) = f32x4{v4[0], v4[1], v4[2], v4[3]};
    }
  }
}

hipError_t launch_inproj_norm(jpi_dtype dt, const float* x, const void* w_in, const float* b_in, float* h,
                              const float* scale, const float* shift, void* y, int M, int W, int A, float eps,
                              const float* corr, int n_lead, int horizon, int n_t0, int64_t t0_delta,
                              hipStream_t s) {
  if (W > ROW_MAX_W || A > 256 || horizon < 1 || n_lead < 0 || (n_lead > 0 && !corr) || M % (n_lead + horizon))
    return hipErrorInvalidValue;
  if (dt == JPI_BF16)
    hipLaunchKernelGGL(k_inproj_norm<bf16>, dim3(M), dim3(256), 0, s, x, (const bf16*)w_in, b_in, h, scale, shift,
                       (bf16*)y, W, A, eps, corr, n_lead, horizon, n_t0, t0_delta);
  else
    hipLaunchKernelGGL(k_inproj_norm<float>, dim3(M), dim3(256), 0, s, x, (const float*)w_in, b_in, h, scale, shift,
                       (float*)y, W, A, eps, corr, n_lead, horizon, n_t0, t0_delta);
  return hipGetLastError();
}

hipError_t launch_resid_norm(jpi_dtype dt, const RowLaunch& r, bool final_step, hipStream_t s) {
  if (r.W > ROW_MAX_W || r.S > ROW_MAX_S || r.S < 1) return hipErrorInvalidValue;
  if (final_step && (r.A > ROW_MAX_A || r.horizon < 1 || r.n_lead < 0 || r.M % (r.n_lead + r.horizon)))
    return hipErrorInvalidValue;
  // a wave per row pays off only with many rows (batch 64: 23 -> 12 us); with
  // fewer rows a workgroup per row keeps more loads in flight
  if (!final_step && r.W % 4 != 0) return hipErrorInvalidValue;
  const bool wave_rows = !final_step && r.M >= 2048;
  const dim3 wave_grid((r.M + 3) / 4);
  if (dt == JPI_BF16) {
    if (final_step) hipLaunchKernelGGL((k_resid_norm<bf16, true>), dim3(r.M), dim3(256), 0, s, r);
    else if (wave_rows && r.W <= 1024) hipLaunchKernelGGL((k_resid_norm_wave<bf16, 4>), wave_grid, dim3(256), 0, s, r);
    else if (wave_rows && r.W <= 2048) hipLaunchKernelGGL((k_resid_norm_wave<bf16, 8>), wave_grid, dim3(256), 0, s, r);
    else if (wave_rows) hipLaunchKernelGGL((k_resid_norm_wave<bf16, 16>), wave_grid, dim3(256), 0, s, r);
    else hipLaunchKernelGGL(k_resid_norm_row<bf16>, dim3(r.M), dim3(256), 0, s, r);
  } else {
    if (final_step) hipLaunchKernelGGL((k_resid_norm<float, true>), dim3(r.M), dim3(256), 0, s, r);
    else if (wave_rows && r.W <= 1024) hipLaunchKernelGGL((k_resid_norm_wave<float, 4>), wave_grid, dim3(256), 0, s, r);
    else if (wave_rows && r.W <= 2048) hipLaunchKernelGGL((k_resid_norm_wave<float, 8>), wave_grid, dim3(256), 0, s, r);
    else if (wave_rows) hipLaunchKernelGGL((k_resid_norm_wave<float, 16>), wave_grid, dim3(256), 0, s, r);
    else hipLaunchKernelGGL(k_resid_norm_row<float>, dim3(r.M), dim3(256), 0, s, r);
  }
  return hipGetLastError();
}

// ===========================================================================
// prefix + self attention, one shared KV head (Appendix: queries from the
// action tokens, keys/values = LLM layer KV ++ action tokens' own KV).
// The concatenated key sequence [prefix 0..pl-1 | action 0..H-1] is cut into
// chunks of KC keys; a workgroup handles one (rollout, head, 64-query block,
// chunk) and writes the chunk's running max, sum and unnormalised output.
// K is read row-major ([key][Dh]); V is read transposed ([Dh][key]) so that
// the P.V operand streams along keys.  Slots j >= pl of the prefix are never
// used: a 16-byte V chunk that reaches past pl is assembled element by
// element with the out-of-range keys set to zero.
// ===========================================================================
template <typename T>
struct AttnShape {
  static constexpr int KC = sizeof(T) == 2 ? 64 : 32;
  static constexpr int PAD = 16 / sizeof(T);
  static constexpr int MAX_CHUNKS = 512;
};

template <typename T, int DH>
__global__ __launch_bounds__(256) void k_attn_partial(AttnLaunch a) {
  using MF = Mfma<T>;
  constexpr int KC = AttnShape<T>::KC, PAD = AttnShape<T>::PAD;
  constexpr int LDK = DH + PAD, LDV = KC + PAD, LDP = KC + PAD;
  constexpr int NST = DH / MF::KSUB;  // k steps over the head dim
  constexpr int NJ = KC / 16;         // key subtiles
  constexpr int VEC = 16 / sizeof(T);
  constexpr int KCH = KC * (DH / VEC) / 256;  // 16-byte K chunks per thread
  constexpr int VCH = DH * (KC / VEC) / 256;  // 16-byte V^T chunks per thread
  static_assert(KCH >= 1 && VCH >= 1, "tile too small");
  __shared__ __attribute__((aligned(16))) T Ks[KC * LDK];
  __shared__ __attribute__((aligned(16))) T Vt[DH * LDV];
  __shared__ __attribute__((aligned(16))) T Ps[64 * LDP];

  const int c = blockIdx.x;
  const int hn = blockIdx.y % a.nH, qb = blockIdx.y / a.nH;
  const int b = blockIdx.z;
  const int H = a.H;
  const int pl = a.prefix_len[b];
  const int nkeys = pl + H;
  const int nch = gridDim.x;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const size_t slot = (size_t)(b * a.nH + hn) * nch + c;
  float* Op = a.opart + slot * H * DH;
  float* Mp = a.mpart + slot * H;
  float* Lp = a.lpart + slot * H;
  const int kbase = c * KC;

  if (kbase >= nkeys) {  // chunk past this rollout's keys
    for (int r = tid; r < 64; r += 256) {
      const int i = qb * 64 + r;
      if (i < H) {
        Mp[i] = -INFINITY;
        Lp[i] = 0.f;
      }
    }
    for (int e = tid; e < 64 * DH; e += 256) {
      const int r = e / DH, d = e - r * DH, i = qb * 64 + r;
      if (i < H) Op[(size_t)i * DH + d] = 0.f;
    }
    return;
  }

  const T* kp = reinterpret_cast<const T*>(a.kp) + (size_t)b * a.kp_bstride;
  const T* vpt = reinterpret_cast<const T*>(a.vpt) + (size_t)b * a.vpt_bstride;
  const T* ksb = reinterpret_cast<const T*>(a.ks) + (size_t)b * (a.ks_bstride ? a.ks_bstride : (int64_t)H * DH);
  const T* vstb = reinterpret_cast<const T*>(a.vst) + (size_t)b * DH * a.vst_ld;

  // issue every global load of the chunk before the first LDS store
  uint4 kr[KCH], vr[VCH];
#pragma unroll
  for (int it = 0; it < KCH; ++it) {
    const int e = tid + it * 256, r = e / (DH / VEC), cc = e - r * (DH / VEC);
    const int key = kbase + r;
    const T* src = key < pl ? kp + (size_t)key * DH : ksb + (size_t)(key - pl) * DH;
    kr[it] = key < nkeys ? *reinterpret_cast<const uint4*>(src + cc * VEC) : make_uint4(0, 0, 0, 0);
  }
#pragma unroll
  for (int it = 0; it < VCH; ++it) {
    const int e = tid + it * 256, d = e / (KC / VEC), kc = e - d * (KC / VEC);
    const int key0 = kbase + kc * VEC;
    if (key0 + VEC <= pl) {
      vr[it] = *reinterpret_cast<const uint4*>(vpt + (size_t)d * a.vpt_dstride + key0);
    } else {
      T tmp[VEC];
#pragma unroll
      for (int j = 0; j < VEC; ++j) {
        const int key = key0 + j;
        tmp[j] = key < pl ? vpt[(size_t)d * a.vpt_dstride + key]
                          : (key < nkeys ? vstb[(size_t)d * a.vst_ld + (key - pl)] : from_f32<T>(0.f));
      }
      __builtin_memcpy(&vr[it], tmp, 16);
    }
  }
  // query fragments of this wave's 16 rows, kept in registers
  const int fr = lane & 15, fk = (lane >> 4) * MF::KPL;
  const int iq = qb * 64 + w * 16 + fr;
  typename MF::frag qf[NST];
  {
    const T* qrow = reinterpret_cast<const T*>(a.q) + (((size_t)b * a.nH + hn) * H + (iq < H ? iq : 0)) * DH;
#pragma unroll
    for (int st = 0; st < NST; ++st) qf[st] = iq < H ? MF::load(qrow + st * MF::KSUB + fk) : typename MF::frag{};
  }
#pragma unroll
  for (int it = 0; it < KCH; ++it) {
    const int e = tid + it * 256, r = e / (DH / VEC), cc = e - r * (DH / VEC);
    *reinterpret_cast<uint4*>(&Ks[r * LDK + cc * VEC]) = kr[it];
  }
#pragma unroll
  for (int it = 0; it < VCH; ++it) {
    const int e = tid + it * 256, d = e / (KC / VEC), kc = e - d * (KC / VEC);
    *reinterpret_cast<uint4*>(&Vt[d * LDV + kc * VEC]) = vr[it];
  }
  __syncthreads();

  f32x4 sc[NJ];
#pragma unroll
  for (int j = 0; j < NJ; ++j) sc[j] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int st = 0; st < NST; ++st)
#pragma unroll
    for (int j = 0; j < NJ; ++j)
      sc[j] = MF::run(qf[st], MF::load(&Ks[(j * 16 + fr) * LDK + st * MF::KSUB + fk]), sc[j]);

  const float scale = 1.0f / sqrtf((float)DH);
  float mrow[4], lrow[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    float mx = -INFINITY;
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
      const int key = kbase + j * 16 + fr;
      const float v = key < nkeys ? sc[j][e] * scale : -INFINITY;
      sc[j][e] = v;
      mx = fmaxf(mx, v);
    }
    mx = group16_max(mx);
    float sum = 0.f;
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
      const float p = mx == -INFINITY ? 0.f : expf(sc[j][e] - mx);
      sc[j][e] = p;
      sum += p;
    }
    mrow[e] = mx;
    lrow[e] = group16_sum(sum);
  }
  const int prow = w * 16 + (lane >> 4) * 4;
#pragma unroll
  for (int j = 0; j < NJ; ++j)
#pragma unroll
    for (int e = 0; e < 4; ++e) Ps[(prow + e) * LDP + j * 16 + fr] = from_f32<T>(sc[j][e]);
  __syncthreads();

  f32x4 o[DH / 16];
#pragma unroll
  for (int nt = 0; nt < DH / 16; ++nt) o[nt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int st = 0; st < KC / MF::KSUB; ++st) {
    const typename MF::frag pa = MF::load(&Ps[(w * 16 + fr) * LDP + st * MF::KSUB + fk]);
#pragma unroll
    for (int nt = 0; nt < DH / 16; ++nt)
      o[nt] = MF::run(pa, MF::load(&Vt[(nt * 16 + fr) * LDV + st * MF::KSUB + fk]), o[nt]);
  }
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const int i = qb * 64 + prow + e;
    if (i < H) {
#pragma unroll
      for (int nt = 0; nt < DH / 16; ++nt) Op[(size_t)i * DH + nt * 16 + fr] = o[nt][e];
      if (fr == 0) {
        Mp[i] = mrow[e];
        Lp[i] = lrow[e];
      }
    }
  }
}

// out[(b*H + i)][hn*Dh + d] = sum_c e^(m_c - m) O_c[d] / sum_c e^(m_c - m) l_c
template <typename TO, int DH>
__global__ __launch_bounds__(256) void k_attn_combine(AttnLaunch a, int nch) {
  __shared__ float wts[AttnShape<float>::MAX_CHUNKS];
  __shared__ float inv_l;
  const int H = a.H;
  const int i = blockIdx.x % H, bh = blockIdx.x / H;
  const int b = bh / a.nH, hn = bh - b * a.nH;
  const float* Mp = a.mpart + (size_t)bh * nch * H;
  const float* Lp = a.lpart + (size_t)bh * nch * H;
  const float* Op = a.opart + (size_t)bh * nch * H * DH;
  if (threadIdx.x < 64) {
    const int lane = threadIdx.x;
    float mx = -INFINITY;
    for (int c = lane; c < nch; c += 64) mx = fmaxf(mx, Mp[c * H + i]);
    mx = wave_max(mx);
    float l = 0.f;
    for (int c = lane; c < nch; c += 64) {
      const float mc = Mp[c * H + i];
      const float wc = mc == -INFINITY ? 0.f : expf(mc - mx);
      wts[c] = wc;
      l += wc * Lp[c * H + i];
    }
    l = wave_sum(l);
    if (lane == 0) inv_l = 1.0f / l;
  }
  __syncthreads();
  TO* out = reinterpret_cast<TO*>(a.out) + ((size_t)b * H + i) * a.nH * DH + hn * DH;
  for (int d = threadIdx.x; d < DH; d += blockDim.x) {
    float acc = 0.f;
    for (int c0 = 0; c0 < nch; c0 += 8) {
      float v[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) v[u] = c0 + u < nch ? Op[((size_t)(c0 + u) * H + i) * DH + d] : 0.f;
#pragma unroll
      for (int u = 0; u < 8; ++u)
        if (c0 + u < nch) acc += wts[c0 + u] * v[u];
    }
    out[d] = from_f32<TO>(acc * inv_l);
  }
}

int attn_chunk(jpi_dtype dt) { return dt == JPI_BF16 ? AttnShape<bf16>::KC : AttnShape<float>::KC; }
int attn_n_chunks(jpi_dtype dt, int P, int H) {
  const int kc = attn_chunk(dt);
  return (P + H + kc - 1) / kc;
}
int attn_max_prefix(jpi_dtype dt, int H) { return AttnShape<float>::MAX_CHUNKS * attn_chunk(dt) - H; }

template <typename T, int DH>
static hipError_t launch_attention_t(const AttnLaunch& a, hipStream_t s) {
  const int nch = attn_n_chunks(sizeof(T) == 2 ? JPI_BF16 : JPI_F32, a.P, a.H);
  if (nch > AttnShape<float>::MAX_CHUNKS) return hipErrorInvalidValue;
  const int nqb = (a.H + 63) / 64;
  JPI_LAUNCH((k_attn_partial<T, DH>), dim3(nch, a.nH * nqb, a.B), dim3(256), 0, s, a.ev_start, (hipEvent_t) nullptr,
             a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int thr = DH < 256 ? DH : 256;
  if (a.out_f32)
    JPI_LAUNCH((k_attn_combine<float, DH>), dim3(a.B * a.nH * a.H), dim3(thr), 0, s, (hipEvent_t) nullptr,
               a.ev_stop, a, nch);
  else
    JPI_LAUNCH((k_attn_combine<T, DH>), dim3(a.B * a.nH * a.H), dim3(thr), 0, s, (hipEvent_t) nullptr, a.ev_stop, a,
               nch);
  return hipGetLastError();
}

hipError_t launch_attention(jpi_dtype dt, const AttnLaunch& a, hipStream_t s) {
  if (dt == JPI_BF16) {
    // key ranges are bounded by the chunk count the opart scratch is sized for
    const int nch = attn_n_chunks(dt, a.P, a.H);
    int S = flash_splits(a.B, a.nH, a.H, a.P, a.n_cu > 0 ? a.n_cu : 256);
    S = S < nch ? S : nch;
    return launch_flash(a, S, s);
  } else {
    switch (a.Dh) {
      case 64: return launch_attention_t<float, 64>(a, s);
      case 128: return launch_attention_t<float, 128>(a, s);
      case 256: return launch_attention_t<float, 256>(a, s);
    }
  }
  return hipErrorInvalidValue;
}

// dst[z][c][r] = src[z][r][c] for r < rows, c < cols; 64 x 64 tiles through LDS.
// src row stride `sld`, dst row stride `dld`, matrix strides sz / dz (elements).
template <typename T>
__global__ __launch_bounds__(256) void k_transpose(const T* __restrict__ src, T* __restrict__ dst, int rows,
                                                   int cols, int64_t sld, int64_t dld, int64_t sz, int64_t dz) {
  __shared__ T tile[64][65];
  const int r0 = blockIdx.x * 64, c0 = blockIdx.y * 64;
  const T* s = src + blockIdx.z * sz;
  T* d = dst + blockIdx.z * dz;
  for (int e = threadIdx.x; e < 64 * 64; e += 256) {
    const int r = e / 64, c = e % 64;
    if (r0 + r < rows && c0 + c < cols) tile[r][c] = s[(size_t)(r0 + r) * sld + c0 + c];
  }
  __syncthreads();
  for (int e = threadIdx.x; e < 64 * 64; e += 256) {
    const int c = e / 64, r = e % 64;
    if (r0 + r < rows && c0 + c < cols) d[(size_t)(c0 + c) * dld + r0 + r] = tile[r][c];
  }
}

hipError_t launch_transpose(jpi_dtype dt, const void* src, void* dst, int rows, int cols, int64_t sld, int64_t dld,
                            int64_t sz, int64_t dz, int nmat, hipStream_t s) {
  if (rows == 0 || cols == 0 || nmat == 0) return hipSuccess;
  dim3 grid((rows + 63) / 64, (cols + 63) / 64, nmat);
  if (dt == JPI_BF16)
    hipLaunchKernelGGL(k_transpose<bf16>, grid, dim3(256), 0, s, (const bf16*)src, (bf16*)dst, rows, cols, sld, dld,
                       sz, dz);
  else
    hipLaunchKernelGGL(k_transpose<float>, grid, dim3(256), 0, s, (const float*)src, (float*)dst, rows, cols, sld,
                       dld, sz, dz);
  return hipGetLastError();
}

// ===========================================================================
// once per (weights, n_steps): timestep embedding, time MLP and the
// modulation table.  fp64 arithmetic; results stored in fp32.
// ===========================================================================
// rows k = 0 .. rows-1 at t = 1 - k/n (row n, when present, is t = 0)
__global__ void k_time_embed(float* emb, int rows, int n, int W) {
  const int idx = blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= rows * W) return;
  const int k = idx / W, j = idx - k * W, half = W / 2;
  const int jj = j < half ? j : j - half;
  const double t = 1.0 - (double)k / (double)n;
  const double f = exp(-log(1.0e4) * (double)jj / (double)half);
  const double arg = 1000.0 * t * f;
  emb[idx] = (float)(j < half ? cos(arg) : sin(arg));
}

hipError_t launch_time_embed(float* emb, int rows, int n, int W, hipStream_t s) {
  hipLaunchKernelGGL(k_time_embed, dim3((rows * W + 255) / 256), dim3(256), 0, s, emb, rows, n, W);
  return hipGetLastError();
}

template <typename T>
__global__ __launch_bounds__(256) void k_rowdot(const float* __restrict__ in, const T* __restrict__ w,
                                                const float* __restrict__ b, float* __restrict__ out, int M, int N,
                                                int K, int act) {
  const int lane = threadIdx.x & 63;
  const int n = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (n >= N) return;
  const T* wr = w + (size_t)n * K;
  for (int m0 = 0; m0 < M; m0 += 8) {
    double acc[8];
#pragma unroll
    for (int r = 0; r < 8; ++r) acc[r] = 0.0;
    for (int k = lane; k < K; k += 64) {
      const double wv = (double)static_cast<float>(wr[k]);
#pragma unroll
      for (int r = 0; r < 8; ++r)
        if (m0 + r < M) acc[r] += wv * (double)in[(size_t)(m0 + r) * K + k];
    }
#pragma unroll
    for (int r = 0; r < 8; ++r) acc[r] = wave_sum_d(acc[r]);
    if (lane == 0) {
#pragma unroll
      for (int r = 0; r < 8; ++r) {
        if (m0 + r < M) {
          double v = acc[r] + (double)b[n];
          if (act == 1) v = v / (1.0 + exp(-v));
          out[(size_t)(m0 + r) * N + n] = (float)v;
        }
      }
    }
  }
}

hipError_t launch_rowdot(jpi_dtype dt, const float* in, const void* w, const float* b, float* out, int M, int N,
                         int K, int act, hipStream_t s) {
  const int blocks = (N + 3) / 4;
  if (dt == JPI_BF16)
    hipLaunchKernelGGL(k_rowdot<bf16>, dim3(blocks), dim3(256), 0, s, in, (const bf16*)w, b, out, M, N, K, act);
  else
    hipLaunchKernelGGL(k_rowdot<float>, dim3(blocks), dim3(256), 0, s, in, (const float*)w, b, out, M, N, K, act);
  return hipGetLastError();
}

// RoPE table: (cos, sin) of (prefix_len[b] + i) * base^(-2d/Dh), fp64 arithmetic.
__global__ void k_rope_table(const int* __restrict__ prefix_len, float2* __restrict__ tab, int B, int H, int Dh,
                             float base) {
  const int half = Dh / 2;
  const int idx = blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= B * H * half) return;
  const int d = idx % half, bi = idx / half, i = bi % H, b = bi / H;
  const double pos = (double)prefix_len[b] + (double)i;
  const double ang = pos * pow((double)base, -2.0 * (double)d / (double)Dh);
  tab[idx] = make_float2((float)cos(ang), (float)sin(ang));
}

hipError_t launch_rope_table(const int* prefix_len, float2* tab, int B, int H, int Dh, float base, hipStream_t s) {
  const int n = B * H * (Dh / 2);
  hipLaunchKernelGGL(k_rope_table, dim3((n + 255) / 256), dim3(256), 0, s, prefix_len, tab, B, H, Dh, base);
  return hipGetLastError();
}

__global__ void k_init_x(const float* __restrict__ noise, const float* __restrict__ committed, float* __restrict__ x,
                         int B, int H, int A, int n_fixed) {
  const int idx = blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= B * H * A) return;
  const int a = idx % A, i = (idx / A) % H, b = idx / (A * H);
  x[idx] = i < n_fixed ? committed[((size_t)b * n_fixed + i) * A + a] : noise[idx];
}

hipError_t launch_init_x(const float* noise, const float* committed, float* x, int B, int H, int A, int n_fixed,
                         hipStream_t s) {
  const int n = B * H * A;
  hipLaunchKernelGGL(k_init_x, dim3((n + 255) / 256), dim3(256), 0, s, noise, committed, x, B, H, A, n_fixed);
  return hipGetLastError();
}

}  // namespace jpi
