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

#include "jpi_internal.h"

namespace jpi {

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

template <typename T>
struct Mfma;

template <>
struct Mfma<bf16> {
  static constexpr int KPL = 8;    // k values per lane per instruction
  static constexpr int KSUB = 32;  // k depth of one instruction
  typedef bf16x8 frag;
  static __device__ __forceinline__ frag load(const bf16* p) { return *reinterpret_cast<const bf16x8*>(p); }
  static __device__ __forceinline__ f32x4 run(frag a, frag b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
  }
};

template <>
struct Mfma<float> {
  static constexpr int KPL = 1;
  static constexpr int KSUB = 4;
  typedef float frag;
  static __device__ __forceinline__ frag load(const float* p) { return *p; }
  static __device__ __forceinline__ f32x4 run(frag a, frag b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
  }
};

template <typename T>
__device__ __forceinline__ T from_f32(float v) { return static_cast<T>(v); }

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

__device__ __forceinline__ double wave_sum_d(double v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

// Sum over the 16 lanes that share lane / 16 (one row group of an MFMA tile).
__device__ __forceinline__ float group16_sum(float v) {
#pragma unroll
  for (int o = 8; o >= 1; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}
__device__ __forceinline__ float group16_max(float v) {
#pragma unroll
  for (int o = 8; o >= 1; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}

// Block of 256 threads: fixed-order sum (wave sums, then the 4 wave totals in order).
__device__ __forceinline__ float block_sum_256(float v, float* red) {
  v = wave_sum(v);
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  __syncthreads();
  if (lane == 0) red[w] = v;
  __syncthreads();
  return ((red[0] + red[1]) + red[2]) + red[3];
}

__device__ __forceinline__ float gelu_tanh(float z) {
  const float c = 0.7978845608028654f;  // sqrt(2 / pi)
  return 0.5f * z * (1.0f + tanhf(c * (z + 0.044715f * z * z * z)));
}

// ===========================================================================
// GEMM: acc[m][n] = sum_k A[m][k] W[n][k], A and W row-major with leading
// dimension K.  Workgroup tile BM x BN, 4 waves in a 2 x 2 arrangement, K
// staged through LDS in BK slices with register double buffering.  With
// splitk > 1, blockIdx.z owns one K slice; each slice writes its fp32 partial
// tile and the last slice to finish (counted with an atomic) sums all slices
// in order z = 0..splitk-1 and runs the epilogue.
// ===========================================================================
template <typename T, int BM, int BN>
struct GemmShape {
  static constexpr int BK = sizeof(T) == 2 ? 64 : 32;
  static constexpr int VEC = 16 / sizeof(T);      // elements per 16-byte chunk
  static constexpr int LDK = BK + VEC;            // padded LDS row (bank spread)
  static constexpr int WM = BM / 2, WN = BN / 2;  // wave tile
  static constexpr int TM = WM / 16, TN = WN / 16;
  static constexpr int CPR = BK / VEC;            // 16-byte chunks per tile row
  static constexpr int A_CH = BM * CPR / 256;
  static constexpr int W_CH = BN * CPR / 256;
  static_assert(TN % 2 == 0, "epilogues pair n-subtiles 2t and 2t+1");
  static_assert(A_CH >= 1 && W_CH >= 1, "tile too small for 256 threads");
};

template <typename T, EpiKind EPI>
__device__ __forceinline__ void epilogue_pair(const EpiParams& ep, int M, int N, int row, int col_lo, float lo,
                                              float hi) {
  if (row >= M) return;
  const int col_hi = col_lo + 16;
  if constexpr (EPI == EPI_STORE_F32) {
    if (col_lo < N) ep.out_f32[(size_t)row * N + col_lo] = lo;
    if (col_hi < N) ep.out_f32[(size_t)row * N + col_hi] = hi;
  } else if constexpr (EPI == EPI_RESID) {
    float* hr = ep.h + (size_t)row * N;
    hr[col_lo] += ep.gate[col_lo] * lo;
    hr[col_hi] += ep.gate[col_hi] * hi;
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
      T* dst = hn >= 0 ? reinterpret_cast<T*>(ep.q) + (((size_t)b * ep.n_heads + hn) * H + i) * Dh
                       : reinterpret_cast<T*>(ep.ks) + ((size_t)b * H + i) * Dh;
      dst[d] = from_f32<T>(r_lo);
      dst[d + half] = from_f32<T>(r_hi);
    } else {
      const int within = col_lo - qcols - Dh;  // v: natural order
      T* dst = reinterpret_cast<T*>(ep.vs) + ((size_t)b * H + i) * Dh;
      dst[within] = from_f32<T>(lo);
      dst[within + 16] = from_f32<T>(hi);
    }
  }
}

template <typename T, int BM, int BN, EpiKind EPI>
__global__ __launch_bounds__(256) void k_gemm(GemmLaunch g) {
  using S = GemmShape<T, BM, BN>;
  using MF = Mfma<T>;
  __shared__ __attribute__((aligned(16))) T As[2][BM * S::LDK];
  __shared__ __attribute__((aligned(16))) T Ws[2][BN * S::LDK];
  __shared__ unsigned s_last;

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
      *reinterpret_cast<uint4*>(&As[buf][r * S::LDK + cc * S::VEC]) = ra[c];
    }
#pragma unroll
    for (int c = 0; c < S::W_CH; ++c) {
      const int e = tid + c * 256, r = e / S::CPR, cc = e - r * S::CPR;
      *reinterpret_cast<uint4*>(&Ws[buf][r * S::LDK + cc * S::VEC]) = rw[c];
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
    const T* as = As[buf] + (wm * S::WM + fr) * S::LDK + fk;
    const T* ws = Ws[buf] + (wn * S::WN + fr) * S::LDK + fk;
#pragma unroll
    for (int kk = 0; kk < S::BK; kk += MF::KSUB) {
      typename MF::frag af[S::TM], bfr[S::TN];
#pragma unroll
      for (int a = 0; a < S::TM; ++a) af[a] = MF::load(as + a * 16 * S::LDK + kk);
#pragma unroll
      for (int b = 0; b < S::TN; ++b) bfr[b] = MF::load(ws + b * 16 * S::LDK + kk);
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
  if (g.splitk > 1) {
    float* P = g.partial + (size_t)blockIdx.z * M * N;
#pragma unroll
    for (int a = 0; a < S::TM; ++a)
#pragma unroll
      for (int b = 0; b < S::TN; ++b)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int row = rbase + a * 16 + i, col = cbase + b * 16;
          if (row < M && col < N) P[(size_t)row * N + col] = acc[a][b][i];
        }
    __threadfence();
    __syncthreads();
    if (tid == 0) {
      const unsigned tile = blockIdx.y * gridDim.x + blockIdx.x;
      const unsigned prev = atomicAdd(&g.counters[tile], 1u);
      s_last = prev == (unsigned)g.splitk - 1u;
      if (s_last) g.counters[tile] = 0u;  // every slice has arrived: ready for the next launch
    }
    __syncthreads();
    if (!s_last) return;
    __threadfence();
#pragma unroll
    for (int a = 0; a < S::TM; ++a)
#pragma unroll
      for (int b = 0; b < S::TN; ++b)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int row = rbase + a * 16 + i, col = cbase + b * 16;
          float sum = 0.f;
          if (row < M && col < N)
            for (int z = 0; z < g.splitk; ++z) sum += g.partial[((size_t)z * M + row) * N + col];
          acc[a][b][i] = sum;
        }
  }
#pragma unroll
  for (int a = 0; a < S::TM; ++a)
#pragma unroll
    for (int b = 0; b < S::TN; b += 2)
#pragma unroll
      for (int i = 0; i < 4; ++i)
        epilogue_pair<T, EPI>(g.ep, M, N, rbase + a * 16 + i, cbase + b * 16, acc[a][b][i], acc[a][b + 1][i]);
}

template <typename T>
static void gemm_tile(int M, int& BM, int& BN) {
  if (sizeof(T) == 2 && M > 64) {
    BM = 128;
    BN = 128;
  } else {
    BM = 64;
    BN = 64;
  }
}

size_t gemm_tiles(jpi_dtype dt, int M, int N) {
  int BM, BN;
  if (dt == JPI_BF16) gemm_tile<bf16>(M, BM, BN);
  else gemm_tile<float>(M, BM, BN);
  return (size_t)((N + BN - 1) / BN) * ((M + BM - 1) / BM);
}

int gemm_pick_splitk(jpi_dtype dt, int M, int N, int K, int n_cu) {
  const int BK = dt == JPI_BF16 ? 64 : 32;
  const size_t tiles = gemm_tiles(dt, M, N);
  int s = 1;
  while (s < 16 && tiles * s < (size_t)(2 * n_cu) && K % (2 * s * BK) == 0) s *= 2;
  return s;
}

template <typename T, int BM, int BN>
static hipError_t launch_gemm_t(const GemmLaunch& g, hipStream_t s) {
  dim3 grid((g.N + BN - 1) / BN, (g.M + BM - 1) / BM, g.splitk);
  switch (g.epi) {
    case EPI_STORE_F32: hipLaunchKernelGGL((k_gemm<T, BM, BN, EPI_STORE_F32>), grid, dim3(256), 0, s, g); break;
    case EPI_QKV: hipLaunchKernelGGL((k_gemm<T, BM, BN, EPI_QKV>), grid, dim3(256), 0, s, g); break;
    case EPI_GEGLU: hipLaunchKernelGGL((k_gemm<T, BM, BN, EPI_GEGLU>), grid, dim3(256), 0, s, g); break;
    case EPI_RESID: hipLaunchKernelGGL((k_gemm<T, BM, BN, EPI_RESID>), grid, dim3(256), 0, s, g); break;
  }
  return hipGetLastError();
}

hipError_t launch_gemm(jpi_dtype dt, const GemmLaunch& g, hipStream_t s) {
  if (dt == JPI_BF16) {
    if (g.M > 64) return launch_gemm_t<bf16, 128, 128>(g, s);
    return launch_gemm_t<bf16, 64, 64>(g, s);
  }
  return launch_gemm_t<float, 64, 64>(g, s);
}

// ===========================================================================
// adaRMSNorm: y[m][k] = h[m][k] / sqrt(mean_k h^2 + eps) * (1 + scale[k]) + shift[k]
// ===========================================================================
template <typename T>
__global__ __launch_bounds__(256) void k_rmsnorm_mod(const float* __restrict__ h, const float* __restrict__ scale,
                                                     const float* __restrict__ shift, T* __restrict__ y, int W,
                                                     float eps) {
  __shared__ float red[4];
  const int m = blockIdx.x;
  const float* hr = h + (size_t)m * W;
  float ss = 0.f;
  for (int k = threadIdx.x; k < W; k += 256) ss += hr[k] * hr[k];
  ss = block_sum_256(ss, red);
  const float r = 1.0f / sqrtf(ss / (float)W + eps);
  for (int k = threadIdx.x; k < W; k += 256)
    y[(size_t)m * W + k] = from_f32<T>(hr[k] * r * (1.0f + scale[k]) + shift[k]);
}

hipError_t launch_rmsnorm_mod(jpi_dtype dt, const float* h, const float* scale, const float* shift, void* y,
                              int M, int W, float eps, hipStream_t s) {
  if (dt == JPI_BF16)
    hipLaunchKernelGGL(k_rmsnorm_mod<bf16>, dim3(M), dim3(256), 0, s, h, scale, shift, (bf16*)y, W, eps);
  else
    hipLaunchKernelGGL(k_rmsnorm_mod<float>, dim3(M), dim3(256), 0, s, h, scale, shift, (float*)y, W, eps);
  return hipGetLastError();
}

// ===========================================================================
// action input projection: h[m][n] = sum_a x[m][a] W_in[n][a] + b_in[n]
// ===========================================================================
template <typename T>
__global__ __launch_bounds__(256) void k_inproj(const float* __restrict__ x, const T* __restrict__ w,
                                                const float* __restrict__ b, float* __restrict__ h, int M, int W,
                                                int A) {
  const int idx = blockIdx.x * 256 + threadIdx.x;
  if (idx >= M * W) return;
  const int m = idx / W, n = idx - m * W;
  float acc = 0.f;
  for (int a = 0; a < A; ++a) acc = fmaf(x[(size_t)m * A + a], static_cast<float>(w[(size_t)n * A + a]), acc);
  h[idx] = acc + b[n];
}

hipError_t launch_inproj(jpi_dtype dt, const float* x, const void* w_in, const float* b_in, float* h, int M,
                         int W, int A, hipStream_t s) {
  const int blocks = (M * W + 255) / 256;
  if (dt == JPI_BF16)
    hipLaunchKernelGGL(k_inproj<bf16>, dim3(blocks), dim3(256), 0, s, x, (const bf16*)w_in, b_in, h, M, W, A);
  else
    hipLaunchKernelGGL(k_inproj<float>, dim3(blocks), dim3(256), 0, s, x, (const float*)w_in, b_in, h, M, W, A);
  return hipGetLastError();
}

// ===========================================================================
// final adaRMSNorm + action-out projection + Euler update of rows i >= n_fixed:
// v = (rms(h) (1 + s_f) + b_f) W_out^T + b_out;  x += dt * v
// ===========================================================================
template <typename T>
__global__ __launch_bounds__(256) void k_final_euler(const float* __restrict__ h, const float* __restrict__ scale,
                                                     const float* __restrict__ shift, const T* __restrict__ w_out,
                                                     const float* __restrict__ b_out, float* __restrict__ x, int W,
                                                     int A, int H, int n_fixed, float dt, float eps) {
  extern __shared__ float ys[];  // [W]
  __shared__ float red[4];
  const int m = blockIdx.x, lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const float* hr = h + (size_t)m * W;
  float ss = 0.f;
  for (int k = threadIdx.x; k < W; k += 256) ss += hr[k] * hr[k];
  ss = block_sum_256(ss, red);
  const float r = 1.0f / sqrtf(ss / (float)W + eps);
  for (int k = threadIdx.x; k < W; k += 256) ys[k] = hr[k] * r * (1.0f + scale[k]) + shift[k];
  __syncthreads();
  const int i = m % H;
  for (int a = wave; a < A; a += 4) {
    float acc = 0.f;
    for (int k = lane; k < W; k += 64) acc = fmaf(ys[k], static_cast<float>(w_out[(size_t)a * W + k]), acc);
    acc = wave_sum(acc);
    if (lane == 0 && i >= n_fixed) x[(size_t)m * A + a] += dt * (acc + b_out[a]);
  }
}

hipError_t launch_final_euler(jpi_dtype dt, const float* h, const float* scale, const float* shift,
                              const void* w_out, const float* b_out, float* x, int M, int W, int A, int horizon,
                              int n_fixed, float dt_step, float eps, hipStream_t s) {
  const size_t lds = (size_t)W * sizeof(float);
  if (dt == JPI_BF16)
    hipLaunchKernelGGL(k_final_euler<bf16>, dim3(M), dim3(256), lds, s, h, scale, shift, (const bf16*)w_out, b_out,
                       x, W, A, horizon, n_fixed, dt_step, eps);
  else
    hipLaunchKernelGGL(k_final_euler<float>, dim3(M), dim3(256), lds, s, h, scale, shift, (const float*)w_out,
                       b_out, x, W, A, horizon, n_fixed, dt_step, eps);
  return hipGetLastError();
}

// ===========================================================================
// prefix + self attention, one shared KV head (Appendix: queries from the
// action tokens, keys/values = LLM layer KV ++ action tokens' own KV).
// The concatenated key sequence [prefix 0..pl-1 | action 0..H-1] is cut into
// chunks of KC keys; a workgroup handles one (rollout, head, 64-query block,
// chunk) and writes the chunk's running max, sum and unnormalised output.
// Slots j >= pl of the prefix are never read.
// ===========================================================================
template <typename T>
struct AttnShape {
  static constexpr int KC = sizeof(T) == 2 ? 64 : 32;
  static constexpr int PAD = 16 / sizeof(T);
};

template <typename T, int DH>
__global__ __launch_bounds__(256) void k_attn_partial(AttnLaunch a) {
  using MF = Mfma<T>;
  constexpr int KC = AttnShape<T>::KC, PAD = AttnShape<T>::PAD;
  constexpr int LDK = DH + PAD, LDV = KC + PAD, LDP = KC + PAD;
  constexpr int NST = DH / MF::KSUB;  // k steps over the head dim
  constexpr int NJ = KC / 16;         // key subtiles
  constexpr int VEC = 16 / sizeof(T);
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
  const T* vp = reinterpret_cast<const T*>(a.vp) + (size_t)b * a.kp_bstride;
  const T* ksb = reinterpret_cast<const T*>(a.ks) + (size_t)b * H * DH;
  const T* vsb = reinterpret_cast<const T*>(a.vs) + (size_t)b * H * DH;
  constexpr int CPR = DH / VEC;
  for (int e = tid; e < KC * CPR; e += 256) {
    const int r = e / CPR, cc = e - r * CPR;
    const int kidx = kbase + r;
    uint4 kv = make_uint4(0, 0, 0, 0), vv = make_uint4(0, 0, 0, 0);
    if (kidx < pl) {
      kv = *reinterpret_cast<const uint4*>(kp + (size_t)kidx * DH + cc * VEC);
      vv = *reinterpret_cast<const uint4*>(vp + (size_t)kidx * DH + cc * VEC);
    } else if (kidx < nkeys) {
      kv = *reinterpret_cast<const uint4*>(ksb + (size_t)(kidx - pl) * DH + cc * VEC);
      vv = *reinterpret_cast<const uint4*>(vsb + (size_t)(kidx - pl) * DH + cc * VEC);
    }
    *reinterpret_cast<uint4*>(&Ks[r * LDK + cc * VEC]) = kv;
    const T* vt = reinterpret_cast<const T*>(&vv);
#pragma unroll
    for (int j = 0; j < VEC; ++j) Vt[(cc * VEC + j) * LDV + r] = vt[j];
  }

  // query fragments of this wave's 16 rows, kept in registers
  const int fr = lane & 15, fk = (lane >> 4) * MF::KPL;
  const int iq = qb * 64 + w * 16 + fr;
  typename MF::frag qf[NST];
  {
    const T* qrow = reinterpret_cast<const T*>(a.q) + (((size_t)b * a.nH + hn) * H + (iq < H ? iq : 0)) * DH;
#pragma unroll
    for (int st = 0; st < NST; ++st) {
      if (iq < H) qf[st] = MF::load(qrow + st * MF::KSUB + fk);
      else qf[st] = typename MF::frag{};
    }
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
  const int H = a.H;
  const int i = blockIdx.x % H, bh = blockIdx.x / H;
  const int b = bh / a.nH, hn = bh - b * a.nH;
  const float* Mp = a.mpart + (size_t)bh * nch * H;
  const float* Lp = a.lpart + (size_t)bh * nch * H;
  const float* Op = a.opart + (size_t)bh * nch * H * DH;
  float mx = -INFINITY;
  for (int c = 0; c < nch; ++c) mx = fmaxf(mx, Mp[c * H + i]);
  float L = 0.f;
  for (int c = 0; c < nch; ++c) {
    const float mc = Mp[c * H + i];
    if (mc != -INFINITY) L += expf(mc - mx) * Lp[c * H + i];
  }
  const float inv = 1.0f / L;
  TO* out = reinterpret_cast<TO*>(a.out) + ((size_t)b * H + i) * a.nH * DH + hn * DH;
  for (int d = threadIdx.x; d < DH; d += blockDim.x) {
    float acc = 0.f;
    for (int c = 0; c < nch; ++c) {
      const float mc = Mp[c * H + i];
      if (mc != -INFINITY) acc += expf(mc - mx) * Op[((size_t)c * H + i) * DH + d];
    }
    out[d] = from_f32<TO>(acc * inv);
  }
}

int attn_chunk(jpi_dtype dt) { return dt == JPI_BF16 ? AttnShape<bf16>::KC : AttnShape<float>::KC; }
int attn_n_chunks(jpi_dtype dt, int P, int H) {
  const int kc = attn_chunk(dt);
  return (P + H + kc - 1) / kc;
}

template <typename T, int DH>
static hipError_t launch_attention_t(const AttnLaunch& a, hipStream_t s) {
  const int nch = attn_n_chunks(sizeof(T) == 2 ? JPI_BF16 : JPI_F32, a.P, a.H);
  const int nqb = (a.H + 63) / 64;
  hipLaunchKernelGGL((k_attn_partial<T, DH>), dim3(nch, a.nH * nqb, a.B), dim3(256), 0, s, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int thr = DH < 256 ? DH : 256;
  if (a.out_f32)
    hipLaunchKernelGGL((k_attn_combine<float, DH>), dim3(a.B * a.nH * a.H), dim3(thr), 0, s, a, nch);
  else
    hipLaunchKernelGGL((k_attn_combine<T, DH>), dim3(a.B * a.nH * a.H), dim3(thr), 0, s, a, nch);
  return hipGetLastError();
}

hipError_t launch_attention(jpi_dtype dt, const AttnLaunch& a, hipStream_t s) {
  if (dt == JPI_BF16) {
    switch (a.Dh) {
      case 64: return launch_attention_t<bf16, 64>(a, s);
      case 128: return launch_attention_t<bf16, 128>(a, s);
      case 256: return launch_attention_t<bf16, 256>(a, s);
    }
  } else {
    switch (a.Dh) {
      case 64: return launch_attention_t<float, 64>(a, s);
      case 128: return launch_attention_t<float, 128>(a, s);
      case 256: return launch_attention_t<float, 256>(a, s);
    }
  }
  return hipErrorInvalidValue;
}

// ===========================================================================
// once per (weights, n_steps): timestep embedding, time MLP and the
// modulation table.  fp64 arithmetic; results stored in fp32.
// ===========================================================================
__global__ void k_time_embed(float* emb, int n, int W) {
  const int idx = blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= n * W) return;
  const int k = idx / W, j = idx - k * W, half = W / 2;
  const int jj = j < half ? j : j - half;
  const double t = 1.0 - (double)k / (double)n;
  const double f = exp(-log(1.0e4) * (double)jj / (double)half);
  const double arg = 1000.0 * t * f;
  emb[idx] = (float)(j < half ? cos(arg) : sin(arg));
}

hipError_t launch_time_embed(const float* /*unused*/, float* emb, int n, int W, hipStream_t s) {
  hipLaunchKernelGGL(k_time_embed, dim3((n * W + 255) / 256), dim3(256), 0, s, emb, n, W);
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
