// Internal declarations shared by the libjpi runtime and its kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/jpi.h"

namespace jpi {

typedef __bf16 bf16;

// ---------------------------------------------------------------------------
// Epilogue descriptors for the GEMM kernel.  A GEMM computes
// acc[m][n] = sum_k A[m][k] W[n][k] (fp32) and hands each value to one of
// these epilogues.  Packed column orders are described in jpi_runtime.hip.
// ---------------------------------------------------------------------------
enum EpiKind { EPI_STORE_F32 = 0, EPI_QKV = 1, EPI_GEGLU = 2, EPI_RESID = 3 };

struct EpiParams {
  // EPI_STORE_F32
  float* out_f32;        // [M][N]
  // EPI_QKV: packed columns [q heads | k | v]; RoPE on q and k
  void* q;               // [B][nH][H][Dh]
  void* ks;              // [B][H][Dh]
  void* vs;              // [B][H][Dh]
  const float2* rope;    // [B][H][Dh/2] (cos, sin) at position prefix_len[b] + i
  int n_heads, head_dim, horizon;
  // EPI_GEGLU: packed columns in 32-wide groups [gate 16 | up 16]
  void* z;               // [M][F]
  int mlp_dim;
  // EPI_RESID: h[m][n] += gate[n] * acc
  float* h;              // [M][N]
  const float* gate;     // [N]
};

struct GemmLaunch {
  const void* A;         // [M][K]
  const void* W;         // [N][K]
  int M, N, K;
  int splitk;
  float* partial;        // [splitk][M][N] fp32 scratch when splitk > 1
  unsigned* counters;    // one per output tile, zero on entry, left zero on exit
  EpiKind epi;
  EpiParams ep;
};

// launchers (jpi_kernels.hip).  All return hipSuccess or the launch error.
hipError_t launch_gemm(jpi_dtype dt, const GemmLaunch& g, hipStream_t s);
size_t gemm_tiles(jpi_dtype dt, int M, int N);          // counters needed
int gemm_pick_splitk(jpi_dtype dt, int M, int N, int K, int n_cu);

hipError_t launch_rmsnorm_mod(jpi_dtype dt, const float* h, const float* scale, const float* shift,
                              void* y, int M, int W, float eps, hipStream_t s);

hipError_t launch_inproj(jpi_dtype dt, const float* x, const void* w_in, const float* b_in, float* h,
                         int M, int W, int A, hipStream_t s);

hipError_t launch_final_euler(jpi_dtype dt, const float* h, const float* scale, const float* shift,
                              const void* w_out, const float* b_out, float* x, int M, int W, int A,
                              int horizon, int n_fixed, float dt_step, float eps, hipStream_t s);

struct AttnLaunch {
  const void* q;          // [B][nH][H][Dh]
  const void* ks;         // [B][H][Dh]
  const void* vs;         // [B][H][Dh]
  const void* kp;         // prefix K for this layer: rollout b at kp + b*kp_bstride elements
  const void* vp;
  int64_t kp_bstride;     // elements between rollouts in kp / vp
  const int* prefix_len;  // device [B]
  int B, nH, H, P, Dh;
  float* opart;           // [B][nH][n_chunks][H][Dh]
  float* mpart;           // [B][nH][n_chunks][H]
  float* lpart;           // [B][nH][n_chunks][H]
  void* out;              // [B*H][nH*Dh] of dtype, or fp32 if out_f32
  int out_f32;
};
int attn_chunk(jpi_dtype dt);
int attn_n_chunks(jpi_dtype dt, int P, int H);
hipError_t launch_attention(jpi_dtype dt, const AttnLaunch& a, hipStream_t s);

hipError_t launch_time_embed(const float* t, float* emb, int n, int W, hipStream_t s);
// out[m][n] = act(sum_k in[m][k] w[n][k] + b[n]), fp64 accumulation; act 0 = none, 1 = swish
hipError_t launch_rowdot(jpi_dtype dt, const float* in, const void* w, const float* b, float* out, int M,
                         int N, int K, int act, hipStream_t s);
hipError_t launch_rope_table(const int* prefix_len, float2* tab, int B, int H, int Dh, float base,
                             hipStream_t s);
hipError_t launch_init_x(const float* noise, const float* committed, float* x, int B, int H, int A,
                         int n_fixed, hipStream_t s);

}  // namespace jpi
