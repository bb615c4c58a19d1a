// Kernels of the action-time expert variant (include/jpi.h,
// JPI_VARIANT_ACTION_TIME): the per-step action-time MLP around the GEMMs,
// the constant modulation table of plain RMSNorm layers, and the state
// token's keys and values written into the prefix slot after each rollout's
// valid prefix.
#include "jpi_device.h"
#include "jpi_internal.h"

namespace jpi {

namespace {

// Table rows [rows][(6L+2)W] of plain RMSNorm layers: norm j < 2L gives
// (scale, shift, gate) = (w_j, 0, 1); the final norm (w_2L, 0).
__global__ void k_const_table(float* __restrict__ tab, const float* __restrict__ norms, int rows, int L, int W) {
  const size_t R = (size_t)(6 * L + 2) * W;
  const size_t n = (size_t)rows * R;
  for (size_t idx = (size_t)blockIdx.x * blockDim.x + threadIdx.x; idx < n; idx += (size_t)gridDim.x * blockDim.x) {
    const size_t c = idx % R;
    const int j = c < (size_t)6 * L * W ? (int)(c / (3 * (size_t)W)) : 2 * L;
    const size_t within = c < (size_t)6 * L * W ? c % (3 * (size_t)W) : c - (size_t)6 * L * W;
    const int part = (int)(within / W), k = (int)(within % W);
    tab[idx] = part == 0 ? norms[(size_t)j * W + k] : part == 1 ? 0.f : 1.f;
  }
}

__global__ void k_plus_one(const int* __restrict__ src, int* __restrict__ dst, int n) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) dst[i] = src[i] + 1;
}

// u[b H + i] = T(W_a x[b][i] + b_a), one workgroup per action row
template <typename T>
__global__ __launch_bounds__(256) void k_action_embed(const float* __restrict__ x, const T* __restrict__ w,
                                                      const float* __restrict__ b, T* __restrict__ u, int W, int A) {
  __shared__ float xs[256];
  const int m = blockIdx.x;
  for (int a = threadIdx.x; a < A; a += 256) xs[a] = x[(size_t)m * A + a];
  __syncthreads();
  for (int n = threadIdx.x; n < W; n += 256) {
    float acc = 0.f;
    for (int a = 0; a < A; ++a) acc = fmaf(xs[a], static_cast<float>(w[(size_t)n * A + a]), acc);
    u[(size_t)m * W + n] = from_f32<T>(acc + b[n]);
  }
}

// z[m][n] = T(swish(sum_s P[s][m][n] + c[n])), one workgroup per row
template <typename T>
__global__ __launch_bounds__(256) void k_swish_slices(const float* __restrict__ part, int S, int M,
                                                      const float* __restrict__ c, T* __restrict__ z, int W) {
  const int m = blockIdx.x;
  const size_t MW = (size_t)M * W;
  for (int n = threadIdx.x; n < W; n += 256) {
    float v = c[n];
    for (int s = 0; s < S; ++s) v += part[s * MW + (size_t)m * W + n];
    z[(size_t)m * W + n] = from_f32<T>(v / (1.0f + expf(-v)));
  }
}

// the state row's key (rotated) and value of one layer into prefix slot prefix_len[b]
template <typename T>
__global__ void k_put_state_kv(const T* __restrict__ ks, const T* __restrict__ vst, int vst_ld, T* __restrict__ kp,
                               int64_t kp_bstride, T* __restrict__ vpt, int64_t vpt_bstride, int vpt_dstride,
                               const int* __restrict__ prefix_len, int Dh) {
  const int b = blockIdx.x;
  const int pl = prefix_len[b];
  for (int d = threadIdx.x; d < Dh; d += blockDim.x) {
    kp[b * kp_bstride + (int64_t)pl * Dh + d] = ks[(size_t)b * Dh + d];
    vpt[b * vpt_bstride + (int64_t)d * vpt_dstride + pl] = vst[((size_t)b * Dh + d) * vst_ld];
  }
}

}  // namespace

hipError_t launch_const_table(float* tab, const float* norms, int rows, int L, int W, hipStream_t s) {
  hipLaunchKernelGGL(k_const_table, dim3(1024), dim3(256), 0, s, tab, norms, rows, L, W);
  return hipGetLastError();
}

hipError_t launch_plus_one(const int* src, int* dst, int n, hipStream_t s) {
  hipLaunchKernelGGL(k_plus_one, dim3((n + 255) / 256), dim3(256), 0, s, src, dst, n);
  return hipGetLastError();
}

hipError_t launch_action_embed(jpi_dtype dt, const float* x, const void* w, const float* b, void* u, int M, int W,
                               int A, hipStream_t s) {
  if (A > 256 || M < 1) return hipErrorInvalidValue;
  if (dt == JPI_BF16)
    hipLaunchKernelGGL(k_action_embed<bf16>, dim3(M), dim3(256), 0, s, x, (const bf16*)w, b, (bf16*)u, W, A);
  else
    hipLaunchKernelGGL(k_action_embed<float>, dim3(M), dim3(256), 0, s, x, (const float*)w, b, (float*)u, W, A);
  return hipGetLastError();
}

hipError_t launch_swish_slices(jpi_dtype dt, const float* part, int S, int M, const float* c, void* z, int W,
                               hipStream_t s) {
  if (M < 1 || S < 1) return hipErrorInvalidValue;
  if (dt == JPI_BF16)
    hipLaunchKernelGGL(k_swish_slices<bf16>, dim3(M), dim3(256), 0, s, part, S, M, c, (bf16*)z, W);
  else
    hipLaunchKernelGGL(k_swish_slices<float>, dim3(M), dim3(256), 0, s, part, S, M, c, (float*)z, W);
  return hipGetLastError();
}

hipError_t launch_put_state_kv(jpi_dtype dt, const void* ks, const void* vst, int vst_ld, void* kp, int64_t kp_bstride,
                               void* vpt, int64_t vpt_bstride, int vpt_dstride, const int* prefix_len, int B, int Dh,
                               hipStream_t s) {
  if (B < 1) return hipErrorInvalidValue;
  if (dt == JPI_BF16)
    hipLaunchKernelGGL(k_put_state_kv<bf16>, dim3(B), dim3(256), 0, s, (const bf16*)ks, (const bf16*)vst, vst_ld,
                       (bf16*)kp, kp_bstride, (bf16*)vpt, vpt_bstride, vpt_dstride, prefix_len, Dh);
  else
    hipLaunchKernelGGL(k_put_state_kv<float>, dim3(B), dim3(256), 0, s, (const float*)ks, (const float*)vst, vst_ld,
                       (float*)kp, kp_bstride, (float*)vpt, vpt_bstride, vpt_dstride, prefix_len, Dh);
  return hipGetLastError();
}

}  // namespace jpi
