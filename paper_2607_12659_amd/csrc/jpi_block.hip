// Pre-norm decoder blocks with constant modulation, shared by the VLM prefill
// and the future correction module.  Such a block (RMSNorm with (1 + w)
// scaling, attention with one shared KV head, a plain residual, a tanh-GeGLU
// MLP) is the action expert's layer with scale = w, shift = 0 and gate = 1,
// so it runs the expert's kernels: the tiled GEMM with the QKV+RoPE, fp32
// split-K and GeGLU epilogues, the batched attention and the residual + norm
// row kernel.  Also the small row kernels and the weight packing both users
// need.
#include <vector>

#include "jpi_device.h"
#include "jpi_internal.h"

namespace jpi {

namespace {

// y[m] = T(h[m] / rms(h[m]) * (1 + w)), one workgroup per row
template <typename T>
__global__ __launch_bounds__(256) void k_norm_rows(const float* __restrict__ h, const float* __restrict__ w,
                                                   T* __restrict__ y, int W, float eps) {
  __shared__ float red[4];
  const float* hr = h + (size_t)blockIdx.x * W;
  float ss = 0.f;
  for (int i = threadIdx.x; i < W; i += 256) ss += hr[i] * hr[i];
  ss = block_sum_256(ss, red);
  const float r = 1.0f / sqrtf(ss / (float)W + eps);
  T* yr = y + (size_t)blockIdx.x * W;
  for (int i = threadIdx.x; i < W; i += 256) yr[i] = from_f32<T>(hr[i] * r * (1.0f + w[i]));
}

__global__ void k_fill_i32(int* p, int n, int v) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = v;
}

__global__ void k_fill_f32(float* p, int n, float v) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = v;
}

__global__ void k_fill_f2(float2* p, int n, float2 v) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = v;
}

// dst[m] = src[m % period], rows of W floats
__global__ void k_bcast_rows(const float* __restrict__ src, float* __restrict__ dst, int period, int W) {
  const float* s = src + (size_t)(blockIdx.x % period) * W;
  float* d = dst + (size_t)blockIdx.x * W;
  for (int i = threadIdx.x; i < W; i += blockDim.x) d[i] = s[i];
}

// dst row map[r] <- src row r (row_bytes each, a multiple of 4)
__global__ void k_scatter(const char* __restrict__ src, char* __restrict__ dst, const int* __restrict__ map,
                          int row_bytes) {
  const char* s = src + (size_t)blockIdx.x * row_bytes;
  char* d = dst + (size_t)map[blockIdx.x] * row_bytes;
  for (int i = threadIdx.x * 4; i < row_bytes; i += blockDim.x * 4)
    *reinterpret_cast<int*>(d + i) = *reinterpret_cast<const int*>(s + i);
}

}  // namespace

hipError_t launch_norm_rows(const float* h, const float* w, void* y, int M, int W, float eps, hipStream_t s,
                            bool f32) {
  if (M < 1) return hipSuccess;
  if (f32) hipLaunchKernelGGL(k_norm_rows<float>, dim3(M), dim3(256), 0, s, h, w, (float*)y, W, eps);
  else hipLaunchKernelGGL(k_norm_rows<bf16>, dim3(M), dim3(256), 0, s, h, w, (bf16*)y, W, eps);
  return hipGetLastError();
}

hipError_t launch_fill_i32(int* p, int n, int v, hipStream_t s) {
  if (n < 1) return hipSuccess;
  hipLaunchKernelGGL(k_fill_i32, dim3((n + 255) / 256), dim3(256), 0, s, p, n, v);
  return hipGetLastError();
}

hipError_t launch_fill_f32(float* p, int n, float v, hipStream_t s) {
  if (n < 1) return hipSuccess;
  hipLaunchKernelGGL(k_fill_f32, dim3((n + 255) / 256), dim3(256), 0, s, p, n, v);
  return hipGetLastError();
}

hipError_t launch_identity_rope(float2* tab, int n, hipStream_t s) {
  if (n < 1) return hipSuccess;
  hipLaunchKernelGGL(k_fill_f2, dim3((n + 255) / 256), dim3(256), 0, s, tab, n, float2{1.f, 0.f});
  return hipGetLastError();
}

hipError_t launch_bcast_rows(const float* src, float* dst, int M, int period, int W, hipStream_t s) {
  if (M < 1) return hipSuccess;
  if (period < 1) return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_bcast_rows, dim3(M), dim3(256), 0, s, src, dst, period, W);
  return hipGetLastError();
}

int block_rope_row(int r, int Dh) {
  const int half = Dh / 2, dd = r % Dh, head = r / Dh, hi = dd >= half ? 1 : 0, d = dd - hi * half;
  return head * Dh + (d / 16) * 32 + hi * 16 + (d % 16);
}

int block_pack_row(BlockMatrix kind, int r, int n_heads, int Dh) {
  switch (kind) {
    case BM_Q: return block_rope_row(r, Dh);
    case BM_K: return n_heads * Dh + block_rope_row(r, Dh);
    case BM_V: return (n_heads + 1) * Dh + r;
    case BM_GATE: return (r / 16) * 32 + (r % 16);
    case BM_UP: return (r / 16) * 32 + 16 + (r % 16);
  }
  return r;
}

hipError_t upload_rows(void* dst, const std::vector<int>& map, int row_bytes, const void* data, bool is_device,
                       hipStream_t s) {
  const int rows = (int)map.size();
  void *src = const_cast<void*>(data), *tmp = nullptr, *dmap = nullptr;
  hipError_t e = hipMalloc(&dmap, rows * sizeof(int));
  if (e != hipSuccess) return e;
  if (!is_device) {
    e = hipMalloc(&tmp, (size_t)rows * row_bytes);
    if (e == hipSuccess) e = hipMemcpyAsync(tmp, data, (size_t)rows * row_bytes, hipMemcpyHostToDevice, s);
    src = tmp;
  }
  if (e == hipSuccess) e = hipMemcpyAsync(dmap, map.data(), rows * sizeof(int), hipMemcpyHostToDevice, s);
  if (e == hipSuccess) {
    hipLaunchKernelGGL(k_scatter, dim3(rows), dim3(256), 0, s, (const char*)src, (char*)dst, (const int*)dmap,
                       row_bytes);
    e = hipGetLastError();
  }
  if (e == hipSuccess) e = hipStreamSynchronize(s);
  (void)hipFree(dmap);
  if (tmp) (void)hipFree(tmp);
  return e;
}

hipError_t enqueue_block(const BlockLaunch& b, hipStream_t s) {
  const int M = b.B * b.H, W = b.W, nH = b.nH, Dh = b.Dh, F = b.F;
  const jpi_dtype dt = b.f32 ? JPI_F32 : JPI_BF16;
  hipError_t e;
  GemmLaunch g{};
  g.A = b.y;
  g.W = b.w;
  g.M = M;
  g.N = (nH + 2) * Dh;
  g.K = W;
  g.splitk = 1;
  g.n_cu = b.n_cu;
  g.epi = EPI_QKV;
  g.ep.q = b.q;
  g.ep.ks = b.ks;
  g.ep.ks_bstride = b.ks_bstride;
  g.ep.vst = b.vst;
  g.ep.vst_ld = b.vst_ld;
  g.ep.rope = b.rope;
  g.ep.n_heads = nH;
  g.ep.head_dim = Dh;
  g.ep.horizon = b.H;
  if ((e = launch_gemm(dt, g, s)) != hipSuccess) return e;
  AttnLaunch a{};
  a.q = b.q;
  a.ks = b.ks;
  a.ks_bstride = b.ks_bstride;
  a.vst = b.vst;
  a.vst_ld = b.vst_ld;
  a.kp = b.kp;
  a.vpt = b.vpt;
  a.kp_bstride = b.kp_bstride;
  a.vpt_bstride = b.vpt_bstride;
  a.vpt_dstride = b.vpt_dstride;
  a.prefix_len = b.prefix_len;
  a.B = b.B;
  a.nH = nH;
  a.H = b.H;
  a.P = b.P;
  a.Dh = Dh;
  a.opart = b.opart;
  if (b.f32) {  // the fp32 attention's chunk maxima and sums follow its partial rows
    const int nch = attn_n_chunks(dt, b.P, b.H);
    a.mpart = b.opart + (size_t)b.B * nH * nch * b.H * Dh;
    a.lpart = a.mpart + (size_t)b.B * nH * nch * b.H;
  }
  a.out = b.o;
  a.out_f32 = 0;
  a.n_cu = b.n_cu;
  if ((e = launch_attention(dt, a, s)) != hipSuccess) return e;
  g = GemmLaunch{};
  g.A = b.o;
  g.W = b.w + b.off_o * (b.f32 ? 4 : 2);
  g.M = M;
  g.N = W;
  g.K = nH * Dh;
  g.splitk = b.s_o;
  g.n_cu = b.n_cu;
  g.epi = EPI_STORE_F32;
  g.ep.out_f32 = b.partial;
  if ((e = launch_gemm(dt, g, s)) != hipSuccess) return e;
  RowLaunch r{};
  r.part = b.partial;
  r.S = b.s_o;
  r.M = M;
  r.W = W;
  r.h = b.h;
  r.gate = b.ones;
  r.scale = b.mlp_norm;
  r.shift = b.zeros;
  r.y = b.y;
  r.eps = b.eps;
  if ((e = launch_resid_norm(dt, r, false, s)) != hipSuccess) return e;
  g = GemmLaunch{};
  g.A = b.y;
  g.W = b.w + b.off_gu * (b.f32 ? 4 : 2);
  g.M = M;
  g.N = 2 * F;
  g.K = W;
  g.splitk = 1;
  g.n_cu = b.n_cu;
  g.epi = EPI_GEGLU;
  g.ep.z = b.z;
  g.ep.mlp_dim = F;
  if ((e = launch_gemm(dt, g, s)) != hipSuccess) return e;
  g = GemmLaunch{};
  g.A = b.z;
  g.W = b.w + b.off_d * (b.f32 ? 4 : 2);
  g.M = M;
  g.N = W;
  g.K = F;
  g.splitk = b.s_d;
  g.n_cu = b.n_cu;
  g.epi = EPI_STORE_F32;
  g.ep.out_f32 = b.partial;
  if ((e = launch_gemm(dt, g, s)) != hipSuccess) return e;
  r.S = b.s_d;
  r.scale = b.next_norm;
  return launch_resid_norm(dt, r, false, s);
}

}  // namespace jpi
