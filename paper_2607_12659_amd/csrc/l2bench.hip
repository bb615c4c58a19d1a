// Microbenchmark of the read rate a compute unit gets from the L2 cache and
// from HBM: the ceiling of the GEMM and attention K loops, whose operand
// tiles are shared by many workgroups and mostly hit in L2.  A standalone
// executable (built by l2bench.py), not part of libjpi.
//
// G workgroups of W waves each read `per_wg` bytes from a region of R bytes,
// every wave U one-kilobyte loads (64 lanes x 16 bytes) at a time, at
// offsets that start at the workgroup's own place in the region and wrap
// around it (R is a power of two, so every offset stays inside the region).
// A 1 MiB region is read by every workgroup and stays in each die's L2 after
// the first pass; a 1 GiB region gives each workgroup a stretch of its own,
// read once from HBM.  Two kinds of load:
//   vector  global_load_dwordx4 into registers, folded into a checksum that
//           each thread stores at the end (so no load is dead)
//   lds     direct-to-LDS buffer loads into a 64 KiB ring (the GEMM and
//           attention rings' load), waited for in batches of U
// The host times each launch with HIP events (median of 5, after one warm-up
// launch) and prints bytes read per unit per second and over the chip.
#include <hip/hip_runtime.h>
#include <stdio.h>
#include <stdlib.h>

#include <algorithm>
#include <vector>

namespace {

typedef unsigned u32;
typedef u32 u32x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) char lds_t;

constexpr int RING = 64 * 1024;

#define CHECK(x)                                                                          \
  do {                                                                                    \
    hipError_t e_ = (x);                                                                  \
    if (e_ != hipSuccess) {                                                               \
      fprintf(stderr, "%s:%d %s: %s\n", __FILE__, __LINE__, #x, hipGetErrorString(e_));  \
      exit(1);                                                                            \
    }                                                                                     \
  } while (0)

// s_waitcnt vmcnt(N), other counters not waited for
template <int N>
__device__ __forceinline__ void wait_vm() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

// vec_mask = R / 16 - 1 (R a power of two); start: this workgroup's first
// 16-byte vector; iters batches of U loads per wave
template <int U>
__global__ __launch_bounds__(1024) void k_vector(const u32x4* __restrict__ src, u32 vec_mask, u32 wg_stride, int iters,
                                                 u32x4* __restrict__ out) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, nw = blockDim.x >> 6;
  u32 base = blockIdx.x * wg_stride + (u32)(w * U * 64);
  u32x4 acc = u32x4{0u, 0u, 0u, 0u};
  for (int it = 0; it < iters; ++it) {
    u32x4 v[U];
#pragma unroll
    for (int u = 0; u < U; ++u) v[u] = src[(base + (u32)(u * 64 + lane)) & vec_mask];
#pragma unroll
    for (int u = 0; u < U; ++u) acc ^= v[u];
    base += (u32)(nw * U * 64);
  }
  out[blockIdx.x * blockDim.x + threadIdx.x] = acc;
}

// The LDS address of a direct-to-LDS load must be the same for the whole
// wave: slot (w * U + u) % 64 of the ring, one kilobyte each.
__device__ __forceinline__ void dma_1k(const void* base, u32 bytes, u32 off, lds_t* dst) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(
      __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), 0, (int)bytes, 0x00020000), dst, 16, off, 0, 0, 0);
}

template <int U>
__global__ __launch_bounds__(1024) void k_lds(const u32x4* __restrict__ src, u32 vec_mask, u32 wg_stride, int iters,
                                              u32 region_bytes, u32x4* __restrict__ out) {
  __shared__ __attribute__((aligned(1024))) char ring[RING];
  const int lane = threadIdx.x & 63, w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), nw = blockDim.x >> 6;
  u32 base = blockIdx.x * wg_stride + (u32)(w * U * 64);
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const u32 vec = (base + (u32)(u * 64 + lane)) & vec_mask;
      dma_1k(src, region_bytes, vec * 16u, (lds_t*)ring + ((w * U + u) % (RING / 1024)) * 1024);
    }
    wait_vm<U>();  // the previous batch has landed: between U and 2U loads in flight
    base += (u32)(nw * U * 64);
  }
  wait_vm<0>();
  __syncthreads();
  // one word of the ring per thread, so the loads have a visible result
  out[blockIdx.x * blockDim.x + threadIdx.x] = *reinterpret_cast<const u32x4*>(ring + (threadIdx.x * 16) % RING);
}

struct Cfg {
  bool lds;
  int wgs, waves, u;
  size_t region;
};

template <int U>
void launch(const Cfg& c, const u32x4* src, u32x4* out, int iters, u32 wg_stride) {
  const u32 mask = (u32)(c.region / 16 - 1);
  if (c.lds)
    hipLaunchKernelGGL(k_lds<U>, dim3(c.wgs), dim3(64 * c.waves), 0, 0, src, mask, wg_stride, iters, (u32)c.region, out);
  else
    hipLaunchKernelGGL(k_vector<U>, dim3(c.wgs), dim3(64 * c.waves), 0, 0, src, mask, wg_stride, iters, out);
}

}  // namespace

int main(int argc, char** argv) {
  const size_t per_wg = (argc > 1 ? (size_t)atol(argv[1]) : 16) << 20;  // MiB read by each workgroup
  hipDeviceProp_t prop;
  CHECK(hipGetDeviceProperties(&prop, 0));
  const int n_cu = prop.multiProcessorCount;
  const size_t big = (size_t)1 << 30;
  u32x4* src = nullptr;
  u32x4* out = nullptr;
  CHECK(hipMalloc(&src, big));
  CHECK(hipMalloc(&out, (size_t)n_cu * 1024 * sizeof(u32x4)));
  CHECK(hipMemset(src, 0x5a, big));
  hipEvent_t e0, e1;
  CHECK(hipEventCreate(&e0));
  CHECK(hipEventCreate(&e1));
  printf("# CUs %d, %zu MiB read per workgroup\n", n_cu, per_wg >> 20);
  std::vector<Cfg> cfgs;
  for (int lds = 0; lds < 2; ++lds)
    for (size_t region : {(size_t)1 << 20, big})
      for (int wgs : {n_cu, n_cu / 2, n_cu / 4})
        for (int waves : {4, 8, 16})
          for (int u : {4, 8, 16}) cfgs.push_back(Cfg{lds == 1, wgs, waves, u, region});
  for (const Cfg& c : cfgs) {
    const size_t per_batch = (size_t)c.waves * c.u * 1024;
    // a 1 GiB region gives each workgroup its own stretch (read once, so at
    // most the stretch); in the 1 MiB one the workgroups start 64 KiB apart
    const size_t stride_bytes = c.region == big ? big / (size_t)n_cu : (size_t)64 * 1024;
    const int iters = (int)((c.region == big ? std::min(per_wg, stride_bytes) : per_wg) / per_batch);
    const u32 wg_stride = (u32)(stride_bytes / 16);
    std::vector<float> ms;
    for (int r = 0; r < 6; ++r) {
      CHECK(hipEventRecord(e0, 0));
      if (c.u == 4) launch<4>(c, src, out, iters, wg_stride);
      else if (c.u == 8) launch<8>(c, src, out, iters, wg_stride);
      else launch<16>(c, src, out, iters, wg_stride);
      CHECK(hipGetLastError());
      CHECK(hipEventRecord(e1, 0));
      CHECK(hipEventSynchronize(e1));
      float t = 0.f;
      CHECK(hipEventElapsedTime(&t, e0, e1));
      if (r > 0) ms.push_back(t);
    }
    std::sort(ms.begin(), ms.end());
    const double t = ms[ms.size() / 2] * 1e-3;
    const double bytes = (double)iters * per_batch;
    printf("%s %s %d %d %d %.1f %.2f %.4f\n", c.lds ? "lds" : "vector", c.region == big ? "hbm" : "l2", c.wgs, c.waves,
           c.u, bytes / t / 1e9, bytes * c.wgs / t / 1e12, t * 1e3);
    fflush(stdout);
  }
  CHECK(hipFree(src));
  CHECK(hipFree(out));
  return 0;
}
