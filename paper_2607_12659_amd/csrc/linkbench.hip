// Microbenchmark of one producer -> consumer link between workgroups of a
// persistent kernel on one GPU: the primitive every phase of the
// single-launch denoise kernel pays per layer.  A standalone executable
// (built by linkbench.py), not part of libjpi.
//
// G workgroups (one per compute unit) run a chain of P phases.  In phase p
// the first `consumers` workgroups read the whole activation act[p] (`kb`
// KiB, a fresh buffer per phase, written once) and reduce it to a checksum;
// the first `producers` workgroups then write their share of act[p + 1] as a
// function of that checksum, so every phase depends on the previous one.
// The host recomputes every checksum.  Modes of the link:
//   flags     producer stores (device-coherent, sc1), waits for their
//             confirmation (s_waitcnt vmcnt(0)), stores its completion flag;
//             consumers poll the producers' flags, then load the data (sc1)
//   flags-l2  as flags, the data loaded without the coherence bit (the
//             buffers are written once per launch, so no stale line exists)
//   flags-dma as flags, the data moved by direct-to-LDS loads (sc1)
//   poll-all  no flags: act[p + 1] starts as 0xFFFFFFFF words and consumers
//             load all of it, reloading 16-byte pieces still holding that
//             value (no producer-side confirmation wait)
//   poll-tail no flags: consumers poll only the last piece each producer
//             writes, then load everything and reload stale pieces
//   flags-xcd each of the 8 XCDs runs its own chain in its own buffers:
//             producers / 8 and consumers / 8 workgroups of the XCD, with
//             the store and load cache-policy bits of the configuration
//             (flags-xcd: device-coherent both ways; flags-xcd-l2store:
//             stores without scope bits, which stay in the XCD's shared L2,
//             and device-coherent loads).
//             Workgroup w must run on XCD w % 8 (the hardware's round-robin
//             placement); each workgroup records the XCD id register and the
//             host reports where the placement held.
// `bg` KiB per workgroup of a background stream (the weight tile of the real
// kernel) are issued at each phase start into LDS and awaited by phase end.
// Every wait is bounded: past a spin limit the run records an error and
// stops waiting, so a launch always ends.
#include <hip/hip_runtime.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <vector>

namespace {

typedef unsigned u32;
typedef u32 u32x4 __attribute__((ext_vector_type(4)));
typedef __amdgpu_buffer_rsrc_t rsrc_t;
typedef __attribute__((address_space(3))) char lds_t;

constexpr int PT = 256;
constexpr u32 SENT = 0xFFFFFFFFu;
constexpr unsigned SPIN = 1u << 18;
constexpr int BG_LDS = 16 * 1024;              // background stream lands here (cycled)
constexpr int LDS_BYTES = BG_LDS + 128 * 1024;  // then room for a whole 128 KiB activation

enum Mode { FLAGS = 0, FLAGS_L2 = 1, FLAGS_DMA = 2, POLL_ALL = 3, POLL_TAIL = 4, FLAGS_XCD = 5 };
const char* const MODE_NAME[] = {"flags", "flags-l2", "flags-dma", "poll-all", "poll-tail", "flags-xcd"};
constexpr int NXCD = 8;

__device__ __forceinline__ rsrc_t rs(const void* b) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(b), 0, 0x7fffffff, 0x00020000);
}
template <int CP>
__device__ __forceinline__ u32x4 ld16(rsrc_t r, u32 off) {
  asm volatile("" ::: "memory");  // a polling load must not be hoisted out of its loop
  return __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, CP);
}
__device__ __forceinline__ u32 ld4c(rsrc_t r, u32 off) {
  asm volatile("" ::: "memory");
  return __builtin_amdgcn_raw_buffer_load_b32(r, off, 0, 16);
}
__device__ __forceinline__ u32 xcc_id() {
  u32 v;
  asm volatile("s_getreg_b32 %0, hwreg(HW_REG_XCC_ID)" : "=s"(v));
  return v & 0xfu;
}
__device__ __forceinline__ void st16c(rsrc_t r, u32 off, u32x4 v) { __builtin_amdgcn_raw_buffer_store_b128(v, r, off, 0, 16); }
__device__ __forceinline__ void st4c(rsrc_t r, u32 off, u32 v) { __builtin_amdgcn_raw_buffer_store_b32(v, r, off, 0, 16); }
// flags-xcd stores: device-coherent (sc1) or without scope bits (kept in the
// XCD's L2); its loads are the device-coherent ones of the other modes
__device__ __forceinline__ void st16x(rsrc_t r, u32 off, u32x4 v, bool l2) {
  if (l2)
    __builtin_amdgcn_raw_buffer_store_b128(v, r, off, 0, 0);
  else
    st16c(r, off, v);
}
__device__ __forceinline__ void st4x(rsrc_t r, u32 off, u32 v, bool l2) {
  if (l2)
    __builtin_amdgcn_raw_buffer_store_b32(v, r, off, 0, 0);
  else
    st4c(r, off, v);
}
__device__ __forceinline__ bool stale(u32x4 v) { return v[0] == SENT || v[1] == SENT || v[2] == SENT || v[3] == SENT; }

__device__ __forceinline__ u32 value(u32 c, int p, u32 i) { return (c * 2654435761u + i * 40503u + (u32)p) & 0x7fffffffu; }

struct Args {
  u32* act;        // [P + 1][words]
  u32* flags;      // [8][256][32]: one 128-byte line per producer (per XCD chain in flags-xcd)
  const u32* bg;   // background stream source
  long long bg_total;
  u32* err;
  u32* csum;       // [8][P] checksum seen by the first workgroup of each chain
  u32* where;      // [G] XCD id register of each workgroup
  int P, words, producers, consumers, mode, bg_bytes;
  int l2store;  // flags-xcd: stores without scope bits
};

template <int PPT>
__global__ __launch_bounds__(PT) void k_chain(Args a) {
  __shared__ __attribute__((aligned(16))) char s_lds[LDS_BYTES];
  __shared__ u32 red[PT / 64];
  __shared__ u32 s_abort;
  const int t = threadIdx.x, G = gridDim.x, lane = t & 63, wave = t >> 6;
  const bool xcd = a.mode == FLAGS_XCD;
  // in flags-xcd the chain of XCD c is run by workgroups c, c + 8, ...
  const int chain = xcd ? (int)blockIdx.x % NXCD : 0, wg = xcd ? (int)blockIdx.x / NXCD : (int)blockIdx.x;
  const int producers = xcd ? a.producers / NXCD : a.producers, consumers = xcd ? a.consumers / NXCD : a.consumers;
  const int pieces = a.words / 4, per = pieces / producers;
  const bool flagged = a.mode == FLAGS || a.mode == FLAGS_L2 || a.mode == FLAGS_DMA || xcd;
  u32* const act = a.act + (size_t)chain * (a.P + 1) * a.words;
  u32* const flg = a.flags + (size_t)chain * 256 * 32;
  if (t == 0) s_abort = 0;
  if (t == 0) a.where[blockIdx.x] = xcc_id();
  __syncthreads();
  for (int p = 0; p < a.P; ++p) {
    if (a.bg_bytes > 0) {
      const long long base = ((long long)p * G + blockIdx.x) * a.bg_bytes % (a.bg_total - a.bg_bytes);
      const char* src = (const char*)a.bg + (base & ~1023LL);
      for (int i = wave; i < a.bg_bytes / 1024; i += PT / 64)
        __builtin_amdgcn_global_load_lds(src + (size_t)i * 1024 + lane * 16, (lds_t*)s_lds + (i % (BG_LDS / 1024)) * 1024,
                                         16, 0, 0);
    }
    if (wg >= consumers) {  // only the chain: nothing to read in this phase
      asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
      __syncthreads();
      continue;
    }
    const rsrc_t rc = rs(act + (size_t)p * a.words);
    if (p > 0 && t < 64 && s_abort == 0 && (flagged || a.mode == POLL_TAIL)) {
      u32 pend = 0;
      for (int u = 0; u < 4; ++u) pend |= (t + 64 * u < producers ? 1u : 0u) << u;
      for (unsigned sp = 0;; ++sp) {
        for (int u = 0; u < 4; ++u) {
          if (!((pend >> u) & 1u)) continue;
          const int w = t + 64 * u;
          const bool ok = flagged ? ld4c(rs(flg), (u32)w * 128u) >= (u32)p
                                  : !stale(ld16<16>(rc, (u32)(w * per + per - 1) * 16u));
          if (ok) pend &= ~(1u << u);
        }
        if (__all(pend == 0u)) break;
        if (sp > SPIN) {
          if (t == 0) { s_abort = 1; st4c(rs(a.err), 0, 1u); }
          break;
        }
      }
    }
    if (flagged || a.mode == POLL_TAIL) __syncthreads();
    u32x4 v[PPT];
    if (a.mode == FLAGS_DMA) {
#pragma unroll
      for (int k = 0; k < PPT; ++k)
        __builtin_amdgcn_raw_ptr_buffer_load_lds(rc, (lds_t*)s_lds + BG_LDS + (size_t)(k * PT + wave * 64) * 16, 16,
                                                 (u32)(t + k * PT) * 16u, 0, 0, 16);
      asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
      __syncthreads();
#pragma unroll
      for (int k = 0; k < PPT; ++k) v[k] = *(const u32x4*)(s_lds + BG_LDS + (size_t)(t + k * PT) * 16);
    } else {
#pragma unroll
      for (int k = 0; k < PPT; ++k)
        v[k] = a.mode == FLAGS_L2 ? ld16<0>(rc, (u32)(t + k * PT) * 16u)
                                  : ld16<16>(rc, (u32)(t + k * PT) * 16u);
    }
    if (!flagged && p > 0 && !s_abort) {
      for (unsigned sp = 0;; ++sp) {
        bool bad = false;
#pragma unroll
        for (int k = 0; k < PPT; ++k)
          if (stale(v[k])) {
            v[k] = ld16<16>(rc, (u32)(t + k * PT) * 16u);
            bad = true;
          }
        if (!bad) break;
        if (sp > SPIN || s_abort) {
          if (!s_abort) { s_abort = 1; st4c(rs(a.err), 0, 2u); }
          break;
        }
      }
    }
    u32 c = 0;
#pragma unroll
    for (int k = 0; k < PPT; ++k) c += v[k][0] + v[k][1] + v[k][2] + v[k][3];
    for (int o = 32; o > 0; o >>= 1) c += __shfl_xor(c, o, 64);
    if (lane == 0) red[wave] = c;
    __syncthreads();
    c = red[0] + red[1] + red[2] + red[3];
    __syncthreads();
    if (wg == 0 && t == 0) a.csum[(size_t)chain * a.P + p] = c;
    if (wg < producers) {
      const rsrc_t rn = rs(act + (size_t)(p + 1) * a.words);
      for (int q = t; q < per; q += PT) {  // the thread with q = per - 1 writes the producer's last piece
        const u32 i0 = (u32)(wg * per + q) * 4u;
        const u32x4 w4{value(c, p, i0), value(c, p, i0 + 1), value(c, p, i0 + 2), value(c, p, i0 + 3)};
        if (xcd)
          st16x(rn, i0 * 4u, w4, a.l2store);
        else
          st16c(rn, i0 * 4u, w4);
      }
    }
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");  // stores (flagged modes) and the background loads
    __syncthreads();
    if (t == 0 && flagged && wg < producers) {
      if (xcd)
        st4x(rs(flg), (u32)wg * 128u, (u32)(p + 1), a.l2store);
      else
        st4c(rs(flg), (u32)wg * 128u, (u32)(p + 1));
    }
  }
}

__global__ void k_fill(u32* p, size_t n, u32 v) {
  for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x) p[i] = v;
}

#define CK(x)                                                                   \
  do {                                                                          \
    hipError_t e_ = (x);                                                        \
    if (e_ != hipSuccess) {                                                     \
      fprintf(stderr, "%s:%d %s\n", __FILE__, __LINE__, hipGetErrorString(e_)); \
      exit(1);                                                                  \
    }                                                                           \
  } while (0)

}  // namespace

// linkbench [P]: one line per configuration "mode kb producers consumers bg us_per_phase errors mismatches"
int main(int argc, char** argv) {
  const int P = argc > 1 ? atoi(argv[1]) : 400;
  hipDeviceProp_t prop;
  CK(hipGetDeviceProperties(&prop, 0));
  const int G = prop.multiProcessorCount;
  const long long bg_total = 1LL << 30;
  const int max_words = 128 * 1024 / 4;
  u32 *act, *flags, *bg, *err, *csum, *where;
  CK(hipMalloc(&act, (size_t)NXCD * (P + 1) * max_words * 4));
  CK(hipMalloc(&flags, NXCD * 256 * 128));
  CK(hipMalloc(&bg, bg_total));
  CK(hipMalloc(&err, 4));
  CK(hipMalloc(&csum, (size_t)NXCD * P * 4));
  CK(hipMalloc(&where, (size_t)G * 4));
  hipLaunchKernelGGL(k_fill, dim3(4096), dim3(256), 0, 0, bg, (size_t)(bg_total / 4), 1u);
  struct Cfg { int mode, kb, producers, consumers, bg, l2store = 0; };
  std::vector<Cfg> cfgs;
  for (int bgk : {0, 64})
    for (int kb : {16, 128})
      for (int mode = 0; mode < 5; ++mode) cfgs.push_back({mode, kb, 64, G, bgk});
  for (int cons : {64, 128}) cfgs.push_back({FLAGS, 128, 64, cons, 0});
  // one XCD's share: 8 producers and 32 consumers, device-coherent and XCD-local
  for (int bgk : {0, 64})
    for (int kb : {16, 128}) cfgs.push_back({FLAGS, kb, 8, 32, bgk});
  if (G == 256) {
    // device-coherent stores and loads (the control), then stores kept in the
    // XCD's L2 with device-coherent loads; loads with the group-scope bit or
    // after a compute-unit cache invalidation never observed another compute
    // unit's stores here and are not run
    for (int bgk : {0, 64})
      for (int kb : {16, 128})
        for (int l2 : {0, 1}) cfgs.push_back({FLAGS_XCD, kb, 64, G, bgk, l2});
  }
  printf("# CUs %d, %d phases per run\n", G, P);
  for (const Cfg& c : cfgs) {
    const int words = c.kb * 256, pieces = words / 4;
    const int chains = c.mode == FLAGS_XCD ? NXCD : 1, prod = c.producers / chains;
    if (pieces % prod || c.producers > G || c.consumers > G || c.producers > c.consumers) continue;
    for (int ch = 0; ch < chains; ++ch) {
      u32* base = act + (size_t)ch * (P + 1) * words;
      hipLaunchKernelGGL(k_fill, dim3(4096), dim3(256), 0, 0, base, (size_t)(P + 1) * words, SENT);
      hipLaunchKernelGGL(k_fill, dim3(64), dim3(256), 0, 0, base, (size_t)words, 3u);
    }
    CK(hipMemset(flags, 0, NXCD * 256 * 128));
    CK(hipMemset(err, 0, 4));
    Args a{act, flags, bg, bg_total, err, csum, where, P, words, c.producers, c.consumers, c.mode, c.bg * 1024,
           c.l2store};
    hipEvent_t e0, e1;
    CK(hipEventCreate(&e0));
    CK(hipEventCreate(&e1));
    CK(hipDeviceSynchronize());
    CK(hipEventRecord(e0, 0));
    if (pieces == 4 * PT)
      hipLaunchKernelGGL(k_chain<4>, dim3(G), dim3(PT), 0, 0, a);
    else
      hipLaunchKernelGGL(k_chain<32>, dim3(G), dim3(PT), 0, 0, a);
    CK(hipGetLastError());
    CK(hipEventRecord(e1, 0));
    CK(hipDeviceSynchronize());
    float ms = 0;
    CK(hipEventElapsedTime(&ms, e0, e1));
    u32 herr = 0;
    CK(hipMemcpy(&herr, err, 4, hipMemcpyDeviceToHost));
    std::vector<u32> hc((size_t)chains * P), cur(words, 3u), nxt(words);
    CK(hipMemcpy(hc.data(), csum, (size_t)chains * P * 4, hipMemcpyDeviceToHost));
    int bad = 0;
    for (int p = 0; p < P; ++p) {
      u32 s = 0;
      for (int i = 0; i < words; ++i) s += cur[i];
      for (int ch = 0; ch < chains; ++ch)
        if (s != hc[(size_t)ch * P + p]) ++bad;
      for (int i = 0; i < words; ++i) nxt[i] = (s * 2654435761u + (u32)i * 40503u + (u32)p) & 0x7fffffffu;
      cur.swap(nxt);
    }
    std::vector<u32> hw(G);
    CK(hipMemcpy(hw.data(), where, (size_t)G * 4, hipMemcpyDeviceToHost));
    int placed = 0, per_xcd[16] = {0};
    for (int w = 0; w < G; ++w) {
      placed += hw[w] == (u32)(w % NXCD);
      ++per_xcd[hw[w] & 15];
    }
    if (c.mode == FLAGS_XCD && placed != G) {
      printf("# %s %d KiB: workgroup w ran on XCD w %% 8 for only %d of %d workgroups; per XCD:", MODE_NAME[c.mode],
             c.kb, placed, G);
      for (int x = 0; x < NXCD; ++x) printf(" %d", per_xcd[x]);
      printf("\n");
    }
    const char* name = c.mode != FLAGS_XCD ? MODE_NAME[c.mode] : c.l2store ? "flags-xcd-l2store" : "flags-xcd";
    printf("%s %d %d %d %d %.3f %u %d\n", name, c.kb, c.producers, c.consumers, c.bg, ms * 1e3 / P, herr,
           bad);
    fflush(stdout);
    CK(hipEventDestroy(e0));
    CK(hipEventDestroy(e1));
  }
  return 0;
}
