// Batched prefix + self attention (bf16) for the multi-kernel path.
//
// Queries come from the action tokens; keys and values are the prefix KV of
// the layer followed by the action tokens' own (Appendix, action expert).
// All query heads share the single KV head, so one rollout's nH x H query rows
// form one [nH*H][Dh] matrix (row r = head * H + i) against one key sequence.
// A workgroup takes 128 of those rows (8 waves x 16) and a range of 64-key
// blocks, and streams each block's K and V^T once through double-buffered LDS
// with a running (max, sum) per row (online softmax).  With one key range the
// workgroup writes the normalised output; with several it writes a bf16
// partial normalised by its own sum plus (max, sum), merged by k_flash_merge.
//
// Products use v_mfma_f32_16x16x32_bf16 with the operands swapped:
// S^T = K q^T puts one query row in each lane (lane % 16) and four keys of a
// 16-key tile in its four result elements; O^T = V^T P^T then takes P^T
// straight from those registers.  The K rows of the two 16-key tiles of a
// 32-key group are interleaved (tile jj, A row 4g + e <-> key 8g + 4jj + e)
// so that a lane's eight probabilities are eight consecutive keys, which
// makes each V^T operand one 16-byte piece of a V^T row.
//
// Key order: the action keys come first (blocks of 64, masked past H), then
// the prefix (masked past prefix_len[b]).  The softmax does not depend on the
// order.  Masked keys get probability 0 and their V entries are zeroed, so
// stale or non-finite memory in unused slots never reaches the output.
#include <math.h>

#include "jpi_device.h"
#include "jpi_internal.h"

namespace jpi {

typedef unsigned int u32;
typedef u32 u32x4 __attribute__((ext_vector_type(4)));
typedef u32 u32x2 __attribute__((ext_vector_type(2)));

template <int DH>
struct Flash {
  static constexpr int NW = 8;             // waves per workgroup (two per SIMD)
  static constexpr int KB = 64;            // keys per block
  static constexpr int QT = 16 * NW;       // query rows per workgroup (16 per wave)
  static constexpr int NST = DH / 32;      // k steps of S^T over the head dim
  static constexpr int NT = DH / 16;       // 16-wide output tiles over the head dim
  static constexpr int KFR = 4 * NST;      // 1 KB K fragments per block (4 key tiles)
  static constexpr int VFR = 2 * NT;       // 1 KB V^T fragments per block (2 key groups)
  static constexpr int KLD = KFR / NW;     // K fragments loaded per wave
  static constexpr int VLD = VFR / NW;
  static constexpr int STAGE = (KFR + VFR) * 1024;
  static_assert(KLD >= 1 && KFR % NW == 0 && VLD >= 1 && VFR % NW == 0, "fragments per wave");
};

constexpr int FLASH_MAX_SPLITS = 16;
constexpr float FLASH_LIMIT = 64.f;  // log2 headroom of the probabilities over the row reference

// elements n_ok .. 7 of 8 packed bf16 set to zero (all of them when n_ok <= 0)
__device__ __forceinline__ u32x4 mask8(u32x4 v, int n_ok) {
#pragma unroll
  for (int q = 0; q < 4; ++q) v[q] &= (2 * q < n_ok ? 0x0000ffffu : 0u) | (2 * q + 1 < n_ok ? 0xffff0000u : 0u);
  return v;
}

typedef __amdgpu_buffer_rsrc_t rsrc_t;
typedef __attribute__((address_space(3))) char lds_t;  // LDS byte pointer (direct-to-LDS loads)

// Buffer resource over [base, base + bytes): loads past the end return zero.
__device__ __forceinline__ rsrc_t rsrc(const void* base, int64_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), 0, (int)bytes, 0x00020000);
}

// Key sources of one rollout.  Action (suffix) keys: K rows [H][Dh], V^T
// rows [Dh][vst_ld].  Prefix keys: K rows [prefix_len][Dh], V^T rows
// [Dh][vpt_dstride].  The K ranges end at the last valid key, so rows past
// it read as zero.
struct FlashSrc {
  rsrc_t k_act, v_act, k_pre, v_pre;
  int nbs;  // action blocks (they come first)
};

// block jb: first key and number of valid keys of its source
__device__ __forceinline__ void flash_block(const FlashSrc& src, int H, int pl, int jb, bool& act, int& key0,
                                            int& n_ok) {
  act = jb < src.nbs;
  key0 = (act ? jb : jb - src.nbs) * 64;
  n_ok = act ? H : pl;
}

// Direct-to-LDS loads of one block into one LDS stage.  Wave w loads
// fragments w, w + NW, ...  K fragment f = kt * NST + st (kt = 2 * group +
// tile): lane row 4g' + e of the A operand is key 32 * group + 8g' +
// 4 * tile + e, k values st * 32 + 8g .. + 8 (g = lane / 16, g' and e from
// lane % 16).  V^T fragment f = group * NT + nt: dim nt * 16 + lane % 16,
// keys 32 * group + 8g .. + 8.  The per-lane part of each address (koff,
// voff) is fixed for the launch; the per-fragment part (sk, sv) is uniform
// and, with the block's first key, goes in the scalar offset.
template <int DH>
struct FlashDma {
  u32 sk[Flash<DH>::KLD], sva[Flash<DH>::VLD], svp[Flash<DH>::VLD];
};

template <int DH>
__device__ __forceinline__ FlashDma<DH> flash_dma_offsets(int vst_ld, int vpt_ld) {
  using FS = Flash<DH>;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  FlashDma<DH> d;
#pragma unroll
  for (int u = 0; u < FS::KLD; ++u) {
    const int fi = w + FS::NW * u, kt = fi / FS::NST, st = fi - kt * FS::NST;
    d.sk[u] = (u32)(((32 * (kt >> 1) + 4 * (kt & 1)) * DH + st * 32) * 2);
  }
#pragma unroll
  for (int u = 0; u < FS::VLD; ++u) {
    const int fi = w + FS::NW * u, grp = fi / FS::NT, nt = fi - grp * FS::NT;
    d.sva[u] = (u32)((nt * 16 * vst_ld + 32 * grp) * 2);
    d.svp[u] = (u32)((nt * 16 * vpt_ld + 32 * grp) * 2);
  }
  return d;
}

template <int DH>
__device__ __forceinline__ void flash_dma(lds_t* stage, const FlashSrc& src, const FlashDma<DH>& d, u32 koff,
                                          u32 vaoff, u32 vpoff, bool act, int key0) {
  using FS = Flash<DH>;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const rsrc_t rk = act ? src.k_act : src.k_pre;
  const rsrc_t rv = act ? src.v_act : src.v_pre;
  const u32 voff = act ? vaoff : vpoff;
  const u32 kb = (u32)(key0 * DH * 2), vb = (u32)(key0 * 2);
#pragma unroll
  for (int u = 0; u < FS::KLD; ++u)
    __builtin_amdgcn_raw_ptr_buffer_load_lds(rk, stage + (w + FS::NW * u) * 1024, 16, koff, kb + d.sk[u], 0, 0);
#pragma unroll
  for (int u = 0; u < FS::VLD; ++u)
    __builtin_amdgcn_raw_ptr_buffer_load_lds(rv, stage + (FS::KFR + w + FS::NW * u) * 1024, 16, voff,
                                             vb + (act ? d.sva[u] : d.svp[u]), 0, 0);
}

// After this thread's direct-to-LDS loads of a block have landed: zero the
// V^T entries of keys past the valid ones in the pieces it loaded (pieces
// past the end of a V^T row hold other data).  Only a block with fewer than
// KB valid keys has any.
template <int DH>
__device__ __forceinline__ void flash_fix(char* stage, int n_valid) {
  using FS = Flash<DH>;
  if (n_valid >= FS::KB) return;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
#pragma unroll
  for (int u = 0; u < FS::VLD; ++u) {
    const int fi = w + FS::NW * u, grp = fi / FS::NT;
    const int n_ok = n_valid - (32 * grp + 8 * (lane >> 4));
    if (n_ok < 8) {
      u32x4* p = reinterpret_cast<u32x4*>(stage + ((FS::KFR + fi) * 64 + lane) * 16);
      *p = mask8(*p, n_ok);
    }
  }
}

// One 64-key block for this wave's 16 query rows.
// Softmax in the log2 domain against a fixed per-row reference m_ref: the
// maximum of the row's first block.  A later block whose maximum exceeds the
// reference by more than FLASH_LIMIT (probabilities up to 2^FLASH_LIMIT) asks
// for a restart of the key range with that maximum as the new reference
// (the return value); the output is never rescaled.  The reference is the
// same in the four lanes of a row.  Keys n_valid .. 63 of the block are masked.
template <int DH>
__device__ __forceinline__ bool flash_compute(const char* cur, int n_valid, const bf16x8 (&qf)[Flash<DH>::NST],
                                              f32x4 (&o)[Flash<DH>::NT], float& m_ref, float& l_run, float qscale) {
  using FS = Flash<DH>;
  using MF = Mfma<bf16>;
  constexpr int NST = FS::NST, NT = FS::NT;
  const int lane = threadIdx.x & 63, g = lane >> 4;
  f32x4 sc[4];
#pragma unroll
  for (int kt = 0; kt < 4; ++kt) sc[kt] = f32x4{0.f, 0.f, 0.f, 0.f};
  // S^T = K q^T: K fragments of k step st + 1 are read from LDS while step st multiplies
  MF::frag kf[2][4];
#pragma unroll
  for (int kt = 0; kt < 4; ++kt) kf[0][kt] = *reinterpret_cast<const MF::frag*>(cur + (kt * NST * 64 + lane) * 16);
#pragma unroll
  for (int st = 0; st < NST; ++st) {
    if (st + 1 < NST) {
#pragma unroll
      for (int kt = 0; kt < 4; ++kt)
        kf[(st + 1) & 1][kt] = *reinterpret_cast<const MF::frag*>(cur + ((kt * NST + st + 1) * 64 + lane) * 16);
    }
#pragma unroll
    for (int kt = 0; kt < 4; ++kt) sc[kt] = MF::run(kf[st & 1][kt], qf[st], sc[kt]);
  }
  // instruction order: the next step's 4 LDS reads, then this step's 4 products
  __builtin_amdgcn_sched_group_barrier(0x100, 4, 0);
#pragma unroll
  for (int st = 0; st < NST; ++st) {
    if (st + 1 < NST) __builtin_amdgcn_sched_group_barrier(0x100, 4, 0);
    __builtin_amdgcn_sched_group_barrier(0x008, 4, 0);
  }

  float m = -INFINITY;
#pragma unroll
  for (int kt = 0; kt < 4; ++kt)
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      if (n_valid < FS::KB) {
        const int key = 32 * (kt >> 1) + 8 * g + 4 * (kt & 1) + e;
        sc[kt][e] = key < n_valid ? sc[kt][e] : -INFINITY;
      }
      m = fmaxf(m, sc[kt][e]);
    }
  m = fmaxf(m, __shfl_xor(m, 16, 64));
  m = fmaxf(m, __shfl_xor(m, 32, 64));
  const float mx = m * qscale;  // finite: the block holds a valid key
  const bool first = m_ref == -INFINITY, over = mx > m_ref + FLASH_LIMIT;
  const bool restart = over && !first;
  m_ref = over ? mx : m_ref;

#pragma unroll
  for (int kt = 0; kt < 4; ++kt)
#pragma unroll
    for (int e = 0; e < 4; ++e) sc[kt][e] = __builtin_amdgcn_exp2f(fmaf(sc[kt][e], qscale, -m_ref));
  // P^T as the B operand: slot 8g + j of key group grp <-> key 32 grp + 8g + j.
  // The row sum adds the same bf16-rounded probabilities that weight V, so a
  // row dominated by one key returns that key's value row exactly.
  MF::frag pb[2];
  float sum = 0.f;
#pragma unroll
  for (int grp = 0; grp < 2; ++grp)
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const bf16 lo = static_cast<bf16>(sc[2 * grp][e]), hi = static_cast<bf16>(sc[2 * grp + 1][e]);
      pb[grp][e] = lo;
      pb[grp][4 + e] = hi;
      sum += static_cast<float>(lo) + static_cast<float>(hi);
    }
  l_run += sum;
  // O^T += V^T P^T: V^T fragments read four at a time, one group ahead of the products
  constexpr int NVG = 2 * NT / 4;
  MF::frag vf[2][4];
#pragma unroll
  for (int v = 0; v < 4; ++v) vf[0][v] = *reinterpret_cast<const MF::frag*>(cur + ((FS::KFR + v) * 64 + lane) * 16);
#pragma unroll
  for (int vg = 0; vg < NVG; ++vg) {
    if (vg + 1 < NVG) {
#pragma unroll
      for (int v = 0; v < 4; ++v)
        vf[(vg + 1) & 1][v] = *reinterpret_cast<const MF::frag*>(cur + ((FS::KFR + 4 * (vg + 1) + v) * 64 + lane) * 16);
    }
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const int fi = 4 * vg + v, grp = fi / NT, nt = fi - grp * NT;
      o[nt] = MF::run(vf[vg & 1][v], pb[grp], o[nt]);
    }
  }
  __builtin_amdgcn_sched_group_barrier(0x100, 4, 1);
#pragma unroll
  for (int vg = 0; vg < NVG; ++vg) {
    if (vg + 1 < NVG) __builtin_amdgcn_sched_group_barrier(0x100, 4, 1);
    __builtin_amdgcn_sched_group_barrier(0x008, 4, 1);
  }
  return __any(restart);
}

// Work items (rollout, 128-row query tile, key range) in that order, T of
// them; the grid is T rounded up to a multiple of 8 workgroups.  The hardware
// hands workgroup i to XCD i % 8, so item (i % 8) * (grid / 8) + i / 8 puts
// consecutive items, which share a rollout's keys and values, in one XCD's L2.
template <int DH>
__global__ __launch_bounds__(512) void k_flash(AttnLaunch a, int S, int nqt, void* part, float2* ml) {
  using FS = Flash<DH>;
  using MF = Mfma<bf16>;
  constexpr int NST = FS::NST, NT = FS::NT, KB = FS::KB;
  __shared__ __attribute__((aligned(16))) char lds[2 * FS::STAGE];
  __shared__ int s_restart;

  const int item = (int)(blockIdx.x % 8) * (int)(gridDim.x / 8) + (int)(blockIdx.x / 8);
  if (item >= a.B * nqt * S) return;
  const int b = item / (nqt * S), split = item % S, qt = (item / S) % nqt;
  const int H = a.H, R = a.nH * H;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int g = lane >> 4, fr = lane & 15;
  const int pl = a.prefix_len[b];
  FlashSrc src;
  src.nbs = (H + KB - 1) / KB;
  const int nb = src.nbs + (pl + KB - 1) / KB;
  const int jb0 = (int)((int64_t)split * nb / S), jb1 = (int)((int64_t)(split + 1) * nb / S);
  const int row0 = qt * FS::QT + w * 16;  // this wave's first query row

  // each split writes its (max, sum) even when it has no keys
  if (jb0 == jb1) {
    if (S > 1) {
      const int r = qt * FS::QT + threadIdx.x;
      if (threadIdx.x < FS::QT && r < R) ml[((size_t)split * a.B + b) * R + r] = float2{-INFINITY, 0.f};
    }
    return;
  }

  src.k_act = rsrc(reinterpret_cast<const bf16*>(a.ks) + (size_t)b * (a.ks_bstride ? a.ks_bstride : (int64_t)H * DH),
                   (int64_t)H * DH * 2);
  src.v_act = rsrc(reinterpret_cast<const bf16*>(a.vst) + (size_t)b * DH * a.vst_ld, (int64_t)DH * a.vst_ld * 2);
  src.k_pre = rsrc(reinterpret_cast<const bf16*>(a.kp) + (size_t)b * a.kp_bstride, (int64_t)pl * DH * 2);
  src.v_pre = rsrc(reinterpret_cast<const bf16*>(a.vpt) + (size_t)b * a.vpt_bstride, (int64_t)DH * a.vpt_dstride * 2);
  const int vst_ld = (int)a.vst_ld, vpt_ld = (int)a.vpt_dstride;
  const u32 koff = (u32)(((8 * (fr >> 2) + (fr & 3)) * DH + 8 * g) * 2);
  const u32 vaoff = (u32)((fr * vst_ld + 8 * g) * 2), vpoff = (u32)((fr * vpt_ld + 8 * g) * 2);
  const FlashDma<DH> dofs = flash_dma_offsets<DH>(vst_ld, vpt_ld);
  if (threadIdx.x == 0) s_restart = 0;

  lds_t* lds3 = (lds_t*)lds;
  bool act;
  int key0, n_ok;
  flash_block(src, H, pl, jb0, act, key0, n_ok);
  flash_dma<DH>(lds3, src, dofs, koff, vaoff, vpoff, act, key0);

  // query fragments (B operand of S^T): lane holds row fr, dims st*32 + 8g .. + 8
  MF::frag qf[NST];
  const bf16* qb = reinterpret_cast<const bf16*>(a.q) + (size_t)b * R * DH;
  {
    const int r = row0 + fr;
#pragma unroll
    for (int st = 0; st < NST; ++st) qf[st] = r < R ? MF::load(qb + (size_t)r * DH + st * 32 + 8 * g) : MF::frag{};
  }
  const bool active = row0 < R;  // wave has query rows (uniform per wave)

  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  flash_fix<DH>(lds, n_ok - key0);
  __syncthreads();

  // log2-domain scores: s * log2(e) / sqrt(Dh)
  const float qscale = 1.4426950408889634f / sqrtf((float)DH);
  f32x4 o[NT];
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) o[nt] = f32x4{0.f, 0.f, 0.f, 0.f};
  float m_ref = -INFINITY, l_run = 0.f;

  for (int jb = jb0;;) {
    const char* cur = lds + ((jb - jb0) & 1) * FS::STAGE;
    char* nxt = lds + ((jb - jb0 + 1) & 1) * FS::STAGE;
    const int n_valid = n_ok - key0;  // valid keys of block jb (>= 1)
    const bool more = jb + 1 < jb1;
    if (more) {
      flash_block(src, H, pl, jb + 1, act, key0, n_ok);
      flash_dma<DH>(lds3 + ((jb - jb0 + 1) & 1) * FS::STAGE, src, dofs, koff, vaoff, vpoff, act, key0);
    }
    if (active && flash_compute<DH>(cur, n_valid, qf, o, m_ref, l_run, qscale) && lane == 0) s_restart = 1;
    if (more) {
      asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
      flash_fix<DH>(nxt, n_ok - key0);
    }
    __syncthreads();
    if (s_restart) {
      // a row's scores outgrew its reference: start the key range again with
      // the new references (rare; the references only grow)
      __syncthreads();
      if (threadIdx.x == 0) s_restart = 0;
      l_run = 0.f;
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) o[nt] = f32x4{0.f, 0.f, 0.f, 0.f};
      jb = jb0;
      flash_block(src, H, pl, jb0, act, key0, n_ok);
      flash_dma<DH>(lds3, src, dofs, koff, vaoff, vpoff, act, key0);
      asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
      flash_fix<DH>(lds, n_ok - key0);
      __syncthreads();
      continue;
    }
    if (++jb == jb1) break;
  }
  if (!active) return;

  // O^T: lane holds dims nt*16 + 4g .. + 4 of query row fr
  float l = l_run;
  l += __shfl_xor(l, 16, 64);
  l += __shfl_xor(l, 32, 64);
  const int r = row0 + fr;
  if (r >= R) return;
  const float rl = 1.0f / l;
  typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
  if (S == 1) {
    const int hn = r / H, i = r - hn * H;
    const size_t base = ((size_t)b * H + i) * (size_t)a.nH * DH + (size_t)hn * DH + 4 * g;
    if (a.out_f32) {
      float* out = reinterpret_cast<float*>(a.out) + base;
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) *reinterpret_cast<f32x4*>(out + nt * 16) = o[nt] * rl;
    } else {
      bf16* out = reinterpret_cast<bf16*>(a.out) + base;
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) {
        const f32x4 v = o[nt] * rl;
        *reinterpret_cast<bf16x4*>(out + nt * 16) =
            bf16x4{static_cast<bf16>(v[0]), static_cast<bf16>(v[1]), static_cast<bf16>(v[2]), static_cast<bf16>(v[3])};
      }
    }
  } else {
    const size_t rowi = ((size_t)split * a.B + b) * R + r;
    bf16* out = reinterpret_cast<bf16*>(part) + rowi * DH + 4 * g;
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      const f32x4 v = o[nt] * rl;
      *reinterpret_cast<bf16x4*>(out + nt * 16) =
          bf16x4{static_cast<bf16>(v[0]), static_cast<bf16>(v[1]), static_cast<bf16>(v[2]), static_cast<bf16>(v[3])};
    }
    if (g == 0) ml[rowi] = float2{m_ref, l};
  }
}

// out row (b, head, i) = sum_s 2^(m_s - m) l_s O_s / sum_s 2^(m_s - m) l_s,
// splits in order; a split without keys (m_s = -inf) is skipped.
// Dh / 4 threads per query row, 4 dims each.
template <int DH, typename TO>
__global__ __launch_bounds__(256) void k_flash_merge(AttnLaunch a, int S, const void* part, const float2* ml) {
  constexpr int TPR = DH / 4, RPB = 256 / TPR;
  const int R = a.nH * a.H;
  const int t = threadIdx.x, rr = blockIdx.x * RPB + t / TPR, q4 = t % TPR;
  if (rr >= a.B * R) return;
  const int b = rr / R, r = rr - b * R;
  const int hn = r / a.H, i = r - hn * a.H;
  float2 mv[FLASH_MAX_SPLITS];
  u32x2 ov[FLASH_MAX_SPLITS];
  float m = -INFINITY;
#pragma unroll
  for (int s = 0; s < FLASH_MAX_SPLITS; ++s) {
    if (s < S) {
      const size_t rowi = ((size_t)s * a.B + b) * R + r;
      mv[s] = ml[rowi];
      ov[s] = *reinterpret_cast<const u32x2*>(reinterpret_cast<const bf16*>(part) + rowi * DH + 4 * q4);
      m = fmaxf(m, mv[s].x);
    }
  }
  f32x4 acc = f32x4{0.f, 0.f, 0.f, 0.f};
  float lsum = 0.f;
#pragma unroll
  for (int s = 0; s < FLASH_MAX_SPLITS; ++s) {
    if (s < S && mv[s].x != -INFINITY) {
      const float wl = exp2f(mv[s].x - m) * mv[s].y;
      const f32x4 v = f32x4{__builtin_bit_cast(float, ov[s][0] << 16), __builtin_bit_cast(float, ov[s][0] & 0xffff0000u),
                            __builtin_bit_cast(float, ov[s][1] << 16), __builtin_bit_cast(float, ov[s][1] & 0xffff0000u)};
      acc += wl * v;
      lsum += wl;
    }
  }
  acc *= 1.0f / lsum;
  TO* out = reinterpret_cast<TO*>(a.out) + ((size_t)b * a.H + i) * (size_t)a.nH * DH + (size_t)hn * DH + 4 * q4;
#pragma unroll
  for (int e = 0; e < 4; ++e) out[e] = from_f32<TO>(acc[e]);
}

// Key ranges per (rollout, 128-row tile): enough workgroups to cover the
// chip once, at least two key blocks per range.
int flash_splits(int B, int nH, int H, int P, int n_cu) {
  const int KB = 64;
  const int nqt = (nH * H + 127) / 128;
  const int nb = (H + KB - 1) / KB + (P + KB - 1) / KB;
  int s = (n_cu + B * nqt - 1) / (B * nqt);
  s = s < nb / 2 ? s : nb / 2;
  s = s < FLASH_MAX_SPLITS ? s : FLASH_MAX_SPLITS;
  return s > 1 ? s : 1;
}

template <int DH>
static hipError_t launch_flash_t(const AttnLaunch& a, int S, hipStream_t s) {
  const int nqt = (a.nH * a.H + Flash<DH>::QT - 1) / Flash<DH>::QT;
  const size_t rows = (size_t)a.B * a.nH * a.H;
  // partial outputs (bf16) then (max, sum) pairs, inside the opart scratch
  void* part = a.opart;
  float2* ml = reinterpret_cast<float2*>(reinterpret_cast<char*>(a.opart) + (size_t)S * rows * DH * 2);
  const int items = a.B * nqt * S;
  JPI_LAUNCH((k_flash<DH>), dim3((items + 7) / 8 * 8), dim3(Flash<DH>::NW * 64), 0, s, a.ev_start,
             S == 1 ? a.ev_stop : (hipEvent_t) nullptr, a, S, nqt, part, ml);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || S == 1) return e;
  constexpr int RPB = 256 / (DH / 4);
  const dim3 grid((unsigned)((rows + RPB - 1) / RPB));
  if (a.out_f32)
    JPI_LAUNCH((k_flash_merge<DH, float>), grid, dim3(256), 0, s, (hipEvent_t) nullptr, a.ev_stop, a, S, part, ml);
  else
    JPI_LAUNCH((k_flash_merge<DH, bf16>), grid, dim3(256), 0, s, (hipEvent_t) nullptr, a.ev_stop, a, S, part, ml);
  return hipGetLastError();
}

size_t flash_scratch_bytes(int B, int nH, int H, int Dh, int S) {
  return (size_t)S * B * nH * H * ((size_t)Dh * 2 + sizeof(float2));
}

hipError_t launch_flash(const AttnLaunch& a, int S, hipStream_t s) {
  if (S < 1 || S > FLASH_MAX_SPLITS || a.H < 1 || a.B < 1) return hipErrorInvalidValue;
  switch (a.Dh) {
    case 64: return launch_flash_t<64>(a, S, s);
    case 128: return launch_flash_t<128>(a, S, s);
    case 256: return launch_flash_t<256>(a, S, s);
  }
  return hipErrorInvalidValue;
}

}  // namespace jpi
