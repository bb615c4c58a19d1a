// Batched prefix + self attention (bf16) for the multi-kernel path.
//
// Queries come from the action tokens; keys and values are the prefix KV of
// the layer followed by the action tokens' own (Appendix, action expert).
// All query heads share the single KV head, so one rollout's nH x H query rows
// form one [nH*H][Dh] matrix (row r = head * H + i) against one key sequence.
// A workgroup (eight waves, two per SIMD) takes 128 of those rows, 16 per
// wave, and a range of 32-key blocks.  The blocks stream through a
// four-stage LDS ring by direct-to-LDS buffer loads, up to three blocks ahead
// of the one being multiplied, so the loads of later blocks overlap the
// products of this one.  A running (max, sum) per row gives the online
// softmax.
// With one key range the workgroup writes the normalised output; with several
// it writes a bf16 partial normalised by its own sum plus (max, sum), merged
// by k_flash_merge.
//
// Products use v_mfma_f32_16x16x32_bf16 with the operands swapped:
// S^T = K q^T puts one query row in each lane (lane % 16) and four keys of a
// 16-key tile in its four result elements; O^T = V^T P^T then takes P^T
// straight from those registers.  The K rows of the two 16-key tiles of a
// block are interleaved (tile jj, A row 4g + e <-> key 8g + 4jj + e) so that
// a lane's eight probabilities are eight consecutive keys, which makes each
// V^T operand one 16-byte piece of a V^T row.
//
// Key order: the action keys come first (blocks of 32, masked past H), then
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
  static constexpr int NW = 8;              // waves per workgroup (two per SIMD)
  static constexpr int RT = 1;              // 16-row query tiles per wave
  static constexpr int KB = 32;             // keys per block
  static constexpr int NS = 4;              // ring stages: three blocks in flight while one is multiplied
  static constexpr int QT = 16 * RT * NW;   // query rows per workgroup
  static constexpr int NST = DH / 32;       // k steps of S^T over the head dim
  static constexpr int NT = DH / 16;        // 16-wide output tiles over the head dim
  static constexpr int KFR = 2 * NST;       // 1 KB K fragments per block (two key tiles)
  static constexpr int VFR = NT;            // 1 KB V^T fragments per block
  static constexpr int LDW = (KFR + VFR) / NW;  // direct-to-LDS loads per wave per block
  static constexpr int STAGE = (KFR + VFR) * 1024;
  static_assert((KFR + VFR) % NW == 0 && LDW >= 1, "fragments split evenly over the waves");
  // fragment w + NW * u is a K fragment iff is_k(w, u); with KFR a multiple of
  // NW that depends on u alone, so every wave's load sequence is known when
  // compiling (which keeps the compiler's count of outstanding loads exact)
  static __device__ __forceinline__ bool is_k(int w, int u) {
    return KFR % NW == 0 ? u < KFR / NW : w + NW * u < KFR;
  }
  static_assert(2 * LDW < 64, "vmcnt range");
};

constexpr int FLASH_MAX_SPLITS = 16;
constexpr float FLASH_LIMIT = 64.f;  // log2 headroom of the probabilities over the row reference

// elements n_ok .. 7 of 8 packed bf16 set to zero (all of them when n_ok <= 0)
__device__ __forceinline__ u32x4 mask8(u32x4 v, int n_ok) {
#pragma unroll
  for (int q = 0; q < 4; ++q) v[q] &= (2 * q < n_ok ? 0x0000ffffu : 0u) | (2 * q + 1 < n_ok ? 0xffff0000u : 0u);
  return v;
}

// s_waitcnt: vmcnt = N, lgkmcnt = 0 when L, other counters not waited for
template <int N, bool L>
__device__ __forceinline__ void flash_wait() {
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | ((L ? 0 : 15) << 8));
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
  int nbs, H, pl;  // action blocks (they come first), action keys, prefix keys
};

// Direct-to-LDS loads of block jb into one ring stage.  Wave w loads
// fragments w, w + NW, ...: the first KFR are K fragments f = kt * NST + st
// (lane row 4g' + e of the A operand is key 8g' + 4kt + e, k values
// st * 32 + 8g .. + 8; g = lane / 16, g' and e from lane % 16), the next VFR
// are V^T fragments nt (dim nt * 16 + lane % 16, keys 8g .. + 8).  The
// per-lane part of each address (koff, vaoff, vpoff) is fixed for the
// launch; the per-fragment part and the block's first key are added to it,
// so that the whole offset is range-checked (an offset in the scalar
// operand is not part of the buffer's range check): K rows past the last
// valid key read as zero and nothing past the source is touched.  Returns
// the block's valid key count (>= 1).
template <int DH>
__device__ __forceinline__ int flash_issue(lds_t* stage, const FlashSrc& src, int jb, u32 koff, u32 vaoff, u32 vpoff,
                                           int vst_ld, int vpt_ld) {
  using FS = Flash<DH>;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const bool act = jb < src.nbs;
  const int key0 = (act ? jb : jb - src.nbs) * FS::KB;
  const rsrc_t rk = act ? src.k_act : src.k_pre;
  const rsrc_t rv = act ? src.v_act : src.v_pre;
  const u32 voff = act ? vaoff : vpoff;
  const int vld = act ? vst_ld : vpt_ld;
#pragma unroll
  for (int u = 0; u < FS::LDW; ++u) {
    const int fi = w + FS::NW * u;
    if (FS::is_k(w, u)) {
      const int kt = fi / FS::NST, st = fi - kt * FS::NST;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rk, stage + fi * 1024, 16,
                                               koff + (u32)(((key0 + 4 * kt) * DH + st * 32) * 2), 0, 0, 0);
    } else {
      const int nt = fi - FS::KFR;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rv, stage + fi * 1024, 16, voff + (u32)((nt * 16 * vld + key0) * 2),
                                               0, 0, 0);
    }
  }
  const int n = (act ? src.H : src.pl) - key0;
  return n < FS::KB ? n : FS::KB;
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
  const int n_ok = n_valid - 8 * (lane >> 4);
  if (n_ok >= 8) return;
#pragma unroll
  for (int u = 0; u < FS::LDW; ++u) {
    const int fi = w + FS::NW * u;
    if (!FS::is_k(w, u)) {
      u32x4* p = reinterpret_cast<u32x4*>(stage + (fi * 64 + lane) * 16);
      *p = mask8(*p, n_ok);
    }
  }
}

// Maximum over the four lanes that hold one query row (lanes r, r + 16,
// r + 32, r + 48): two lane-swap instructions, no LDS round trip.  (The
// swapped pair is copied into scalars before the bit casts: a bit cast of an
// element of the returned vector reads element 0 for both.)
__device__ __forceinline__ float row4_max(float v) {
  const auto a = __builtin_amdgcn_permlane32_swap(__builtin_bit_cast(u32, v), __builtin_bit_cast(u32, v), false, false);
  const u32 a0 = a[0], a1 = a[1];
  v = fmaxf(__builtin_bit_cast(float, a0), __builtin_bit_cast(float, a1));
  const auto b = __builtin_amdgcn_permlane16_swap(__builtin_bit_cast(u32, v), __builtin_bit_cast(u32, v), false, false);
  const u32 b0 = b[0], b1 = b[1];
  return fmaxf(__builtin_bit_cast(float, b0), __builtin_bit_cast(float, b1));
}

// One 32-key block for this wave's 16-row query tiles.
// Softmax in the log2 domain against a per-row reference m_ref: the maximum
// of the row's first block.  A later block whose maximum exceeds the
// reference by more than FLASH_LIMIT (probabilities up to 2^FLASH_LIMIT)
// moves the reference up to that maximum and rescales the row's running
// output and sum by 2^(old - new); otherwise the reference stays, so rows
// whose scores stay within that headroom are never rescaled.  The reference
// is the same in the four lanes of a row.  Keys n_valid .. 31 of the block
// are masked.
template <int DH>
__device__ __forceinline__ void flash_compute(const char* cur, int n_valid,
                                              const bf16x8 (&qf)[Flash<DH>::RT][Flash<DH>::NST],
                                              f32x4 (&o)[Flash<DH>::RT][Flash<DH>::NT], float (&m_ref)[Flash<DH>::RT],
                                              float (&l_run)[Flash<DH>::RT], float qscale) {
  using FS = Flash<DH>;
  using MF = Mfma<bf16>;
  constexpr int NST = FS::NST, NT = FS::NT, RT = FS::RT;
  const int lane = threadIdx.x & 63, g = lane >> 4;
  // S^T = K q^T: all K fragments of the block are read from LDS first, then multiplied
  MF::frag kf[NST][2];
#pragma unroll
  for (int st = 0; st < NST; ++st)
#pragma unroll
    for (int kt = 0; kt < 2; ++kt) kf[st][kt] = *reinterpret_cast<const MF::frag*>(cur + ((kt * NST + st) * 64 + lane) * 16);
  f32x4 sc[RT][2];
#pragma unroll
  for (int rt = 0; rt < RT; ++rt) sc[rt][0] = sc[rt][1] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int st = 0; st < NST; ++st)
#pragma unroll
    for (int kt = 0; kt < 2; ++kt)
#pragma unroll
      for (int rt = 0; rt < RT; ++rt) sc[rt][kt] = MF::run(kf[st][kt], qf[rt][st], sc[rt][kt]);
  // the V^T fragments are read while the softmax runs
  MF::frag vf[NT];
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) vf[nt] = *reinterpret_cast<const MF::frag*>(cur + ((FS::KFR + nt) * 64 + lane) * 16);
  __builtin_amdgcn_sched_group_barrier(0x100, 2 * NST, 0);
  __builtin_amdgcn_sched_group_barrier(0x008, 2 * NST * RT, 0);
  __builtin_amdgcn_sched_group_barrier(0x100, NT, 0);

  if (n_valid < FS::KB) {
    asm volatile("" ::: "memory");  // a real branch: full blocks skip the masking
#pragma unroll
    for (int rt = 0; rt < RT; ++rt)
#pragma unroll
      for (int kt = 0; kt < 2; ++kt)
#pragma unroll
        for (int e = 0; e < 4; ++e) sc[rt][kt][e] = 8 * g + 4 * kt + e < n_valid ? sc[rt][kt][e] : -INFINITY;
  }
  MF::frag pb[RT];
#pragma unroll
  for (int rt = 0; rt < RT; ++rt) {
    float m = -INFINITY;
#pragma unroll
    for (int kt = 0; kt < 2; ++kt)
#pragma unroll
      for (int e = 0; e < 4; ++e) m = fmaxf(m, sc[rt][kt][e]);
    const float mx = row4_max(m) * qscale;  // finite: the block holds a valid key
    const bool over = mx > m_ref[rt] + FLASH_LIMIT;  // always on the row's first block (m_ref = -inf)
    if (__any(over)) {
      // 2^(-inf) = 0 on the first block, where the output and sum are still zero
      const float f = over ? __builtin_amdgcn_exp2f(m_ref[rt] - mx) : 1.f;
      l_run[rt] *= f;
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) o[rt][nt] *= f;
      m_ref[rt] = over ? mx : m_ref[rt];
    }
    // P^T as the B operand: slot j of the lane's eight <-> key 8g + j.  The
    // row sum adds the same bf16-rounded probabilities that weight V, so a
    // row dominated by one key returns that key's value row exactly.
    float sum = 0.f;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const bf16 lo = static_cast<bf16>(__builtin_amdgcn_exp2f(fmaf(sc[rt][0][e], qscale, -m_ref[rt])));
      const bf16 hi = static_cast<bf16>(__builtin_amdgcn_exp2f(fmaf(sc[rt][1][e], qscale, -m_ref[rt])));
      pb[rt][e] = lo;
      pb[rt][4 + e] = hi;
      sum += static_cast<float>(lo) + static_cast<float>(hi);
    }
    l_run[rt] += sum;
  }
  // O^T += V^T P^T
#pragma unroll
  for (int nt = 0; nt < NT; ++nt)
#pragma unroll
    for (int rt = 0; rt < RT; ++rt) o[rt][nt] = MF::run(vf[nt], pb[rt], o[rt][nt]);
}

// Work items (rollout, 128-row query tile, key range) in that order, T of
// them; the grid is T rounded up to a multiple of 8 workgroups.  The hardware
// hands workgroup i to XCD i % 8, so item (i % 8) * (grid / 8) + i / 8 puts
// consecutive items, which share a rollout's keys and values, in one XCD's L2.
template <int DH>
__global__ __launch_bounds__(512) void k_flash(AttnLaunch a, int S, int nqt, int qrows, void* part, float2* ml) {
  using FS = Flash<DH>;
  using MF = Mfma<bf16>;
  constexpr int NST = FS::NST, NT = FS::NT, RT = FS::RT, NS = FS::NS, LDW = FS::LDW;
  // one LDS array: the compiler then does not make the ring's LDS reads wait
  // for every outstanding direct-to-LDS load
  __shared__ __attribute__((aligned(1024))) char lds[NS * FS::STAGE];
  static_assert(FS::NW * 64 == 512, "launch bounds");

  const int item = (int)(blockIdx.x % 8) * (int)(gridDim.x / 8) + (int)(blockIdx.x / 8);
  if (item >= a.B * nqt * S) return;
  const int b = item / (nqt * S), split = item % S, qt = (item / S) % nqt;
  const int H = a.H, R = a.nH * H;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int g = lane >> 4, fr = lane & 15;
  const int pl = a.prefix_len[b];
  FlashSrc src;
  src.nbs = (H + FS::KB - 1) / FS::KB;
  src.H = H;
  src.pl = pl;
  const int nb = src.nbs + (pl + FS::KB - 1) / FS::KB;
  const int jb0 = (int)((int64_t)split * nb / S), jb1 = (int)((int64_t)(split + 1) * nb / S);
  const int nblk = jb1 - jb0;
  // this wave's first query row; tile qt holds rows [qt * qrows, (qt + 1) * qrows)
  const int row0 = qt * qrows + w * 16 * RT;

  // each split writes its (max, sum) even when it has no keys
  if (nblk == 0) {
    if (S > 1) {
      for (int t = threadIdx.x; t < qrows; t += FS::NW * 64) {
        const int r = qt * qrows + t;
        if (r < R) ml[((size_t)split * a.B + b) * R + r] = float2{-INFINITY, 0.f};
      }
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

  // query fragments (B operand of S^T): lane holds row fr of tile rt, dims st*32 + 8g .. + 8
  MF::frag qf[RT][NST];
  const bf16* qb = reinterpret_cast<const bf16*>(a.q) + (size_t)b * R * DH;
#pragma unroll
  for (int rt = 0; rt < RT; ++rt) {
    const int r = row0 + 16 * rt + fr;
#pragma unroll
    for (int st = 0; st < NST; ++st) qf[rt][st] = r < R ? MF::load(qb + (size_t)r * DH + st * 32 + 8 * g) : MF::frag{};
  }
  const bool active = row0 < R && 16 * RT * w < qrows;  // wave has query rows of this tile (uniform per wave)

  lds_t* ring = (lds_t*)lds;
  // valid keys of the blocks in the ring, by stage.  The first NS - 1 blocks
  // are issued whatever the range's length (a block past the range reads
  // zeros or other keys into a stage that is never multiplied), so that the
  // count of loads issued after the query fragments is fixed: waiting until
  // at most that many are pending means the fragments have landed, without
  // draining the ring.
  int nval[NS];
#pragma unroll
  for (int s = 0; s < NS - 1; ++s)
    nval[s] = flash_issue<DH>(ring + s * FS::STAGE, src, jb0 + s, koff, vaoff, vpoff, vst_ld, vpt_ld);
  flash_wait<(NS - 1) * LDW, false>();

  // log2-domain scores: s * log2(e) / sqrt(Dh)
  const float qscale = 1.4426950408889634f / sqrtf((float)DH);
  f32x4 o[RT][NT];
  float m_ref[RT], l_run[RT];
#pragma unroll
  for (int rt = 0; rt < RT; ++rt) {
    m_ref[rt] = -INFINITY;
    l_run[rt] = 0.f;
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) o[rt][nt] = f32x4{0.f, 0.f, 0.f, 0.f};
  }

  for (int j = 0; j < nblk; ++j) {
    const int slot = j % NS;
    int n_valid = 0;
#pragma unroll
    for (int s = 0; s < NS; ++s) n_valid = s == slot ? nval[s] : n_valid;
    // block j has landed once at most min(NS - 2, nblk - 1 - j) later blocks
    // of the range are pending (blocks issued past the range, when it is
    // shorter than NS - 1, only make this wait longer)
    const int later = nblk - 1 - j;
    if (later >= 2) flash_wait<2 * LDW, false>();
    else if (later == 1) flash_wait<LDW, false>();
    else flash_wait<0, false>();
    flash_fix<DH>(lds + slot * FS::STAGE, n_valid);
    // the V^T masks visible; every wave's part of block j landed; block j - 1
    // fully consumed, so its stage can take block j + NS - 1
    flash_wait<63, true>();
    __builtin_amdgcn_s_barrier();
    if (j + NS - 1 < nblk) {
      const int ns = (j + NS - 1) % NS;
      const int nv = flash_issue<DH>(ring + ns * FS::STAGE, src, jb0 + j + NS - 1, koff, vaoff, vpoff, vst_ld, vpt_ld);
#pragma unroll
      for (int s = 0; s < NS; ++s) nval[s] = s == ns ? nv : nval[s];
    }
    if (active) flash_compute<DH>(lds + slot * FS::STAGE, n_valid, qf, o, m_ref, l_run, qscale);
  }
  if (!active) return;

  // O^T: lane holds dims nt*16 + 4g .. + 4 of query row fr of each tile
  typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
#pragma unroll
  for (int rt = 0; rt < RT; ++rt) {
    float l = l_run[rt];
    l += __shfl_xor(l, 16, 64);
    l += __shfl_xor(l, 32, 64);
    const int r = row0 + 16 * rt + fr;
    if (r >= R) continue;
    const float rl = 1.0f / l;
    if (S == 1) {
      const int hn = r / H, i = r - hn * H;
      const size_t base = ((size_t)b * H + i) * (size_t)a.nH * DH + (size_t)hn * DH + 4 * g;
      if (a.out_f32) {
        float* out = reinterpret_cast<float*>(a.out) + base;
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) *reinterpret_cast<f32x4*>(out + nt * 16) = o[rt][nt] * rl;
      } else {
        bf16* out = reinterpret_cast<bf16*>(a.out) + base;
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) {
          const f32x4 v = o[rt][nt] * rl;
          *reinterpret_cast<bf16x4*>(out + nt * 16) = bf16x4{static_cast<bf16>(v[0]), static_cast<bf16>(v[1]),
                                                             static_cast<bf16>(v[2]), static_cast<bf16>(v[3])};
        }
      }
    } else {
      const size_t rowi = ((size_t)split * a.B + b) * R + r;
      bf16* out = reinterpret_cast<bf16*>(part) + rowi * DH + 4 * g;
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) {
        const f32x4 v = o[rt][nt] * rl;
        *reinterpret_cast<bf16x4*>(out + nt * 16) = bf16x4{static_cast<bf16>(v[0]), static_cast<bf16>(v[1]),
                                                           static_cast<bf16>(v[2]), static_cast<bf16>(v[3])};
      }
      if (g == 0) ml[rowi] = float2{m_ref[rt], l};
    }
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
  const int KB = 32;
  const int nqt = (nH * H + 127) / 128;
  const int nb = (H + KB - 1) / KB + (P + KB - 1) / KB;
  int s = (n_cu + B * nqt - 1) / (B * nqt);
  s = s < nb / 2 ? s : nb / 2;
  s = s < FLASH_MAX_SPLITS ? s : FLASH_MAX_SPLITS;
  return s > 1 ? s : 1;
}

template <int DH>
static hipError_t launch_flash_t(const AttnLaunch& a, int S, hipStream_t s) {
  // ceil(rows / 128) tiles per rollout, the rows spread evenly in whole 16-row wave tiles (400 rows: four
  // tiles of 112 instead of 128 + 128 + 128 + 16, so that the critical tiles keep seven waves busy)
  const int R = a.nH * a.H;
  const int nqt = (R + Flash<DH>::QT - 1) / Flash<DH>::QT;
  const int qrows = ((R + nqt - 1) / nqt + 15) / 16 * 16;
  const size_t rows = (size_t)a.B * a.nH * a.H;
  // partial outputs (bf16) then (max, sum) pairs, inside the opart scratch
  void* part = a.opart;
  float2* ml = reinterpret_cast<float2*>(reinterpret_cast<char*>(a.opart) + (size_t)S * rows * DH * 2);
  const int items = a.B * nqt * S;
  JPI_LAUNCH((k_flash<DH>), dim3((items + 7) / 8 * 8), dim3(Flash<DH>::NW * 64), 0, s, a.ev_start,
             S == 1 ? a.ev_stop : (hipEvent_t) nullptr, a, S, nqt, qrows, part, ml);
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
