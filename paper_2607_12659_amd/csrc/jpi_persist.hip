// Persistent single-launch denoise for small batches (M = batch * horizon <= 64,
// bf16 weights).  One workgroup per compute unit runs every Euler step of the
// flow-matching loop and every layer of the action expert (paper: Appendix
// "Model Architecture of pi series Models" for the expert, Section "System
// Design" for running all denoising steps as one unrolled unit).  Phases are
// ordered by per-workgroup completion flags: before a phase in which it has
// work, a workgroup waits only for the workgroups that produce that work's
// inputs (see phase_deps), so the per-head and per-slice chains of a layer
// overlap.
//
// Phases of one layer (items are distributed over the workgroups):
//   0 QKV     adaRMSNorm'd activations y x packed [q|k|v] weights, RoPE
//             epilogue; the action rows' V goes into the transposed prefix V
//             buffer right after each rollout's valid prefix
//   1 ATTN    (rollout, head, 32-key chunk) items over prefix + action keys:
//             per-chunk max, probability sum and output row / sum (bf16)
//   2 COMB    chunk combine per (rollout, head, query row) -> o
//   3 OPROJ   o x W_o, split-K slices -> part
//   4 ROWS    row owner: residual += gate * sum of slices (polled, not
//             flagged); MLP adaRMSNorm -> y
//   5 GATEUP  y x [gate|up], GeGLU epilogue -> z
//   6 DOWN    z x W_down, split-K slices -> part
//   7 ROWS    row owner: residual update + next layer's attention norm, or
//             (last layer) final norm, action-out projection, Euler update
//             of x and the next step's in-projection + first norm
//
// Code size: every phase has exactly one call site (the kernel loops over a
// phase index) and the four GEMM phases share one GEMM body, so the kernel
// stays within the instruction cache; a phase whose code was evicted since
// the previous layer pays instruction-fetch latency on every new cache line.
//
// Operand layout: every matrix that feeds an MFMA (the layer weights, a
// fragment-ordered copy made by the host, and the activations y, o, z, q
// written by the phases) is stored as 16x32 blocks in (row group, k step)
// order, each block holding the 64 lanes' 8-element fragments in lane order.
// A wave then loads a whole fragment as one contiguous kilobyte; row-major
// fragments would touch half of sixteen cache lines per instruction, which
// halves the load throughput of a compute unit.  Activation matrices are
// padded to 64 rows; rows >= M are never written and stay zero.
//
// Row ownership: workgroup m < M owns action row m.  Its residual row and
// b_in live in LDS for the whole launch and x[m][a] lives in a register of
// thread a.
//
// Memory model: data that one workgroup writes and another reads within the
// launch (activations, slices, attention partials, the action rows' K and V,
// completion flags) is stored and loaded with device-scope coherent buffer
// accesses (cache policy sc1); a completion flag is stored only after
// s_waitcnt vmcnt(0) confirms the workgroup's stores.  The split-K slices are
// the exception: each word has one reader (its row owner), which polls the
// words themselves until they leave the EMPTY pattern and writes EMPTY back,
// so their producers neither wait for store confirmation nor store a flag
// (the confirmation round trip and the flag hop leave the critical path).
// No agent-scope fences are used (on gfx950 they serialise across the chip).
// Weights, the prefix K, the prefix part of the transposed V, the modulation
// table and the RoPE table are read-only during the launch and use plain
// loads.
//
// Every wait is bounded: a flag wait gives up after a.spin_limit unsuccessful
// polls (default SPIN_LIMIT), a row owner's slice wait after SPIN_LIMIT polls
// or as soon as its workgroup gave up elsewhere. Giving up records an error
// word and stops all later waits of the workgroup, so a launch always
// terminates; the host reports the error from jpi_sync. (A variable bound in
// the slice wait costs the kernel register spills; the fixed one does not.)
#include <algorithm>

#include "jpi_device.h"
#include "jpi_internal.h"

namespace jpi {

namespace {

constexpr int PT = 256;  // threads per workgroup (one wave per SIMD)
constexpr int NWV = PT / 64;
constexpr int CPOL_DEV = 16;  // sc1: device-scope coherent access
constexpr int KC = 32;        // keys per attention chunk
constexpr int MAX_CH = 128;   // attention chunks per rollout
constexpr unsigned SPIN_LIMIT = 1u << 21;
constexpr int SMEM_BYTES = 42496;      // per-phase scratch (attention staging at Dh = 256)
constexpr int MAX_W = 2048;            // model width held in LDS by a row owner
constexpr int WT_STEPS = 32;           // weight tile in LDS: 32-wide k steps of a 32-row tile (64 KB)
constexpr int RMAX_S = 16;             // split-K slices summed by the row phases
constexpr int MAX_GRID = 256;          // completion flags are polled as 64 lanes x 4 lines
constexpr int FLAG_STRIDE = 32;        // words between completion flags: one 128-byte line per workgroup
constexpr int FLAG_WORDS = MAX_GRID * FLAG_STRIDE;
constexpr int CPT = 16;    // combine: chunks per thread per round trip
constexpr int OUT_G = 16;  // action-out projection: 16-byte weight granules per thread
#ifndef A_BATCH
#define A_BATCH 4  // k steps of activation fragments per wave in flight (measured best)
#endif
// Trace build (-DJPI_PERSIST_TRACE=1, never the default): every workgroup
// stores the real-time counter at its start and at the end of every phase,
// trace[workgroup][1 + phase], so that the critical path of each link can be
// reconstructed on the host.
#ifndef JPI_PERSIST_TRACE
#define JPI_PERSIST_TRACE 0
#endif

enum : int { EPI_QKV = 0, EPI_GEGLU = 1, EPI_SLICE = 2 };

typedef unsigned u32;
typedef u32 u32x2 __attribute__((ext_vector_type(2)));
typedef u32 u32x4 __attribute__((ext_vector_type(4)));
typedef __amdgpu_buffer_rsrc_t rsrc_t;
typedef __attribute__((address_space(3))) char lds_t;  // LDS byte pointer (direct-to-LDS loads)
typedef __attribute__((address_space(3))) const bf16x8 lds_frag;

// Buffer resource over [base, base + bytes): loads beyond the range return
// zero and stores beyond it are dropped.
__device__ __forceinline__ rsrc_t rsrc(const void* base, u32 bytes = 0x7fffffffu) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), 0, (int)bytes, 0x00020000);
}
__device__ __forceinline__ u32x4 ld16(rsrc_t r, u32 off) {
  return __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, CPOL_DEV);
}
// Bit casts take scalars by value: with this compiler, __builtin_bit_cast
// applied directly to an element of an ext_vector_type value (v[i]) reads
// element 0 whatever the index.
__device__ __forceinline__ u32 f2u(float v) { return __builtin_bit_cast(u32, v); }
__device__ __forceinline__ float u2f(u32 v) { return __builtin_bit_cast(float, v); }
__device__ __forceinline__ u32x2 ld8(rsrc_t r, u32 off) {
  return __builtin_amdgcn_raw_buffer_load_b64(r, off, 0, CPOL_DEV);
}
__device__ __forceinline__ float2 ld8f(rsrc_t r, u32 off) {
  return __builtin_bit_cast(float2, __builtin_amdgcn_raw_buffer_load_b64(r, off, 0, CPOL_DEV));
}
// A polling load: the empty asm with a memory clobber keeps the compiler from
// treating the load as loop-invariant and hoisting it out of the wait loop.
__device__ __forceinline__ u32 poll4(rsrc_t r, u32 off) {
  asm volatile("" ::: "memory");
  return __builtin_amdgcn_raw_buffer_load_b32(r, off, 0, CPOL_DEV);
}
// A 16-byte polling load (see poll4).
__device__ __forceinline__ u32x4 poll16(rsrc_t r, u32 off) {
  asm volatile("" ::: "memory");
  return __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, CPOL_DEV);
}
// Split-K slices travel without completion flags: every 32-bit word of the
// slice buffer holds EMPTY until its producer writes a value, and the row
// owner that reads it (its only reader) writes EMPTY back.  Producers
// canonicalise NaN, so a value never has the EMPTY pattern.
constexpr u32 EMPTY = 0xffffffffu;
__device__ __forceinline__ bool has_empty(u32x4 v) {
  return v[0] == EMPTY || v[1] == EMPTY || v[2] == EMPTY || v[3] == EMPTY;
}
__device__ __forceinline__ u32 f2u_value(float v) { return v == v ? __builtin_bit_cast(u32, v) : 0x7fc00000u; }

__device__ __forceinline__ void st4(rsrc_t r, u32 off, u32 v) { __builtin_amdgcn_raw_buffer_store_b32(v, r, off, 0, CPOL_DEV); }
__device__ __forceinline__ void st16(rsrc_t r, u32 off, u32x4 v) {
  __builtin_amdgcn_raw_buffer_store_b128(v, r, off, 0, CPOL_DEV);
}
__device__ __forceinline__ void st8(rsrc_t r, u32 off, u32x2 v) {
  __builtin_amdgcn_raw_buffer_store_b64(v, r, off, 0, CPOL_DEV);
}
__device__ __forceinline__ u32 bf16_bits(float v) { return __builtin_bit_cast(unsigned short, static_cast<bf16>(v)); }
__device__ __forceinline__ void st_bf16(rsrc_t r, u32 off, float v) {
  __builtin_amdgcn_raw_buffer_store_b16((unsigned short)bf16_bits(v), r, off, 0, CPOL_DEV);
}
__device__ __forceinline__ u32x2 pack4_bf16(f32x4 v) {
  return u32x2{bf16_bits(v[0]) | (bf16_bits(v[1]) << 16), bf16_bits(v[2]) | (bf16_bits(v[3]) << 16)};
}
__device__ __forceinline__ float bf16_lo(u32 w) { return u2f(w << 16); }
__device__ __forceinline__ float bf16_hi(u32 w) { return u2f(w & 0xffff0000u); }
__device__ __forceinline__ f32x4 as_f4(u32x4 v) { return __builtin_bit_cast(f32x4, v); }

// Element offset of (row, k) in the fragment-ordered layout of a bf16 matrix
// with KS = K / 32 k steps.
__device__ __forceinline__ u32 frag_off(int row, int k, int KS) {
  return (u32)((((row >> 4) * KS + (k >> 5)) * 64 + (row & 15) + 16 * ((k & 31) >> 3)) * 8 + (k & 7));
}

// Fixed-order sum over the waves of a workgroup.
__device__ __forceinline__ float block_sum_wg(float v, float* red) {
  v = wave_sum(v);
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  __syncthreads();
  if (lane == 0) red[w] = v;
  __syncthreads();
  float t = red[0];
#pragma unroll
  for (int i = 1; i < NWV; ++i) t += red[i];
  return t;
}

struct GemmJob {
  const void* A;  // activations, fragment-ordered [64][K] bf16
  const bf16* w;  // weights, fragment-ordered [N][K] bf16
  int K;          // reduction length
  int tiles;      // N / 32
  int S;          // split-K slices
  int kind;       // EPI_*
};

// Direct-to-LDS loads of k steps [ks0, ks0 + nk) of row groups rg0, rg0 + 1 of
// the fragment-ordered matrix W (KS k steps per row group) into the tile
// [2][nk][64 lanes][16 B]; waves w0 .. NWV-1 take the 1 KB blocks round-robin.
__device__ __forceinline__ void load_wtile(lds_t* lds, const bf16* W, int KS, int rg0, int ks0, int nk, int w0) {
  const int lane = threadIdx.x & 63, wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  if (wave < w0) return;
  for (int i = wave - w0; i < 2 * nk; i += NWV - w0) {
    const int rgl = i >= nk, kk = i - rgl * nk;
    __builtin_amdgcn_global_load_lds(W + ((size_t)((rg0 + rgl) * KS + ks0 + kk) * 64 + lane) * 8, lds + i * 1024, 16,
                                     0, 0);
  }
}

// trace build: the first two stamps of the current phase (thread 0)
__shared__ unsigned long long s_note[2];

// Trace build only.  Slot 0 of trace[workgroup][...] is the workgroup's
// start; phase ph has slots 1 + 3 ph + {0: its producers seen, 1: its
// operands loaded, 2: its end}.  A workgroup with no work in a phase records
// the phase's end time in all three.  s_note holds the first two stamps of
// the current phase until the phase ends.
__device__ __forceinline__ void trace_start(const PersistArgs& a, unsigned long long* s_note) {
  if (JPI_PERSIST_TRACE && a.trace && threadIdx.x == 0) {
    a.trace[(size_t)blockIdx.x * a.trace_slots] = __builtin_amdgcn_s_memrealtime();
    s_note[0] = s_note[1] = 0ull;
  }
}
// kind 0: the producers' flags were seen; kind 1: the phase's operands are loaded
__device__ __forceinline__ void trace_note(unsigned long long* s_note, int kind) {
  if (JPI_PERSIST_TRACE && threadIdx.x == 0 && s_note[kind] == 0ull) s_note[kind] = __builtin_amdgcn_s_memrealtime();
}
__device__ __forceinline__ void trace_end(const PersistArgs& a, unsigned long long* s_note, int ph) {
  if (JPI_PERSIST_TRACE && a.trace && threadIdx.x == 0 && 3 + 3 * ph < a.trace_slots) {
    const unsigned long long t = __builtin_amdgcn_s_memrealtime();
    unsigned long long* row = a.trace + (size_t)blockIdx.x * a.trace_slots + 1 + 3 * ph;
    const unsigned long long w = s_note[0] ? s_note[0] : t;
    row[0] = w;
    row[1] = s_note[1] ? s_note[1] : w;
    row[2] = t;
    s_note[0] = s_note[1] = 0ull;
  }
}

// Phase completion flags.  After phase ph a workgroup confirms its stores
// (s_waitcnt vmcnt(0)) and writes ph + 2 into its own 128-byte flag line;
// the values only grow within a launch.  A workgroup that has work in phase
// ph first waits until the flags of the workgroups that produce its inputs
// reach ph + 1 (they finished phase ph - 1).  Producer sets are one or two
// ranges of workgroup indices; the row phases, which reduce the split-K slices
// of every workgroup, wait for all of them.  Buffers are reused only after a
// row phase that (through the producer chains) follows every reader of the
// previous contents.
struct Deps {
  int lo0, hi0, lo1, hi1;  // workgroups [lo0, hi0) and [lo1, hi1)
};
__device__ __forceinline__ Deps deps_none() { return Deps{0, 0, 0, 0}; }
__device__ __forceinline__ Deps deps_all() { return Deps{0, (int)gridDim.x, 0, 0}; }
// workgroups that run items [i0, i1) of a phase whose item it runs on
// workgroup it % grid
__device__ __forceinline__ Deps deps_items(int i0, int i1) {
  const int G = gridDim.x;
  if (i1 - i0 >= G) return deps_all();
  const int lo = i0 % G, hi = lo + (i1 - i0);
  return hi <= G ? Deps{lo, hi, 0, 0} : Deps{lo, G, 0, hi - G};
}

// Wave 0 polls the producers' flags (lane l covers the l-th, l+64-th, ...
// workgroup of the two ranges) until all reach `value`; waves 1..3 meanwhile
// start the direct-to-LDS loads of the first weight tile of a GEMM phase.
// Every wait is bounded: past a.spin_limit polls the workgroup records an error
// word and stops waiting, so the launch always terminates.
__device__ __forceinline__ void wait_producers(const PersistArgs& a, const Deps& d, u32 value, u32* s_abort,
                                               bool tile, const GemmJob& j, lds_t* wt) {
  if (tile && (int)blockIdx.x < j.tiles * j.S) {
    const int it = blockIdx.x, t = it % j.tiles, sl = it / j.tiles, nk_item = j.K / j.S / 32;
    load_wtile(wt, j.w, j.K / 32, 2 * t, sl * nk_item, min(WT_STEPS, nk_item), 1);
  }
  const int n0 = d.hi0 - d.lo0, n = n0 + (d.hi1 - d.lo1);
  if (threadIdx.x < 64 && n > 0 && *s_abort == 0u) {
    const rsrc_t rf = rsrc(a.flags);
    u32 off[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int i = (int)threadIdx.x + 64 * u;
      off[u] = (u32)(i < n0 ? d.lo0 + i : d.lo1 + (i - n0)) * (FLAG_STRIDE * 4u);
    }
    // flags only grow: a flag seen at `value` is not polled again, so the
    // poll traffic shrinks to the producers that are still working
    u32 pend = 0u;
#pragma unroll
    for (int u = 0; u < 4; ++u) pend |= ((int)threadIdx.x + 64 * u < n ? 1u : 0u) << u;
    for (u32 spins = 0;; ++spins) {
      u32 f[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) f[u] = (pend >> u) & 1u ? poll4(rf, off[u]) : value;
#pragma unroll
      for (int u = 0; u < 4; ++u)
        if (f[u] >= value) pend &= ~(1u << u);
      if (__all(pend == 0u)) break;
      if (spins + 1 >= s_abort[1]) {
        if (threadIdx.x == 0) {
          *s_abort = 1u;
          st4(rsrc(a.err), 0, 1u);
        }
        break;
      }
    }
  }
  asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");  // s_abort
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
  trace_note(s_note, 0);
}

// End of phase ph: every wave's stores are complete, then the flag.
__device__ __forceinline__ void phase_done(const PersistArgs& a, u32 value) {
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  __syncthreads();
  if (threadIdx.x == 0) st4(rsrc(a.flags), blockIdx.x * (FLAG_STRIDE * 4u), value);
}

// ---------------------------------------------------------------------------
// GEMM items: 32 output columns (two 16-row groups of W) x all 64 padded rows
// x a K range of 32-wide k steps, split evenly over the waves.  The weight
// part lives in the LDS tile (filled by direct-to-LDS loads: for a
// workgroup's first item while it waits for its producers, otherwise here);
// A (fragment-ordered, read coherently) contributes its first `mgroups`
// 16-row groups.  K ranges longer than the tile are processed in chunks.
// ---------------------------------------------------------------------------
__device__ __forceinline__ void gemm_chunk(rsrc_t ra, int mgroups, int KS, int ksA, const lds_t* wt, int nk,
                                           f32x4 (&acc)[4][2]) {
  using MF = Mfma<bf16>;
  constexpr int BATCH = A_BATCH;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  // Every workgroup reads the same activation rows.  The k range of each wave
  // and the order of its k steps are rotated by the workgroup index so that
  // the workgroups do not request the same lines at the same moment.
  const int nsub = nk / NWV, kk0 = ((wave + (int)blockIdx.x) & (NWV - 1)) * nsub;
  const int rot = nsub > 0 ? ((int)blockIdx.x >> 2) % nsub : 0;
  const u32 aoff = (u32)((ksA + kk0) * 64 + lane) * 16u;
  const u32 astep = (u32)KS * 1024u;  // bytes per 16-row group of A
  for (int s0 = 0; s0 < nsub; s0 += BATCH) {
    MF::frag af[BATCH][4];
#pragma unroll
    for (int c = 0; c < BATCH; ++c) {
      int kc = s0 + c + rot;
      kc = kc >= nsub ? kc - nsub : kc;
#pragma unroll
      for (int a = 0; a < 4; ++a)
        af[c][a] = (s0 + c < nsub && a < mgroups)
                       ? __builtin_bit_cast(MF::frag, ld16(ra, aoff + a * astep + (u32)kc * 1024u))
                       : MF::frag{};
    }
    if (s0 == 0) {  // every wave's part of the tile has landed
      asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
      __syncthreads();
      trace_note(s_note, 1);
    }
#pragma unroll
    for (int c = 0; c < BATCH; ++c) {
      if (s0 + c >= nsub) break;
      int kc = s0 + c + rot;
      kc = kc >= nsub ? kc - nsub : kc;
      const int kk = kk0 + kc;
      const MF::frag w0 = *(lds_frag*)(wt + (kk * 64 + lane) * 16);
      const MF::frag w1 = *(lds_frag*)(wt + ((nk + kk) * 64 + lane) * 16);
#pragma unroll
      for (int a = 0; a < 4; ++a) {
        acc[a][0] = MF::run(af[c][a], w0, acc[a][0]);
        acc[a][1] = MF::run(af[c][a], w1, acc[a][1]);
      }
    }
  }
}


// ---- phases 0, 3, 5, 6: GEMM with a per-kind epilogue ----------------------
__device__ __forceinline__ void phase_gemm(const PersistArgs& a, const GemmJob& j, int l, lds_t* wt, char* smem) {
  f32x4* red = reinterpret_cast<f32x4*>(smem);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, fr = lane & 15;
  const int Dh = a.Dh, half = Dh / 2, H = a.H, nH = a.nH, qcols = nH * Dh, M = a.M, Wd = a.W;
  const int klen = j.K / j.S, KS = j.K / 32, nk_item = klen / 32, mgroups = (M + 15) / 16;
  const rsrc_t ra = rsrc(j.A, (u32)(64 * j.K * 2));
  const rsrc_t rq = rsrc(a.q), rk = rsrc(a.ks), rz = rsrc(a.z), rp = rsrc(a.part);
  const rsrc_t rv = rsrc(reinterpret_cast<const bf16*>(a.vpt) + (size_t)l * a.vpt_lstride);
  for (int it = blockIdx.x; it < j.tiles * j.S; it += gridDim.x) {
    const int t = it % j.tiles, s = it / j.tiles;
    const int col = t * 32 + fr;  // column of lo; hi is col + 16
    // QKV: q/k columns are packed so that a RoPE pair (d, d + Dh/2) sits in
    // lo/hi of one lane.  The rotation factors and the prefix lengths do not
    // depend on the GEMM, so their loads are issued first.
    const bool qkv = j.kind == EPI_QKV;
    const bool roped = qkv && col < qcols + Dh;
    const int hn = col < qcols ? col / Dh : -1;
    const int within = col < qcols ? col - hn * Dh : col - qcols;
    const int d = (within >> 5) * 16 + (within & 15);
    float2 cs[4];
    int plv[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int row = wave * 16 + (lane >> 4) * 4 + e;
      cs[e] = (roped && row < M) ? a.rope[(size_t)row * half + d] : float2{1.f, 0.f};
      plv[e] = (qkv && !roped && row < M) ? a.prefix_len[row / H] : 0;
    }
    f32x4 acc[4][2];
#pragma unroll
    for (int q = 0; q < 4; ++q) acc[q][0] = acc[q][1] = f32x4{0.f, 0.f, 0.f, 0.f};
    for (int cs0 = 0; cs0 < nk_item; cs0 += WT_STEPS) {
      const int nk = min(WT_STEPS, nk_item - cs0);
      if (it != (int)blockIdx.x || cs0 != 0) {  // not loaded during the wait
        __syncthreads();                         // every wave is done with the tile
        load_wtile(wt, j.w, KS, 2 * t, s * nk_item + cs0, nk, 0);
      }
      gemm_chunk(ra, mgroups, KS, s * nk_item + cs0, wt, nk, acc);
    }
    // reduce the four waves' K partial sums; wave w keeps m-subtile w
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      red[((wave * 4 + q) * 2 + 0) * 64 + lane] = acc[q][0];
      red[((wave * 4 + q) * 2 + 1) * 64 + lane] = acc[q][1];
    }
    __syncthreads();
    f32x4 lo = red[((0 * 4 + wave) * 2 + 0) * 64 + lane];
    f32x4 hi = red[((0 * 4 + wave) * 2 + 1) * 64 + lane];
#pragma unroll
    for (int v = 1; v < NWV; ++v) {
      lo += red[((v * 4 + wave) * 2 + 0) * 64 + lane];
      hi += red[((v * 4 + wave) * 2 + 1) * 64 + lane];
    }
    __syncthreads();  // red and the tile are reused by the next item
    // Slices and z leave through LDS (the freed reduction area, a region per
    // wave) so that each store instruction writes whole lines: a slice row's
    // 32 columns are one 128-byte line, a wave's 16 x 16 z values one half of
    // a fragment block (512 contiguous bytes).  Rows >= M are not stored.
    char* sw = smem + wave * 16 * 144;
    if (j.kind == EPI_SLICE) {
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int rl = (lane >> 4) * 4 + e;
        *reinterpret_cast<u32*>(sw + rl * 144 + fr * 4) = f2u_value(lo[e]);
        *reinterpret_cast<u32*>(sw + rl * 144 + 64 + fr * 4) = f2u_value(hi[e]);
      }
#pragma unroll
      for (int k = 0; k < 2; ++k) {
        const int rl = k * 8 + (lane >> 3), row = wave * 16 + rl;
        if (row < M)
          st16(rp, (u32)(((size_t)s * M + row) * Wd + t * 32 + (lane & 7) * 4) * 4u,
               *reinterpret_cast<const u32x4*>(sw + rl * 144 + (lane & 7) * 16));
      }
      continue;
    }
    if (j.kind == EPI_GEGLU) {  // gate/up rows interleaved in 16-row groups: z column t * 16 + fr
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const u32 v = bf16_bits(gelu_tanh(lo[e]) * hi[e]);
        const u32 pair = v | (__shfl_xor(v, 1, 64) << 16);  // columns fr, fr + 1 (fr even)
        if ((fr & 1) == 0) *reinterpret_cast<u32*>(sw + ((lane >> 4) * 4 + e) * 48 + fr * 2) = pair;
      }
      const int rl = lane & 15, row = wave * 16 + rl;
      if (lane < 32 && row < M)
        st16(rz, frag_off(row, t * 16 + (lane >> 4) * 8, a.F / 32) * 2u,
             *reinterpret_cast<const u32x4*>(sw + rl * 48 + (lane >> 4) * 16));
      continue;
    }
    // q columns: the tile holds 16 RoPE pairs (d, d + Dh/2), d = 16 jq + fr.
    // When the wave's 16 rows are rows of one rollout starting at a multiple
    // of 16 (one rollout, or H % 16 == 0) they form two half fragment blocks
    // of that rollout's q, stored whole through LDS.
    if (qkv && hn >= 0 && (a.B == 1 || (H & 15) == 0)) {
      const int jq = (within >> 5);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float r_lo = lo[e] * cs[e].x - hi[e] * cs[e].y;
        const float r_hi = lo[e] * cs[e].y + hi[e] * cs[e].x;
        const u32 vl = bf16_bits(r_lo), vh = bf16_bits(r_hi);
        const u32 pl2 = vl | (__shfl_xor(vl, 1, 64) << 16), ph2 = vh | (__shfl_xor(vh, 1, 64) << 16);
        char* rowp = sw + ((lane >> 4) * 4 + e) * 80;
        if ((fr & 1) == 0) {
          *reinterpret_cast<u32*>(rowp + fr * 2) = pl2;
          *reinterpret_cast<u32*>(rowp + 32 + fr * 2) = ph2;
        }
      }
      const int part = lane >> 5, r = lane & 15, cc = (lane >> 4) & 1;
      const int row = wave * 16 + r, b = row / H, i = row - b * H;
      if (row < M)
        st16(rq, ((u32)(((size_t)b * nH + hn) * 64 * Dh) + frag_off(i, 16 * jq + part * half + cc * 8, Dh / 32)) * 2u,
             *reinterpret_cast<const u32x4*>(sw + r * 80 + part * 32 + cc * 16));
      continue;
    }
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int row = wave * 16 + (lane >> 4) * 4 + e;
      if (row >= M) continue;
      {
        const int b = row / H, i = row - b * H;
        if (roped) {
          const float r_lo = lo[e] * cs[e].x - hi[e] * cs[e].y;
          const float r_hi = lo[e] * cs[e].y + hi[e] * cs[e].x;
          if (hn >= 0) {  // q: fragment-ordered [b][head][64 rows][Dh]
            const u32 base = (u32)(((size_t)b * nH + hn) * 64 * Dh);
            st_bf16(rq, (base + frag_off(i, d, Dh / 32)) * 2u, r_lo);
            st_bf16(rq, (base + frag_off(i, d + half, Dh / 32)) * 2u, r_hi);
          } else {  // action K rows: row-major [b][H][Dh]
            const u32 base = (u32)(((size_t)b * H + i) * Dh);
            st_bf16(rk, (base + d) * 2u, r_lo);
            st_bf16(rk, (base + d + half) * 2u, r_hi);
          }
        } else {
          // V of action row i: transposed prefix V buffer at key prefix_len + i
          const int dv = col - qcols - Dh;
          const u32 off = (u32)((size_t)b * a.vpt_bstride + (size_t)dv * a.vpt_dstride + plv[e] + i) * 2u;
          st_bf16(rv, off, lo[e]);
          st_bf16(rv, off + (u32)(16 * a.vpt_dstride * 2), hi[e]);
        }
      }
    }
  }
}

// ---- phase 1: attention chunk partials ----------------------------------------
template <int DH>
__device__ __forceinline__ void phase_attn(const PersistArgs& a, int l, char* smem, const Deps& deps, u32 value,
                                           u32* s_abort, lds_t* wt, char* stage) {
  // The workgroup stages the chunk's K and V^T in LDS with coalesced loads
  // (one workgroup barrier); after that every wave works alone on its 16 query rows,
  // with P and the partial output in registers.
  using MF = Mfma<bf16>;
  constexpr int PAD = 8, LDK = DH + PAD, LDV = KC + PAD;
  constexpr int NST = DH / MF::KSUB, NJ = KC / 16, NT = DH / 16;
  constexpr int KCH = KC * (DH / 8) / PT, VCH = DH * (KC / 8) / PT;
  static_assert(KCH >= 1 && VCH >= 1, "chunk too small for the workgroup");
  static_assert(KC == MF::KSUB, "one P.V step per chunk");
  static_assert((KC * LDK + DH * LDV) * 2 <= SMEM_BYTES, "attention LDS");
  static_assert(NWV * 16 * (DH * 2 + 16) <= WT_STEPS * 2 * 1024, "attention output staging");
  bf16* Ks = reinterpret_cast<bf16*>(smem);
  bf16* Vt = Ks + KC * LDK;
  const int H = a.H, nH = a.nH, C = a.C;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int fr = lane & 15, fk = (lane >> 4) * MF::KPL;
  const int n_items = a.B * nH * C;
  const bf16* kpl = reinterpret_cast<const bf16*>(a.kp) + (size_t)l * a.kp_lstride;
  const bf16* vpl = reinterpret_cast<const bf16*>(a.vpt) + (size_t)l * a.vpt_lstride;
  const rsrc_t rv = rsrc(vpl), rks = rsrc(a.ks), rq = rsrc(a.q), ro = rsrc(a.opart), rml = rsrc(a.ml);
  bool waited = false;
  for (int it = blockIdx.x; it < n_items; it += gridDim.x) {
    const int c = it % C, hn = (it / C) % nH, b = it / (C * nH);
    const int pl = a.prefix_len[b];
    const int nkeys = pl + H;
    const int kbase = c * KC;
    if (kbase >= nkeys) continue;  // uniform across the workgroup; combine skips it
    const bf16* kp = kpl + (size_t)b * a.kp_bstride;
    const bf16* vb = vpl + (size_t)b * a.vpt_bstride;
    const u32 vboff = (u32)((size_t)b * a.vpt_bstride * 2);
    // The prefix keys and values were bound before the launch (plain loads):
    // they are loaded before waiting for this layer's QKV tiles.  The action
    // keys and values and q come from those tiles (coherent loads, after the
    // wait); keys past the end are zeroed so that stale memory never meets a
    // zero probability.
    u32x4 kr[KCH], vr[VCH];
#pragma unroll
    for (int u = 0; u < KCH; ++u) {
      const int e = tid + u * PT, r = e / (DH / 8), cc = e - r * (DH / 8);
      const int key = kbase + r;
      kr[u] = key < pl ? *reinterpret_cast<const u32x4*>(kp + (size_t)key * DH + cc * 8) : u32x4{0u, 0u, 0u, 0u};
    }
#pragma unroll
    for (int u = 0; u < VCH; ++u) {
      const int e = tid + u * PT, d = e / (KC / 8), kc = e - d * (KC / 8);
      const int key0 = kbase + kc * 8;
      vr[u] = key0 + 8 <= pl ? *reinterpret_cast<const u32x4*>(vb + (size_t)d * a.vpt_dstride + key0)
                             : u32x4{0u, 0u, 0u, 0u};
    }
    if (!waited) {  // (the producers of every item of this workgroup)
      wait_producers(a, deps, value, s_abort, false, GemmJob{}, wt);
      waited = true;
    }
#pragma unroll
    for (int u = 0; u < KCH; ++u) {
      const int e = tid + u * PT, r = e / (DH / 8), cc = e - r * (DH / 8);
      const int key = kbase + r;
      if (key >= pl && key < nkeys) kr[u] = ld16(rks, (u32)((((size_t)b * H + (key - pl)) * DH + cc * 8) * 2));
    }
#pragma unroll
    for (int u = 0; u < VCH; ++u) {
      const int e = tid + u * PT, d = e / (KC / 8), kc = e - d * (KC / 8);
      const int key0 = kbase + kc * 8;
      if (key0 + 8 > pl && key0 < nkeys) {
        u32x4 v = ld16(rv, vboff + (u32)(((size_t)d * a.vpt_dstride + key0) * 2));
        const int n_ok = nkeys - key0;
#pragma unroll
        for (int q = 0; q < 4; ++q)
          v[q] &= (2 * q < n_ok ? 0x0000ffffu : 0u) | (2 * q + 1 < n_ok ? 0xffff0000u : 0u);
        vr[u] = v;
      }
    }
    // wave w: query rows w*16 .. +16 of head hn (fragment-ordered; rows >= H are zero)
    MF::frag qf[NST];
    const u32 qoff = (u32)(((((size_t)b * nH + hn) * 4 + w) * NST) * 64 + lane) * 16u;
#pragma unroll
    for (int st = 0; st < NST; ++st)
      qf[st] = w * 16 < H ? __builtin_bit_cast(MF::frag, ld16(rq, qoff + (u32)st * 1024u)) : MF::frag{};
#pragma unroll
    for (int u = 0; u < KCH; ++u) {
      const int e = tid + u * PT, r = e / (DH / 8), cc = e - r * (DH / 8);
      *reinterpret_cast<u32x4*>(&Ks[r * LDK + cc * 8]) = kr[u];
    }
#pragma unroll
    for (int u = 0; u < VCH; ++u) {
      const int e = tid + u * PT, d = e / (KC / 8), kc = e - d * (KC / 8);
      *reinterpret_cast<u32x4*>(&Vt[d * LDV + kc * 8]) = vr[u];
    }
    __syncthreads();
    trace_note(s_note, 1);
    // S^T = K q^T with the operands swapped, so that a lane holds one query
    // row (fr) and keys jj*16 + 4g + e (g = lane / 16): the softmax of a row
    // needs only the four lanes that share fr, and P stays in registers as
    // the B operand of O^T = V^T P^T.
    const int g = lane >> 4;
    f32x4 sc[NJ];
#pragma unroll
    for (int jj = 0; jj < NJ; ++jj) sc[jj] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int st = 0; st < NST; ++st)
#pragma unroll
      for (int jj = 0; jj < NJ; ++jj)
        sc[jj] = MF::run(MF::load(&Ks[(jj * 16 + fr) * LDK + st * MF::KSUB + fk]), qf[st], sc[jj]);
    const float scale = 1.0f / sqrtf((float)DH);
    float mx = -INFINITY;
#pragma unroll
    for (int jj = 0; jj < NJ; ++jj)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int key = kbase + jj * 16 + 4 * g + e;
        const float v = key < nkeys ? sc[jj][e] * scale : -INFINITY;
        sc[jj][e] = v;
        mx = fmaxf(mx, v);
      }
    mx = fmaxf(mx, __shfl_xor(mx, 16, 64));
    mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
    float sum = 0.f;
#pragma unroll
    for (int jj = 0; jj < NJ; ++jj)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float p = mx == -INFINITY ? 0.f : expf(sc[jj][e] - mx);
        sc[jj][e] = p;
        sum += p;
      }
    sum += __shfl_xor(sum, 16, 64);
    sum += __shfl_xor(sum, 32, 64);
    // contraction position 8g + j <-> key (j < 4 ? 4g + j : 16 + 4g + j - 4),
    // the same order in P^T (registers) and in V^T (two 8-byte LDS reads)
    static_assert(NJ == 2, "two 16-key halves per chunk");
    MF::frag pb;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      pb[e] = static_cast<bf16>(sc[0][e]);
      pb[4 + e] = static_cast<bf16>(sc[1][e]);
    }
    f32x4 o[NT];
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      const bf16* vrow = &Vt[(nt * 16 + fr) * LDV + 4 * g];
      const u32x2 v0 = *reinterpret_cast<const u32x2*>(vrow);
      const u32x2 v1 = *reinterpret_cast<const u32x2*>(vrow + 16);
      const MF::frag va = __builtin_bit_cast(MF::frag, u32x4{v0[0], v0[1], v1[0], v1[1]});
      o[nt] = MF::run(va, pb, f32x4{0.f, 0.f, 0.f, 0.f});
    }
    // O^T: lane holds dims nt*16 + 4g .. +4 of query row w*16 + fr.  The
    // chunk's output rows, divided by their probability sums in bf16 (the
    // combine weights them by the sums again, in fp32), are row-major and
    // contiguous per wave in memory; they leave through LDS so that every
    // global store instruction writes whole 128-byte lines (scattered partial
    // lines cost several times more to store and confirm).
    constexpr int SROW = DH * 2 + 16;  // staged row stride in bytes (spreads the LDS banks)
    char* stw = stage + w * 16 * SROW;
    const float rl = sum > 0.f ? 1.0f / sum : 0.f;
#pragma unroll
    for (int nt = 0; nt < NT; ++nt)
      *reinterpret_cast<u32x2*>(stw + fr * SROW + nt * 32 + 8 * g) = pack4_bf16(o[nt] * rl);
    const size_t slot = ((size_t)b * nH + hn) * C + c;
    const int nrows = min(16, H - w * 16);  // rows of this wave that exist
    if (nrows > 0) {
      const u32 base = (u32)(((slot * H + w * 16) * DH) * 2);
      const int bytes = nrows * DH * 2;
      for (int off = lane * 16; off < bytes; off += 1024) {
        const int row = off / (DH * 2), col = off - row * (DH * 2);
        st16(ro, base + (u32)off, *reinterpret_cast<const u32x4*>(stw + row * SROW + col));
      }
      if (g == 0 && fr < nrows) st8(rml, (u32)((slot * H + w * 16 + fr) * 8), u32x2{f2u(mx), f2u(sum)});
    }
    __syncthreads();  // LDS reused by the next item
  }
}

// ---- phase 2: combine chunk partials -> o -------------------------------------
// Two (rollout, head, query row) items per workgroup at a time, one per half
// of the threads, so that every chunk load of both rows is in flight together.
// Within a half, nq = Dh/4 threads cover the Dh positions of a partial row
// (4 each) and G groups of them split the chunks; each pass loads CPT chunks'
// partial outputs and (max, sum) pairs in one round trip and folds them into
// a running (max, sum, acc); the G groups are then merged through LDS.
__device__ __forceinline__ void phase_combine(const PersistArgs& a, char* smem) {
  constexpr int TPR = PT / 2;
  const int H = a.H, nH = a.nH, C = a.C, Dh = a.Dh;
  const int nq = Dh / 4, G = TPR / nq;
  const int t = threadIdx.x, hf = t / TPR, tr = t - hf * TPR, q4 = tr % nq, g = tr / nq;
  float* sm = reinterpret_cast<float*>(smem);  // [PT] max, [PT] sum, [PT][4] acc
  float* sl = sm + PT;
  f32x4* sacc = reinterpret_cast<f32x4*>(sl + PT);
  const rsrc_t ro = rsrc(a.opart), rml = rsrc(a.ml), rout = rsrc(a.o);
  const int rows = a.B * nH * H, pairs = (rows + 1) / 2;
  for (int pr = blockIdx.x; pr < pairs; pr += gridDim.x) {
    const int r = 2 * pr + hf;
    const bool live = r < rows;
    const int i = live ? r % H : 0, bh = live ? r / H : 0;
    const int b = bh / nH, hn = bh - b * nH;
    const int nch = live ? (a.prefix_len[b] + H + KC - 1) / KC : 0;
    const size_t slot0 = (size_t)bh * C;
    float m = -INFINITY, lsum = 0.f;
    f32x4 acc = f32x4{0.f, 0.f, 0.f, 0.f};
    for (int c0 = g; c0 < nch; c0 += G * CPT) {
      u32x2 ov[CPT];
      float2 mv[CPT];  // (chunk max, chunk sum)
#pragma unroll
      for (int u = 0; u < CPT; ++u) {
        const int c = c0 + G * u;
        const bool ok = c < nch;
        ov[u] = ok ? ld8(ro, (u32)((((slot0 + c) * H + i) * Dh + q4 * 4) * 2)) : u32x2{0u, 0u};
        mv[u] = ok ? ld8f(rml, (u32)(((slot0 + c) * H + i) * 8)) : float2{-INFINITY, 0.f};
      }
      float mp = m;
#pragma unroll
      for (int u = 0; u < CPT; ++u) mp = fmaxf(mp, mv[u].x);
      const float f = m == -INFINITY ? 0.f : expf(m - mp);
      acc *= f;
      lsum *= f;
#pragma unroll
      for (int u = 0; u < CPT; ++u) {
        const float wc = mv[u].x == -INFINITY ? 0.f : expf(mv[u].x - mp);
        const float wl = wc * mv[u].y;  // the chunk's row is normalised by its sum
        acc += wl * f32x4{bf16_lo(ov[u][0]), bf16_hi(ov[u][0]), bf16_lo(ov[u][1]), bf16_hi(ov[u][1])};
        lsum += wl;
      }
      m = mp;
    }
    sm[t] = m;
    sl[t] = lsum;
    sacc[t] = acc;
    __syncthreads();
    trace_note(s_note, 1);
    if (live && g == 0) {
      const int b0 = hf * TPR + q4;
      float mx = -INFINITY;
      for (int gg = 0; gg < G; ++gg) mx = fmaxf(mx, sm[b0 + gg * nq]);
      float L = 0.f;
      f32x4 o4 = f32x4{0.f, 0.f, 0.f, 0.f};
      for (int gg = 0; gg < G; ++gg) {
        const float mg = sm[b0 + gg * nq];
        const float wg = mg == -INFINITY ? 0.f : expf(mg - mx);
        o4 += wg * sacc[b0 + gg * nq];
        L += wg * sl[b0 + gg * nq];
      }
      o4 *= 1.0f / L;
      st8(rout, frag_off(b * H + i, hn * Dh + q4 * 4, nH * Dh / 32) * 2u, pack4_bf16(o4));
    }
    __syncthreads();
  }
}

constexpr int NGRP = MAX_W / (4 * PT);  // 4-column groups per thread of a row

// Modulation (scale, shift) of this thread's column groups k4 = 4t + 4*PT*jg.
__device__ __forceinline__ void load_mod(const PersistArgs& a, const float* scale, const float* shift, f32x4* sc,
                                         f32x4* sh) {
#pragma unroll
  for (int jg = 0; jg < NGRP; ++jg) {
    const int k4 = 4 * threadIdx.x + 4 * PT * jg;
    const bool ok = k4 < a.W;
    sc[jg] = ok ? *reinterpret_cast<const f32x4*>(scale + k4) : f32x4{0.f, 0.f, 0.f, 0.f};
    sh[jg] = ok ? *reinterpret_cast<const f32x4*>(shift + k4) : f32x4{0.f, 0.f, 0.f, 0.f};
  }
}

// adaRMSNorm of the owner's residual row (LDS) -> y row (bf16, coherent).
__device__ __forceinline__ void store_y(const PersistArgs& a, const float* hrow, float rs, const f32x4* sc,
                                        const f32x4* sh) {
  const rsrc_t ry = rsrc(a.y);
  const int m = blockIdx.x, W = a.W;
#pragma unroll
  for (int jg = 0; jg < NGRP; ++jg) {
    const int k4 = 4 * threadIdx.x + 4 * PT * jg;
    if (k4 < W) {
      const f32x4 h = *reinterpret_cast<const f32x4*>(hrow + k4);
      st8(ry, frag_off(m, k4, W / 32) * 2u, pack4_bf16(h * rs * (1.0f + sc[jg]) + sh[jg]));
    }
  }
}

// In-projection of the owner's row: h = x W_in^T + b_in (x in LDS, W_in
// [W][A] in global memory; with A % 8 == 0 a thread loads its rows as
// 16-byte pieces, all in flight), then the step's first adaRMSNorm -> y.
// A correction row, or every row when the caller hands the rows over
// (crow != nullptr), starts from that row instead.
__device__ __forceinline__ void inproj_row(const PersistArgs& a, const float* scale, const float* shift, float* hrow,
                                           const float* bin, const float* xs, float* red, const float* crow) {
  const int W = a.W, A = a.A;
  const bf16* win = reinterpret_cast<const bf16*>(a.w_in);
  f32x4 sc[NGRP], sh[NGRP];
  load_mod(a, scale, shift, sc, sh);
  __syncthreads();  // xs
  if (crow) {
    for (int k4 = 4 * threadIdx.x; k4 < W; k4 += 4 * PT)
      *reinterpret_cast<f32x4*>(hrow + k4) = *reinterpret_cast<const f32x4*>(crow + k4);
  } else if ((A & 7) == 0) {
    constexpr int NJ = MAX_W / PT;  // rows per thread
    for (int j0 = 0; j0 < NJ; j0 += 4) {
      if (PT * j0 >= W) break;
      u32x4 v[4][8];
#pragma unroll
      for (int jj = 0; jj < 4; ++jj) {
        const int n = threadIdx.x + PT * (j0 + jj);
#pragma unroll
        for (int c8 = 0; c8 < 8; ++c8)
          v[jj][c8] = (n < W && c8 * 8 < A) ? *reinterpret_cast<const u32x4*>(win + (size_t)n * A + c8 * 8)
                                             : u32x4{0u, 0u, 0u, 0u};
      }
#pragma unroll
      for (int jj = 0; jj < 4; ++jj) {
        const int n = threadIdx.x + PT * (j0 + jj);
        if (n >= W) continue;
        float acc = 0.f;
#pragma unroll
        for (int c8 = 0; c8 < 8; ++c8) {
          if (c8 * 8 >= A) break;
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            acc = fmaf(xs[c8 * 8 + 2 * q], bf16_lo(v[jj][c8][q]), acc);
            acc = fmaf(xs[c8 * 8 + 2 * q + 1], bf16_hi(v[jj][c8][q]), acc);
          }
        }
        hrow[n] = acc + bin[n];
      }
    }
  } else {
    for (int n = threadIdx.x; n < W; n += PT) {
      float acc = 0.f;
      for (int c = 0; c < A; ++c) acc = fmaf(xs[c], static_cast<float>(win[(size_t)n * A + c]), acc);
      hrow[n] = acc + bin[n];
    }
  }
  __syncthreads();
  float ss = 0.f;
  for (int k = threadIdx.x; k < W; k += PT) ss += hrow[k] * hrow[k];
  const float rs = 1.0f / sqrtf(block_sum_wg(ss, red) / (float)W + a.eps);
  store_y(a, hrow, rs, sc, sh);
}

struct RowJob {
  int S;               // split-K slices to sum
  const float* gate;   // residual gate of the finished sublayer
  const float* scale;  // next adaRMSNorm (or the final norm)
  const float* shift;
  bool final_step;     // last layer: final norm, action-out projection, Euler update
};

// ---- phases 4, 7: row owner updates -----------------------------------------------
__device__ __forceinline__ void phase_rows(const PersistArgs& a, const RowJob& r, float& xreg, float* hrow,
                                           const float* bin, float* xs, char* smem, u32* s_abort) {
  const int m = blockIdx.x, W = a.W, A = a.A, t = threadIdx.x;
  if (m >= a.M) return;
  float* red = reinterpret_cast<float*>(smem);  // [NWV]
  float* ys = red + 16;                         // [MAX_W] final normalised row
  float* pp = ys + MAX_W;                       // [PT] projection partials
  // final step: the action-out weights do not depend on this step's data, so
  // their loads go out together with the slice loads
  const int apad = A <= 8 ? 8 : A <= 16 ? 16 : A <= 32 ? 32 : 64;
  const int tpa = PT / apad, kper = W / tpa, ao = t % apad, kso = t / apad;
  u32x4 wv[OUT_G];
  float bo = 0.f;
  if (r.final_step) {
    const bf16* wo = reinterpret_cast<const bf16*>(a.w_out) + (size_t)ao * W + kso * kper;
#pragma unroll
    for (int gi = 0; gi < OUT_G; ++gi)
      wv[gi] = (gi * 8 < kper && ao < A) ? *reinterpret_cast<const u32x4*>(wo + gi * 8) : u32x4{0u, 0u, 0u, 0u};
    if (t < A) bo = a.b_out[t];
  }
  f32x4 sc[NGRP], sh[NGRP];
  load_mod(a, r.scale, r.shift, sc, sh);
  // The slices of this row: polled until no word is EMPTY (bounded), then
  // reset to EMPTY for the next writer.
  const rsrc_t rp = rsrc(a.part, (u32)((size_t)r.S * a.M * W * 4));
  trace_note(s_note, 0);
#pragma unroll
  for (int jg = 0; jg < NGRP; ++jg) {
    const int k4 = 4 * t + 4 * PT * jg;
    if (k4 >= W) break;
    u32x4 v[RMAX_S];
#pragma unroll
    for (int z = 0; z < RMAX_S; ++z)
      v[z] = z < r.S ? poll16(rp, (u32)(((size_t)z * a.M + m) * W + k4) * 4u) : u32x4{0u, 0u, 0u, 0u};
    for (u32 spins = 0;; ++spins) {
      u32 pend = 0u;
#pragma unroll
      for (int z = 0; z < RMAX_S; ++z) pend |= (z < r.S && has_empty(v[z]) ? 1u : 0u) << z;
      if (pend == 0u) break;
      if (spins > SPIN_LIMIT || *s_abort != 0u) {
        *s_abort = 1u;
        st4(rsrc(a.err), 0, 1u);
        break;
      }
#pragma unroll
      for (int z = 0; z < RMAX_S; ++z)
        if ((pend >> z) & 1u) v[z] = poll16(rp, (u32)(((size_t)z * a.M + m) * W + k4) * 4u);
    }
#pragma unroll
    for (int z = 0; z < RMAX_S; ++z)
      if (z < r.S) st16(rp, (u32)(((size_t)z * a.M + m) * W + k4) * 4u, u32x4{EMPTY, EMPTY, EMPTY, EMPTY});
    const f32x4 g4 = *reinterpret_cast<const f32x4*>(r.gate + k4);
    f32x4 sum = as_f4(v[0]);
#pragma unroll
    for (int z = 1; z < RMAX_S; ++z) sum += as_f4(v[z]);
    f32x4* hp = reinterpret_cast<f32x4*>(hrow + k4);
    *hp = *hp + g4 * sum;
  }
  __syncthreads();
  trace_note(s_note, 1);
  float ss = 0.f;
  for (int k = t; k < W; k += PT) ss += hrow[k] * hrow[k];
  const float rs = 1.0f / sqrtf(block_sum_wg(ss, red) / (float)W + a.eps);
  if (!r.final_step) {
    store_y(a, hrow, rs, sc, sh);
    return;
  }
#pragma unroll
  for (int jg = 0; jg < NGRP; ++jg) {
    const int k4 = 4 * t + 4 * PT * jg;
    if (k4 < W)
      *reinterpret_cast<f32x4*>(ys + k4) = *reinterpret_cast<const f32x4*>(hrow + k4) * rs * (1.0f + sc[jg]) + sh[jg];
  }
  __syncthreads();
  float p = 0.f;
  const float* yk = ys + kso * kper;
#pragma unroll
  for (int gi = 0; gi < OUT_G; ++gi) {
    if (gi * 8 >= kper) break;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      p = fmaf(yk[gi * 8 + 2 * q], bf16_lo(wv[gi][q]), p);
      p = fmaf(yk[gi * 8 + 2 * q + 1], bf16_hi(wv[gi][q]), p);
    }
  }
  pp[t] = p;
  __syncthreads();
  if (t < A) {
    float v = pp[t];
    for (int s = 1; s < tpa; ++s) v += pp[s * apad + t];
    if (m % a.H - a.n_corr >= a.n_fixed) xreg += a.dt * (v + bo);  // action rows past the committed ones
    xs[t] = xreg;
  }
}

__device__ __forceinline__ GemmJob make_job(const PersistArgs& a, int p, int l) {
  const bf16* lay = reinterpret_cast<const bf16*>(a.w_frag) + (size_t)l * a.layer_elems;
  if (p == 0) return GemmJob{a.y, lay, a.W, (a.nH + 2) * a.Dh / 32, 1, EPI_QKV};
  if (p == 3) return GemmJob{a.o, lay + a.off_o, a.nH * a.Dh, a.W / 32, a.s_o, EPI_SLICE};
  if (p == 5) return GemmJob{a.y, lay + a.off_gu, a.W, 2 * a.F / 32, 1, EPI_GEGLU};
  return GemmJob{a.z, lay + a.off_d, a.F, a.W / 32, a.s_d, EPI_SLICE};
}

// Producers of this workgroup's inputs in phase p of layer l (none if the
// workgroup has no work in that phase).  Item layouts: GEMM item it = tile +
// slice * tiles, attention item (rollout, head, chunk), combine item = a pair
// of (rollout, head, query) rows; each runs on workgroup it % grid.
__device__ __forceinline__ Deps phase_deps(const PersistArgs& a, int p, const GemmJob& j) {
  const int G = gridDim.x, bid = blockIdx.x;
  const int M = a.M, H = a.H, nH = a.nH, Dh = a.Dh, C = a.C;
  if (p == 4 || p == 7) return deps_none();  // row phases poll the slice data instead of flags
  if (p == 0 || p == 5) return bid < j.tiles ? Deps{0, M, 0, 0} : deps_none();  // QKV, GateUp: the row owners
  if (p == 1) {  // attention: the QKV tiles of this head, and of k and v if the chunk holds action keys
    const int n_items = a.B * nH * C;
    if (bid >= n_items) return deps_none();
    if (n_items > G) return deps_all();
    const int c = bid % C, hn = (bid / C) % nH, b = bid / (C * nH);
    const int pl = a.prefix_len[b], kbase = c * KC;
    if (kbase >= pl + H) return deps_none();
    const int tq = Dh / 32;
    if ((nH + 2) * tq > G) return deps_all();
    const Deps q = deps_items(hn * tq, (hn + 1) * tq);
    if (kbase + KC <= pl) return q;
    const Deps kv = deps_items(nH * tq, (nH + 2) * tq);
    return Deps{q.lo0, q.hi0, kv.lo0, kv.hi0};
  }
  if (p == 2) {  // combine: the attention chunks of the heads of its two rows
    const int rows = a.B * nH * H, pairs = (rows + 1) / 2;
    if (bid >= pairs) return deps_none();
    if (pairs > G) return deps_all();
    const int bh0 = (2 * bid) / H, bh1 = min(2 * bid + 1, rows - 1) / H;
    return deps_items(bh0 * C, (bh1 + 1) * C);
  }
  const int n_items = j.tiles * j.S;
  if (bid >= n_items) return deps_none();
  if (n_items > G) return deps_all();
  const int klen = j.K / j.S, s0 = (bid / j.tiles) * klen;
  if (p == 3) {  // O-proj slice: the combine rows of the heads its K range covers, every rollout
    const int hn0 = s0 / Dh, hn1 = (s0 + klen - 1) / Dh;
    const int r0 = hn0 * H, r1 = ((a.B - 1) * nH + hn1) * H + H;  // rows [r0, r1) cover them
    return deps_items(r0 / 2, (r1 + 1) / 2);
  }
  // Down slice: the GateUp tiles that wrote z columns [s0, s0 + klen) (16 per tile)
  return deps_items(s0 / 16, (s0 + klen) / 16);
}

template <int DH>
__global__ __launch_bounds__(PT) void k_persist(PersistArgs a) {
  __shared__ __attribute__((aligned(16))) char smem[SMEM_BYTES];
  __shared__ __attribute__((aligned(16))) char s_wt[WT_STEPS * 2 * 1024];  // weight tile of the current GEMM
  __shared__ __attribute__((aligned(16))) float s_hrow[MAX_W];  // residual row of the owned action row
  __shared__ __attribute__((aligned(16))) float s_bin[MAX_W];
  __shared__ float s_x[64];
  __shared__ u32 s_ctl[2];  // [0]: a wait gave up (stop waiting); [1]: polls per wait (read where tested,
                            // so that the bound occupies no register across the kernel)
  const int t = threadIdx.x, m = blockIdx.x;
  const int L = a.L, W = a.W, A = a.A;
  const bool owner = m < a.M;
  // owned row: rollout m / H, suffix row m % H; action index ia < 0 for a correction row
  const int ia = m % a.H - a.n_corr;
  const size_t xrow = (size_t)(m / a.H) * (a.H - a.n_corr) + ia;
  const float* crow = a.h_in ? a.h_in + (size_t)m * W
                   : ia < 0   ? a.corr + ((size_t)(m / a.H) * a.n_corr + (m % a.H)) * W
                              : nullptr;
  const bool at_t0 = ia >= 0 && ia < a.n_t0;  // a committed row modulated at t = 0 (table row n_steps)
  float xreg = 0.f;
  if (t == 0) {
    s_ctl[0] = 0u;
    s_ctl[1] = a.spin_limit;
  }
  if (owner) {
    for (int k4 = 4 * t; k4 < W; k4 += 4 * PT)
      *reinterpret_cast<f32x4*>(s_bin + k4) = *reinterpret_cast<const f32x4*>(a.b_in + k4);
    if (t < A && ia >= 0) {
      xreg = a.x[xrow * A + t];
      s_x[t] = xreg;
    }
  }
  trace_start(a, s_note);
  __syncthreads();
  lds_t* wt = (lds_t*)s_wt;
  const int last_phase = a.n_steps * L * 8 - 1;
  // ph = -1 is the first step's in-projection; the later ones follow the final
  // row phase of the previous step in the same workgroup (no wait between)
  for (int ph = -1; ph <= last_phase; ++ph) {
    // in-projection + first norm of step ki (one call site for every step)
    int ki = ph < 0 ? 0 : -1;
    const int k = ph < 0 ? 0 : ph / (8 * L), l = ph < 0 ? 0 : (ph / 8) % L, p = ph < 0 ? -1 : ph % 8;
    const float* tk = a.table + (size_t)(at_t0 ? a.n_steps : k) * a.R;
    const float* am = tk + (size_t)(2 * l) * 3 * W;      // attention modulation: scale | shift | gate
    const float* mm = tk + (size_t)(2 * l + 1) * 3 * W;  // MLP modulation
    const bool gemm = p == 0 || p == 3 || p == 5 || p == 6;
    const GemmJob job = make_job(a, gemm ? p : 0, l);
    // producers of this phase's inputs finished phase ph - 1 (attention waits
    // inside, after loading the prefix part of its chunk)
    const bool rows = p == 4 || p == 7;
    if (ph >= 0 && p != 1 && !rows) wait_producers(a, phase_deps(a, p, job), (u32)(ph + 1), s_ctl, gemm, job, wt);
    if (p < 0) {
    } else if (p == 1) {
      phase_attn<DH>(a, l, smem, phase_deps(a, p, job), (u32)(ph + 1), s_ctl, wt, s_wt);
    } else if (p == 2) {
      phase_combine(a, smem);
    } else if (p == 4 || p == 7) {
      RowJob r;
      r.final_step = false;
      if (p == 4) {
        r.S = a.s_o;
        r.gate = am + 2 * W;
        r.scale = mm;
        r.shift = mm + W;
      } else {
        r.S = a.s_d;
        r.gate = mm + 2 * W;
        if (l + 1 < L) {
          r.scale = am + 6 * W;  // next layer's attention modulation
          r.shift = am + 7 * W;
        } else {
          const float* fm = tk + (size_t)(6 * L) * W;
          r.scale = fm;
          r.shift = fm + W;
          r.final_step = true;
        }
      }
      phase_rows(a, r, xreg, s_hrow, s_bin, s_x, smem, s_ctl);
      if (r.final_step && k + 1 < a.n_steps) ki = k + 1;  // same workgroup, no wait needed
    } else {
      phase_gemm(a, job, l, wt, smem);
    }
    if (ki >= 0 && owner) {
      const float* ti = a.table + (size_t)(at_t0 ? a.n_steps : ki) * a.R;
      inproj_row(a, ti, ti + W, s_hrow, s_bin, s_x, reinterpret_cast<float*>(smem), crow);
    }
    // Completion flags: the row owners poll the split-K slices themselves, so
    // the slice producers (phases 3, 6) and the workgroups without a row
    // (row phases) have nothing to signal and go straight on.
    const bool signal = !(p == 3 || p == 6) && !(rows && !owner);
    if (ph < last_phase && signal) phase_done(a, (u32)(ph + 2));
    if (ph >= 0) trace_end(a, s_note, ph);
  }
  if (owner && t < A && ia >= 0) a.x[xrow * A + t] = xreg;
}

// dst = fragment-ordered copy of the row-major bf16 matrix src [R][K]
// (R % 16 == 0, K % 32 == 0); one 16-byte chunk per thread.
__global__ void k_frag_order(const u32x4* __restrict__ src, u32x4* __restrict__ dst, int R, int K) {
  const int KS = K / 32;
  const size_t n = (size_t)(R / 16) * KS * 64;
  for (size_t c = (size_t)blockIdx.x * blockDim.x + threadIdx.x; c < n; c += (size_t)gridDim.x * blockDim.x) {
    const size_t blk = c / 64;
    const int l = (int)(c % 64);
    const size_t row = (blk / KS) * 16 + (l & 15);
    const int k = (int)(blk % KS) * 32 + (l >> 4) * 8;
    dst[c] = src[(row * K + k) / 8];
  }
}

// Before every launch: completion flags to zero, the split-K slice words to
// EMPTY.
__global__ void k_persist_reset(u32* flags, int n, u32x4* part, int n_part4) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) flags[i] = 0u;  // n = FLAG_WORDS
  for (int j = i; j < n_part4; j += gridDim.x * blockDim.x) part[j] = u32x4{EMPTY, EMPTY, EMPTY, EMPTY};
}

}  // namespace

bool persist_supported(jpi_dtype dt, int M, int W, int nH, int Dh, int F, int H, int A, int Pmax) {
  if (dt != JPI_BF16 || M > 64 || H > 64 || nH % 2 != 0 || !(Dh == 64 || Dh == 128 || Dh == 256)) return false;
  if (W % (NWV * 32) != 0 || F % (NWV * 32) != 0 || (nH * Dh) % (NWV * 32) != 0) return false;
  if (W > MAX_W || A < 1 || A > 64 || Pmax + H > MAX_CH * KC) return false;
  const int apad = A <= 8 ? 8 : A <= 16 ? 16 : A <= 32 ? 32 : 64;
  const int kper = W / (PT / apad);  // action-out projection: columns per thread
  return kper % 8 == 0 && kper <= OUT_G * 8;
}

int persist_chunks(int P, int H) { return (P + H + KC - 1) / KC; }

int persist_pick_split(int tiles, int K, int grid) {
  int s = 1;
  while (s < RMAX_S && tiles * s < grid && K % (2 * s * NWV * 32) == 0) s *= 2;
  return s;
}

int persist_block_threads() { return PT; }

unsigned persist_default_spin() { return SPIN_LIMIT; }

int persist_max_grid() { return MAX_GRID; }

int persist_flag_words() { return FLAG_WORDS; }

bool persist_trace_build() { return JPI_PERSIST_TRACE != 0; }

hipError_t launch_frag_order(const void* src, void* dst, int R, int K, hipStream_t s) {
  if (R % 16 != 0 || K % 32 != 0) return hipErrorInvalidValue;
  const size_t n = (size_t)(R / 16) * (K / 32) * 64;
  const int grid = (int)std::min<size_t>((n + 255) / 256, 4096);
  hipLaunchKernelGGL(k_frag_order, dim3(grid), dim3(256), 0, s, reinterpret_cast<const u32x4*>(src),
                     reinterpret_cast<u32x4*>(dst), R, K);
  return hipGetLastError();
}

hipError_t persist_occupancy(int Dh, int* blocks_per_cu) {
  switch (Dh) {
    case 64: return hipOccupancyMaxActiveBlocksPerMultiprocessor(blocks_per_cu, k_persist<64>, PT, 0);
    case 128: return hipOccupancyMaxActiveBlocksPerMultiprocessor(blocks_per_cu, k_persist<128>, PT, 0);
    case 256: return hipOccupancyMaxActiveBlocksPerMultiprocessor(blocks_per_cu, k_persist<256>, PT, 0);
  }
  return hipErrorInvalidValue;
}

hipError_t launch_persist(const PersistArgs& a, int grid, hipStream_t s) {
  if (grid > MAX_GRID) return hipErrorInvalidValue;
  const int n_part4 = std::max(a.s_o, a.s_d) * a.M * a.W / 4;  // the slice words start EMPTY
  hipLaunchKernelGGL(k_persist_reset, dim3(std::max((FLAG_WORDS + 255) / 256, std::min((n_part4 + 255) / 256, 1024))),
                     dim3(256), 0, s, a.flags, FLAG_WORDS, reinterpret_cast<u32x4*>(a.part), n_part4);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  switch (a.Dh) {
    case 64: JPI_LAUNCH((k_persist<64>), dim3(grid), dim3(PT), 0, s, a.ev_start, a.ev_stop, a); break;
    case 128: JPI_LAUNCH((k_persist<128>), dim3(grid), dim3(PT), 0, s, a.ev_start, a.ev_stop, a); break;
    case 256: JPI_LAUNCH((k_persist<256>), dim3(grid), dim3(PT), 0, s, a.ev_start, a.ev_stop, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace jpi
