// Internal declarations shared by the libjpi runtime and its kernels.
#pragma once

#include <hip/hip_runtime.h>

#include <vector>
#include <stdint.h>

#include <hip/hip_ext.h>

#include "../../include/jpi.h"

namespace jpi {

typedef __bf16 bf16;

// ---------------------------------------------------------------------------
// Epilogue descriptors for the GEMM kernel.  A GEMM computes
// acc[m][n] = sum_k A[m][k] W[n][k] (fp32) and hands each value to one of
// these epilogues.  Packed column orders are described in jpi_runtime.hip.
// ---------------------------------------------------------------------------
enum EpiKind { EPI_STORE_F32 = 0, EPI_QKV = 1, EPI_GEGLU = 2 };

struct EpiParams {
  // EPI_STORE_F32: [splitk][M][N] (slice z at out_f32 + z*M*N)
  float* out_f32;
  // EPI_QKV: packed columns [q heads | k | v]; RoPE on q and k
  void* q;               // [B][nH][H][Dh]
  void* ks;              // [B][H][Dh], rollout b at ks + b * ks_bstride elements
  int64_t ks_bstride;    // 0 means H * Dh
  void* vst;             // [B][Dh][vst_ld] (v stored transposed)
  int vst_ld;            // row stride of vst in elements (>= horizon)
  const float2* rope;    // [B][H][Dh/2] (cos, sin) at position prefix_len[b] + i
  int n_heads, head_dim, horizon;
  // EPI_GEGLU: packed columns in 32-wide groups [gate 16 | up 16]
  void* z;               // [M][F]
  int mlp_dim;
};

struct GemmLaunch {
  const void* A;         // [M][K]
  const void* W;         // [N][K]
  int M, N, K;
  int splitk;            // > 1 only with EPI_STORE_F32
  int n_cu;              // compute units of the device (tile choice); 0 = assume 256
  EpiKind epi;
  EpiParams ep;
  hipEvent_t ev_start, ev_stop;  // optional: timestamps of this launch (measurement)
};

// launchers (jpi_kernels.hip).  All return hipSuccess or the launch error.
hipError_t launch_gemm(jpi_dtype dt, const GemmLaunch& g, hipStream_t s);
size_t gemm_tiles(jpi_dtype dt, int M, int N);          // workgroup tiles of one K slice
int gemm_pick_splitk(jpi_dtype dt, int M, int N, int K, int n_cu);

hipError_t launch_sum_slices(const float* P, float* C, int S, size_t MN, hipStream_t s);
int gemm_k_quantum(jpi_dtype dt, int M);  // K of every split must be a multiple of this

// Per-row residual update + next adaRMSNorm (see k_resid_norm).
struct RowLaunch {
  const float* part;     // [S][M][W] split-K slices of the sublayer output
  int S, M, W;
  float* h;              // [M][W] residual stream (updated in place)
  const float* gate;     // [W]
  const float* scale;    // [W] next norm (final norm when final_step)
  const float* shift;    // [W]
  void* y;               // [M][W] normalised activations (not final_step)
  float eps;
  // final_step only: action-out projection and Euler update
  const void* w_out;     // [A][W]
  const float* b_out;    // [A]
  float* x;              // [B][horizon][A]
  int A, horizon, n_fixed;
  int n_lead;            // correction rows ahead of each rollout's action rows (rows m = b*(n_lead+horizon)+r)
  float dt;
  int n_t0;              // leading action rows (committed) that take the t = 0 modulation
  int64_t t0_delta;      // offset (floats) from the step's modulation row to the t = 0 row
};
// corr: [B][n_lead][W] correction tokens (rows r < n_lead of each rollout), may be NULL when n_lead == 0
// n_t0 / t0_delta: the first n_t0 action rows read scale and shift at +t0_delta floats (the t = 0 table row)
hipError_t launch_inproj_norm(jpi_dtype dt, const float* x, const void* w_in, const float* b_in, float* h,
                              const float* scale, const float* shift, void* y, int M, int W, int A, float eps,
                              const float* corr, int n_lead, int horizon, int n_t0, int64_t t0_delta,
                              hipStream_t s);
hipError_t launch_resid_norm(jpi_dtype dt, const RowLaunch& r, bool final_step, hipStream_t s);

struct AttnLaunch {
  const void* q;          // [B][nH][H][Dh]
  const void* ks;         // [B][H][Dh], rollout b at ks + b * ks_bstride elements
  int64_t ks_bstride;     // 0 means H * Dh
  const void* vst;        // [B][Dh][vst_ld]   suffix V, transposed
  int64_t vst_ld;         // row stride of vst in elements: >= H, a multiple of 8 on the bf16 path
  const void* kp;         // prefix K: rollout b at kp + b*kp_bstride, key j at + j*Dh
  const void* vpt;        // prefix V transposed: rollout b at vpt + b*vpt_bstride, dim d at + d*vpt_dstride
  int64_t kp_bstride, vpt_bstride, vpt_dstride;  // elements; vpt_dstride a multiple of 8
  const int* prefix_len;  // device [B]
  int B, nH, H, P, Dh;
  float* opart;           // [B][nH][n_chunks][H][Dh]
  float* mpart;           // [B][nH][n_chunks][H]
  float* lpart;           // [B][nH][n_chunks][H]
  void* out;              // [B*H][nH*Dh] of dtype, or fp32 if out_f32
  int out_f32;
  int n_cu;               // compute units of the device (sizes the bf16 key ranges)
  hipEvent_t ev_start, ev_stop;  // optional: start of the chunk pass, end of the combine
};
int attn_chunk(jpi_dtype dt);
int attn_n_chunks(jpi_dtype dt, int P, int H);
int attn_max_prefix(jpi_dtype dt, int H);
// dst[z][c][r] = src[z][r][c] (r < rows, c < cols) for nmat matrices
hipError_t launch_transpose(jpi_dtype dt, const void* src, void* dst, int rows, int cols, int64_t sld, int64_t dld,
                            int64_t sz, int64_t dz, int nmat, hipStream_t s);
hipError_t launch_attention(jpi_dtype dt, const AttnLaunch& a, hipStream_t s);
// bf16 attention (jpi_flash.hip): S key ranges per 128-row query tile; with
// S > 1 the partials live in a.opart (flash_scratch_bytes(...) bytes)
int flash_splits(int B, int nH, int H, int P, int n_cu);
size_t flash_scratch_bytes(int B, int nH, int H, int Dh, int S);
hipError_t launch_flash(const AttnLaunch& a, int S, hipStream_t s);

// Persistent single-launch denoise (jpi_persist.hip), M <= 64, bf16.
struct PersistArgs {
  int L, W, nH, Dh, F, A, H, B, M;  // H: suffix rows per rollout (n_corr correction rows, then the action rows)
  int n_corr;               // correction rows ahead of each rollout's action rows
  const float* corr;        // [B][n_corr][W] correction tokens (rows restart from them every step)
  const float* h_in;        // [M][W] or null: every row starts from it instead of the in-projection
                            // (the action-time expert's MLP output; then n_steps is 1)
  int C;                    // attention chunks (32 keys) per rollout
  int n_steps, n_fixed, s_o, s_d, R;
  int n_t0;                 // leading action rows (committed) modulated at t = 0: table row n_steps
  float eps, dt;
  const void* w_layers;     // packed layer weights (bf16)
  const void* w_frag;       // the same, each matrix fragment-ordered
  int64_t layer_elems, off_o, off_gu, off_d;
  const void* w_in;
  const float* b_in;
  const void* w_out;
  const float* b_out;
  const float* table;       // [n_steps + 1][R] modulation (row n_steps: t = 0)
  const void* kp;           // prefix K [L][Bmax][Pmax][Dh]
  const void* vpt;          // prefix V transposed [L][Bmax][Dh][Ppad]
  int64_t kp_lstride, kp_bstride, vpt_lstride, vpt_bstride, vpt_dstride;
  const int* prefix_len;    // [B]
  const float2* rope;       // [B][H][Dh/2]
  float* x;                 // [B][H - n_corr][A] action rows
  float* h;                 // [M][W]
  void* y;                  // fragment-ordered [64][W] bf16 (single-launch path)
  void* q;                  // fragment-ordered [B][nH][64][Dh]
  void* ks;                 // [B][H][Dh]
  void* vst;                // [B][Dh][H]
  float* opart;             // [B][nH][C][H][Dh] bf16: each chunk's output row / its probability sum
  float* ml;                // [B][nH][C][H][2] (chunk max, probability sum)
  void* o;                  // fragment-ordered [64][nH*Dh]
  float* part;              // [max(s_o, s_d)][M][W]
  void* z;                  // fragment-ordered [64][F]
  unsigned* flags;          // [grid][32] completion flags: the last phase index + 2 each workgroup finished
  unsigned* err;            // set to 1 if a wait for producers timed out
  unsigned spin_limit;      // unsuccessful polls after which a wait gives up (>= 1)
  hipEvent_t ev_start, ev_stop;
  unsigned long long* trace;  // trace build only: [grid][trace_slots] real-time stamps (else null)
  int trace_slots;            // 1 + phases recorded per workgroup
};
bool persist_supported(jpi_dtype dt, int M, int W, int nH, int Dh, int F, int H, int A, int Pmax);
int persist_chunks(int P, int H);
int persist_pick_split(int tiles, int K, int grid);
int persist_block_threads();
unsigned persist_default_spin();  // polls a wait makes before it gives up
int persist_max_grid();    // largest grid the completion flags support
int persist_flag_words();  // size of the completion flag buffer in 32-bit words
bool persist_trace_build(); // the kernel was compiled with JPI_PERSIST_TRACE (phase timestamps)
// dst = fragment-ordered copy of the row-major bf16 matrix src [R][K]
hipError_t launch_frag_order(const void* src, void* dst, int R, int K, hipStream_t s);
hipError_t persist_occupancy(int Dh, int* blocks_per_cu);
hipError_t launch_persist(const PersistArgs& a, int grid, hipStream_t s);

// The resident prefix buffers of an action-expert context, for a producer
// that writes them in place (the VLM prefill).  ae_prefix_target checks that
// the producer's shape fits (L, Dh, dtype, batch, prefix) and returns the
// buffers; ae_prefix_bound records them as bound with prefix_len = prefix for
// rollouts 0..batch-1 (the caller has enqueued the writes, the prefix_len
// fill and the rope table on its stream).
struct AePrefixTarget {
  void* kp;             // K [L][Bmax][Pmax][Dh]
  void* vpt;            // V^T [L][Bmax][Dh][Ppad]
  int64_t kp_lstride, kp_bstride, vpt_lstride, vpt_bstride;
  int vpt_ld;           // Ppad
  int* prefix_len;      // device [Bmax]
  float2* rope_tab;     // device [Bmax][H][Dh/2]: the expert's own rows' positions
  int H;                // suffix rows per rollout the rope table covers (correction tokens + horizon)
  float rope_base;
};
jpi_status ae_prefix_target(jpi_ctx* c, int L, int Dh, jpi_dtype dt, int batch, int prefix, AePrefixTarget* t,
                            const char** why);
jpi_status ae_prefix_bound(jpi_ctx* c, int batch, int prefix, int rope_rows);

// ---- pre-norm decoder blocks with constant modulation (VLM prefill, correction module)
// Packed layer (bf16, the expert's layout): [q heads | k | v] rows (q and k in
// RoPE pack order) | O [W][nH Dh] | gate/up rows interleaved in 32-row groups | Down [W][F].
enum BlockMatrix { BM_Q, BM_K, BM_V, BM_GATE, BM_UP };
int block_pack_row(BlockMatrix kind, int r, int n_heads, int Dh);  // packed row of source row r
// dst row map[r] <- row r of data (host or device), then synchronise s
hipError_t upload_rows(void* dst, const std::vector<int>& map, int row_bytes, const void* data, bool is_device,
                       hipStream_t s);
struct BlockLaunch {
  int B, H, W, nH, Dh, F, n_cu;  // B rollouts of H rows each
  const char* w;                 // packed layer
  size_t off_o, off_gu, off_d;   // element offsets inside it
  float* h;                      // [M][W] residual stream, updated in place
  void* y;                       // [M][W] bf16: in the attention norm of h, out next_norm of the result
  void *q, *o, *z;               // [M][nH Dh], [M][nH Dh], [M][F] bf16 scratch
  float* partial;                // [max(s_o, s_d)][M][W]
  int s_o, s_d;                  // split-K of the O and Down projections
  float* opart;                  // attention scratch
  void* ks;                      // own keys (rotated), rollout b at ks + b * ks_bstride
  int64_t ks_bstride;            // 0 means H * Dh
  void* vst;                     // own values transposed [B][Dh][vst_ld]
  int vst_ld;
  const void *kp, *vpt;          // earlier keys [B][..][Dh] and values transposed [B][Dh][vpt_dstride]
  int64_t kp_bstride, vpt_bstride;
  int vpt_dstride;
  const int* prefix_len;         // device [B]: earlier keys each row sees
  int P;                         // bound on prefix_len
  const float2* rope;            // [B][H][Dh/2] (an identity table for no rotation)
  const float *mlp_norm, *next_norm, *ones, *zeros;
  float eps;
  bool f32;                      // fp32 weights and activations (default bf16)
};
hipError_t enqueue_block(const BlockLaunch& b, hipStream_t s);
// y[m] = rms(h[m]) (1 + w) in bf16 (or fp32 with f32)
hipError_t launch_norm_rows(const float* h, const float* w, void* y, int M, int W, float eps, hipStream_t s,
                            bool f32 = false);
hipError_t launch_fill_i32(int* p, int n, int v, hipStream_t s);
hipError_t launch_fill_f32(float* p, int n, float v, hipStream_t s);
hipError_t launch_identity_rope(float2* tab, int n, hipStream_t s);
hipError_t launch_bcast_rows(const float* src, float* dst, int M, int period, int W, hipStream_t s);

// emb[k] for k < rows at t = 1 - k/n
// ---- action-time expert variant (jpi_variant.hip)
hipError_t launch_const_table(float* tab, const float* norms, int rows, int L, int W, hipStream_t s);
hipError_t launch_plus_one(const int* src, int* dst, int n, hipStream_t s);
// u[m] = W_a x[m] + b_a in the context dtype
hipError_t launch_action_embed(jpi_dtype dt, const float* x, const void* w, const float* b, void* u, int M, int W,
                               int A, hipStream_t s);
// z[m] = swish(sum of S split-K slices + c) in the context dtype
hipError_t launch_swish_slices(jpi_dtype dt, const float* part, int S, int M, const float* c, void* z, int W,
                               hipStream_t s);
// key row b and value column 0 of rollout b into slot prefix_len[b] of one layer's K and V^T
hipError_t launch_put_state_kv(jpi_dtype dt, const void* ks, const void* vst, int vst_ld, void* kp, int64_t kp_bstride,
                               void* vpt, int64_t vpt_bstride, int vpt_dstride, const int* prefix_len, int B, int Dh,
                               hipStream_t s);

hipError_t launch_time_embed(float* emb, int rows, int n, int W, hipStream_t s);
// out[m][n] = act(sum_k in[m][k] w[n][k] + b[n]), fp64 accumulation; act 0 = none, 1 = swish
hipError_t launch_rowdot(jpi_dtype dt, const float* in, const void* w, const float* b, float* out, int M,
                         int N, int K, int act, hipStream_t s);
hipError_t launch_rope_table(const int* prefix_len, float2* tab, int B, int H, int Dh, float base,
                             hipStream_t s);
hipError_t launch_init_x(const float* noise, const float* committed, float* x, int B, int H, int A,
                         int n_fixed, hipStream_t s);

}  // namespace jpi
