// Future correction module (include/jpi_corr.h): Section "Foresight-Aligned
// Asynchronous Correction", Appendix "Architecture of Future Correction
// Module".  Every Transformer block is a pre-norm decoder block with constant
// modulation and runs through enqueue_block (the action expert's GEMM,
// batched attention and row kernels):
//   compress: the VLM tokens' keys and values come from one GEMM with the QKV
//     epilogue (no query heads, identity rotation) into a [B][T][Dh] key
//     buffer and a [B][Dh][T] transposed value buffer; the learned queries
//     are the block's rows and see those keys as their prefix.
//   predict: action MLP (a row kernel for A -> W, then a GEMM), the action
//     block with RoPE at 0..n-1, the feature concatenation [c_j ; s] gathered
//     in bf16, the fusion GEMM, two blocks over the T' tokens, the correction
//     head GEMM, a row kernel that adds its bias and one that computes the
//     confidence.
// Linear layers with bias run as: residual rows preset to the bias, fp32
// split-K GEMM slices, then the residual + norm row kernel with gate 1, which
// also gives the next block's normalised input.
#include <cstring>
#include <string>
#include <vector>

#include "../../include/jpi_corr.h"
#include "jpi_device.h"
#include "jpi_internal.h"

using namespace jpi;

namespace {

constexpr int NBLK = 4;
const char* block_prefix[NBLK] = {"qformer.", "action_block.", "blocks.0.", "blocks.1."};
enum { BLK_QF, BLK_ACT, BLK_J0, BLK_J1 };
enum BKind { B_ATTN_NORM, B_Q, B_K, B_V, B_O, B_MLP_NORM, B_GATE, B_UP, B_DOWN, B_N };
const char* bkind_suffix[B_N] = {"attn_norm.w", "q.w", "k.w", "v.w", "o.w", "mlp_norm.w", "gate.w", "up.w", "down.w"};
// tensors outside the blocks
enum GKind { G_QUERY, G_XK, G_XV, G_A0W, G_A0B, G_A1W, G_A1B, G_FUSEW, G_FUSEB, G_FINAL, G_CORRW, G_CORRB, G_CONFW,
             G_CONFB, G_N };
const char* gkind_name[G_N] = {"qformer.query", "qformer.xk.w", "qformer.xv.w", "action_mlp.0.w", "action_mlp.0.b",
                               "action_mlp.1.w", "action_mlp.1.b", "fuse.w", "fuse.b", "final_norm.w",
                               "corr_head.w", "corr_head.b", "conf_head.w", "conf_head.b"};

// u[m][n] = bf16(gelu_tanh(sum_a x[m][a] w[n][a] + b[n])), one workgroup per row
__global__ __launch_bounds__(256) void k_action_in(const float* __restrict__ x, const bf16* __restrict__ w,
                                                   const float* __restrict__ b, bf16* __restrict__ u, int W, int A) {
  __shared__ float xs[256];
  const int m = blockIdx.x;
  for (int a = threadIdx.x; a < A; a += 256) xs[a] = x[(size_t)m * A + a];
  __syncthreads();
  for (int n = threadIdx.x; n < W; n += 256) {
    float acc = 0.f;
    for (int a = 0; a < A; ++a) acc = fmaf(xs[a], static_cast<float>(w[(size_t)n * A + a]), acc);
    u[(size_t)m * W + n] = static_cast<bf16>(gelu_tanh(acc + b[n]));
  }
}

// X[b T' + j] = bf16([c[b][j] ; s_b]) with s_b = row (b n + n - 1) of the action stream
__global__ __launch_bounds__(256) void k_fuse_in(const float* __restrict__ c, const float* __restrict__ hact,
                                                 bf16* __restrict__ X, int T, int n, int W) {
  const int m = blockIdx.x, b = m / T;
  const float* cr = c + (size_t)m * W;
  const float* sr = hact + ((size_t)b * n + n - 1) * W;
  bf16* xr = X + (size_t)m * 2 * W;
  for (int k = threadIdx.x; k < W; k += 256) {
    xr[k] = static_cast<bf16>(cr[k]);
    xr[W + k] = static_cast<bf16>(sr[k]);
  }
}

// item[m] = sum_z P[z][m] + b_c, one workgroup per token row m, four columns per thread
__global__ __launch_bounds__(256) void k_item(const float* __restrict__ part, int S, int M,
                                              const float* __restrict__ bc, float* __restrict__ item, int W) {
  const int m = blockIdx.x;
  const size_t MW = (size_t)M * W;
  for (int k = 4 * threadIdx.x; k < W; k += 1024) {
    const size_t o = (size_t)m * W + k;
    f32x4 v = *reinterpret_cast<const f32x4*>(bc + k);
    for (int z = 0; z < S; ++z) v += *reinterpret_cast<const f32x4*>(part + z * MW + o);
    *reinterpret_cast<f32x4*>(item + o) = v;
  }
}

// conf[b] = sum_k w_conf[k] mean_j y[b T + j][k] + b_conf, one workgroup per rollout
__global__ __launch_bounds__(256) void k_conf(const bf16* __restrict__ y, const bf16* __restrict__ wconf,
                                              const float* __restrict__ bconf, float* __restrict__ conf, int T,
                                              int W) {
  __shared__ float red[4];
  const int b = blockIdx.x;
  float acc = 0.f;
  for (int k = threadIdx.x; k < W; k += 256) {
    float ym = 0.f;
    for (int j = 0; j < T; ++j) ym += static_cast<float>(y[((size_t)b * T + j) * W + k]);
    acc = fmaf(static_cast<float>(wconf[k]), ym / (float)T, acc);
  }
  acc = block_sum_256(acc, red);
  if (threadIdx.x == 0) conf[b] = acc + bconf[0];
}

}  // namespace

struct jpi_corr {
  jpi_corr_config cfg;
  int device = 0, n_cu = 0;
  std::string err;
  int W, nH, Dh, F, A, V, T, Bmax, Nmax, Tmax, Hmax, Mmax, Tpad;
  // weights
  void* w_blocks = nullptr;  // [NBLK][layer_elems] packed (jpi_internal.h block layout)
  size_t layer_elems = 0, off_o = 0, off_gu = 0, off_d = 0;
  float* norms = nullptr;    // [NBLK][2][W] (attention, MLP)
  void* w_xkv = nullptr;     // [2 Dh][V]: k rows in RoPE pack order, then v rows
  float* query = nullptr;    // [T'][W]
  void *w_a0 = nullptr, *w_a1 = nullptr, *w_fuse = nullptr, *w_corr = nullptr, *w_conf = nullptr;
  float *b_a0 = nullptr, *b_a1 = nullptr, *b_fuse = nullptr, *final_norm = nullptr, *b_corr = nullptr,
        *b_conf = nullptr;
  std::vector<char> have;    // [NBLK * B_N + G_N]
  bool finalized = false;
  // activations
  float* h = nullptr;
  void *y = nullptr, *q = nullptr, *o = nullptr, *z = nullptr, *u = nullptr, *xcat = nullptr;
  void *ks = nullptr, *vst = nullptr, *xk = nullptr, *xvt = nullptr;
  float *partial = nullptr, *opart = nullptr;
  float *ones = nullptr, *zeros = nullptr;
  int *tlen = nullptr, *zero_len = nullptr;
  float2 *rope_id = nullptr, *rope_act = nullptr;
};

namespace {

jpi_status cfail(jpi_corr* m, jpi_status st, const std::string& msg) {
  if (m) m->err = msg;
  return st;
}

#define CCHK(m, expr)                                                                                  \
  do {                                                                                                 \
    hipError_t e_ = (expr);                                                                            \
    if (e_ != hipSuccess) return cfail(m, JPI_ERR_HIP, std::string(#expr) + ": " + hipGetErrorString(e_)); \
  } while (0)

BlockLaunch block_base(const jpi_corr* m, int blk, int B, int H) {
  BlockLaunch b{};
  b.B = B;
  b.H = H;
  b.W = m->W;
  b.nH = m->nH;
  b.Dh = m->Dh;
  b.F = m->F;
  b.n_cu = m->n_cu;
  b.w = (const char*)m->w_blocks + (size_t)blk * m->layer_elems * 2;
  b.off_o = m->off_o;
  b.off_gu = m->off_gu;
  b.off_d = m->off_d;
  b.h = m->h;
  b.y = m->y;
  b.q = m->q;
  b.o = m->o;
  b.z = m->z;
  b.partial = m->partial;
  const int M = B * H;
  b.s_o = gemm_pick_splitk(JPI_BF16, M, m->W, m->nH * m->Dh, m->n_cu);
  b.s_d = gemm_pick_splitk(JPI_BF16, M, m->W, m->F, m->n_cu);
  b.opart = m->opart;
  b.ks = m->ks;
  b.ks_bstride = 0;
  b.vst = m->vst;
  b.vst_ld = (H + 7) / 8 * 8;
  // no earlier keys unless the caller sets them (prefix_len 0 reads none)
  b.kp = m->ks;
  b.vpt = m->vst;
  b.kp_bstride = 0;
  b.vpt_bstride = (int64_t)m->Dh * b.vst_ld;
  b.vpt_dstride = b.vst_ld;
  b.prefix_len = m->zero_len;
  b.P = 0;
  b.rope = m->rope_id;
  b.mlp_norm = m->norms + ((size_t)2 * blk + 1) * m->W;
  b.next_norm = m->norms + (size_t)2 * blk * m->W;
  b.ones = m->ones;
  b.zeros = m->zeros;
  b.eps = m->cfg.rms_eps;
  return b;
}

// out (M rows) = bias + A Wt^T via split-K slices, then y = rms(out) (1 + next_norm)
hipError_t linear_norm(jpi_corr* m, const void* A, const void* Wt, const float* bias, int M, int K,
                       const float* next_norm, hipStream_t s) {
  hipError_t e = launch_bcast_rows(bias, m->h, M, 1, m->W, s);
  if (e != hipSuccess) return e;
  GemmLaunch g{};
  g.A = A;
  g.W = Wt;
  g.M = M;
  g.N = m->W;
  g.K = K;
  g.splitk = gemm_pick_splitk(JPI_BF16, M, m->W, K, m->n_cu);
  g.n_cu = m->n_cu;
  g.epi = EPI_STORE_F32;
  g.ep.out_f32 = m->partial;
  if ((e = launch_gemm(JPI_BF16, g, s)) != hipSuccess) return e;
  RowLaunch r{};
  r.part = m->partial;
  r.S = g.splitk;
  r.M = M;
  r.W = m->W;
  r.h = m->h;
  r.gate = m->ones;
  r.scale = next_norm;
  r.shift = m->zeros;
  r.y = m->y;
  r.eps = m->cfg.rms_eps;
  return launch_resid_norm(JPI_BF16, r, false, s);
}

}  // namespace

extern "C" {

jpi_status jpi_corr_destroy(jpi_corr* m) {
  if (!m) return JPI_OK;
  (void)hipSetDevice(m->device);
  for (void* p : {m->w_blocks, (void*)m->norms, m->w_xkv, (void*)m->query, m->w_a0, m->w_a1, m->w_fuse, m->w_corr,
                  m->w_conf, (void*)m->b_a0, (void*)m->b_a1, (void*)m->b_fuse, (void*)m->final_norm,
                  (void*)m->b_corr, (void*)m->b_conf, (void*)m->h, m->y, m->q, m->o, m->z, m->u, m->xcat, m->ks,
                  m->vst, m->xk, m->xvt, (void*)m->partial, (void*)m->opart, (void*)m->ones, (void*)m->zeros,
                  (void*)m->tlen, (void*)m->zero_len, (void*)m->rope_id, (void*)m->rope_act})
    if (p) (void)hipFree(p);
  delete m;
  return JPI_OK;
}

jpi_status jpi_corr_create(const jpi_corr_config* cfg, int device, jpi_corr** out) {
  if (!cfg || !out) return JPI_ERR_ARG;
  *out = nullptr;
  const jpi_corr_config& g = *cfg;
  if (g.width < 256 || g.width % 256 || g.width > 4096 || g.n_heads < 1 || g.n_kv_heads != 1 ||
      (g.head_dim != 64 && g.head_dim != 128 && g.head_dim != 256) || (g.n_heads * g.head_dim) % 256 ||
      g.mlp_dim < 256 || g.mlp_dim % 256 || g.action_dim < 1 || g.action_dim > 256 || g.vlm_width < 256 ||
      g.vlm_width % 256 || g.n_query < 1 || g.n_query > 64 || g.max_batch < 1 || g.max_actions < 1 ||
      g.max_vlm_tokens < 1 || !(g.rms_eps > 0.f) || !(g.rope_base > 1.f) ||
      (size_t)g.max_batch * g.max_vlm_tokens > (1u << 20) || (size_t)g.max_batch * g.max_actions > (1u << 16))
    return JPI_ERR_ARG;
  if (g.max_vlm_tokens > attn_max_prefix(JPI_BF16, g.n_query)) return JPI_ERR_ARG;
  if (g.dtype != JPI_BF16) return JPI_ERR_UNSUPPORTED;
  jpi_corr* m = new jpi_corr();
  m->cfg = g;
  m->device = device;
  m->W = g.width;
  m->nH = g.n_heads;
  m->Dh = g.head_dim;
  m->F = g.mlp_dim;
  m->A = g.action_dim;
  m->V = g.vlm_width;
  m->T = g.n_query;
  m->Bmax = g.max_batch;
  m->Nmax = g.max_actions;
  m->Tmax = g.max_vlm_tokens;
  m->Hmax = g.n_query > g.max_actions ? g.n_query : g.max_actions;
  m->Mmax = g.max_batch * m->Hmax;
  m->Tpad = (g.max_vlm_tokens + 7) / 8 * 8;
  if (hipSetDevice(device) != hipSuccess) {
    jpi_corr_destroy(m);
    return JPI_ERR_HIP;
  }
  hipDeviceProp_t prop;
  if (hipGetDeviceProperties(&prop, device) != hipSuccess) {
    jpi_corr_destroy(m);
    return JPI_ERR_HIP;
  }
  m->n_cu = prop.multiProcessorCount;
  const size_t W = m->W, Dh = m->Dh, nH = m->nH, F = m->F, M = m->Mmax, B = m->Bmax;
  m->off_o = (nH + 2) * Dh * W;
  m->off_gu = m->off_o + W * nH * Dh;
  m->off_d = m->off_gu + 2 * F * W;
  m->layer_elems = m->off_d + W * F;
  // attention scratch: the Q-Former (T' rows over T keys) or a block over its own rows
  const int nch_q = attn_n_chunks(JPI_BF16, m->Tmax, m->T), nch_b = attn_n_chunks(JPI_BF16, 0, m->Hmax);
  const size_t attn_q = flash_scratch_bytes((int)B, (int)nH, m->T, (int)Dh, nch_q);
  const size_t attn_b = flash_scratch_bytes((int)B, (int)nH, m->Hmax, (int)Dh, nch_b);
  const size_t rope_rows = (size_t)B * (m->Tmax > m->Hmax ? m->Tmax : m->Hmax);
  bool ok = true;
  auto alloc = [&](void** p, size_t bytes) {
    if (ok && hipMalloc(p, bytes) != hipSuccess) ok = false;
  };
  alloc(&m->w_blocks, (size_t)NBLK * m->layer_elems * 2);
  alloc((void**)&m->norms, (size_t)NBLK * 2 * W * 4);
  alloc(&m->w_xkv, 2 * Dh * m->V * 2);
  alloc((void**)&m->query, (size_t)m->T * W * 4);
  alloc(&m->w_a0, W * m->A * 2);
  alloc(&m->w_a1, W * W * 2);
  alloc(&m->w_fuse, W * 2 * W * 2);
  alloc(&m->w_corr, W * W * 2);
  alloc(&m->w_conf, W * 2);
  alloc((void**)&m->b_a0, W * 4);
  alloc((void**)&m->b_a1, W * 4);
  alloc((void**)&m->b_fuse, W * 4);
  alloc((void**)&m->final_norm, W * 4);
  alloc((void**)&m->b_corr, W * 4);
  alloc((void**)&m->b_conf, 4);
  alloc((void**)&m->h, M * W * 4);
  alloc(&m->y, M * W * 2);
  alloc(&m->q, M * nH * Dh * 2);
  alloc(&m->o, M * nH * Dh * 2);
  alloc(&m->z, M * F * 2);
  alloc(&m->u, M * W * 2);
  alloc(&m->xcat, B * m->T * 2 * W * 2);
  alloc(&m->ks, M * Dh * 2);
  alloc(&m->vst, B * Dh * ((m->Hmax + 7) / 8 * 8) * 2);
  alloc(&m->xk, B * m->Tmax * Dh * 2);
  alloc(&m->xvt, B * Dh * m->Tpad * 2);
  alloc((void**)&m->partial, (size_t)16 * M * W * 4);
  alloc((void**)&m->opart, attn_q > attn_b ? attn_q : attn_b);
  alloc((void**)&m->ones, W * 4);
  alloc((void**)&m->zeros, W * 4);
  alloc((void**)&m->tlen, B * 4);
  alloc((void**)&m->zero_len, B * 4);
  alloc((void**)&m->rope_id, rope_rows * (Dh / 2) * sizeof(float2));
  alloc((void**)&m->rope_act, B * m->Nmax * (Dh / 2) * sizeof(float2));
  if (!ok) {
    (void)hipGetLastError();
    jpi_corr_destroy(m);
    return JPI_ERR_OOM;
  }
  if (launch_fill_f32(m->ones, (int)W, 1.0f, 0) != hipSuccess || launch_fill_f32(m->zeros, (int)W, 0.0f, 0) != hipSuccess ||
      launch_fill_i32(m->zero_len, (int)B, 0, 0) != hipSuccess ||
      launch_identity_rope(m->rope_id, (int)(rope_rows * (Dh / 2)), 0) != hipSuccess ||
      hipDeviceSynchronize() != hipSuccess) {
    jpi_corr_destroy(m);
    return JPI_ERR_HIP;
  }
  m->have.assign((size_t)NBLK * B_N + G_N, 0);
  *out = m;
  return JPI_OK;
}

jpi_status jpi_corr_set_weight(jpi_corr* m, const char* name, const void* data, int64_t n_elems, jpi_dtype dt,
                               int is_device, void* stream) {
  if (!m) return JPI_ERR_ARG;
  if (!name || !data) return cfail(m, JPI_ERR_ARG, "jpi_corr_set_weight: name or data is NULL");
  int blk = -1, kind = -1;
  for (int k = 0; k < G_N; ++k)
    if (strcmp(name, gkind_name[k]) == 0) kind = k;
  if (kind < 0)
    for (int bl = 0; bl < NBLK && kind < 0; ++bl) {
      const size_t pl = strlen(block_prefix[bl]);
      if (strncmp(name, block_prefix[bl], pl) != 0) continue;
      for (int k = 0; k < B_N; ++k)
        if (strcmp(name + pl, bkind_suffix[k]) == 0) {
          blk = bl;
          kind = k;
        }
    }
  if (kind < 0) return cfail(m, JPI_ERR_ARG, std::string("unknown tensor name: ") + name);
  const int64_t W = m->W, Dh = m->Dh, nH = m->nH, F = m->F;
  int64_t want = 0;
  bool vec = false;
  if (blk >= 0) {
    switch (kind) {
      case B_ATTN_NORM: case B_MLP_NORM: want = W; vec = true; break;
      case B_Q: want = nH * Dh * W; break;
      case B_K: case B_V: want = Dh * W; break;
      case B_O: want = W * nH * Dh; break;
      case B_GATE: case B_UP: want = F * W; break;
      case B_DOWN: want = W * F; break;
    }
  } else {
    switch (kind) {
      case G_QUERY: want = (int64_t)m->T * W; vec = true; break;
      case G_XK: case G_XV: want = Dh * m->V; break;
      case G_A0W: want = W * m->A; break;
      case G_A1W: case G_CORRW: want = W * W; break;
      case G_FUSEW: want = W * 2 * W; break;
      case G_CONFW: want = W; break;
      case G_CONFB: want = 1; vec = true; break;
      default: want = W; vec = true; break;  // biases, final norm
    }
  }
  if (n_elems != want)
    return cfail(m, JPI_ERR_SHAPE, std::string(name) + ": expected " + std::to_string(want) + " elements, got " +
                                       std::to_string(n_elems));
  if (dt != (vec ? JPI_F32 : JPI_BF16))
    return cfail(m, JPI_ERR_DTYPE, std::string(name) + (vec ? ": vectors must be JPI_F32" : ": matrices must be JPI_BF16"));
  CCHK(m, hipSetDevice(m->device));
  hipStream_t s = (hipStream_t)stream;
  const hipMemcpyKind ck = is_device ? hipMemcpyDeviceToDevice : hipMemcpyHostToDevice;
  const size_t bytes = (size_t)n_elems * (vec ? 4 : 2);
  hipError_t e = hipSuccess;
  if (blk >= 0) {
    char* lay = (char*)m->w_blocks + (size_t)blk * m->layer_elems * 2;
    if (vec) {
      e = hipMemcpyAsync(m->norms + ((size_t)2 * blk + (kind == B_MLP_NORM)) * W, data, bytes, ck, s);
    } else if (kind == B_O || kind == B_DOWN) {
      e = hipMemcpyAsync(lay + (kind == B_O ? m->off_o : m->off_d) * 2, data, bytes, ck, s);
    } else {
      const BlockMatrix bm = kind == B_Q ? BM_Q : kind == B_K ? BM_K : kind == B_V ? BM_V : kind == B_GATE ? BM_GATE : BM_UP;
      std::vector<int> map((size_t)(n_elems / W));
      for (size_t r = 0; r < map.size(); ++r) map[r] = block_pack_row(bm, (int)r, (int)nH, (int)Dh);
      e = upload_rows(kind == B_GATE || kind == B_UP ? lay + m->off_gu * 2 : lay, map, (int)(W * 2), data,
                      is_device != 0, s);
    }
  } else if (kind == G_XK || kind == G_XV) {
    // [k rows (RoPE pack order, rotated by the identity) | v rows] over d_VLM columns
    std::vector<int> map((size_t)Dh);
    for (int r = 0; r < (int)Dh; ++r) map[r] = block_pack_row(kind == G_XK ? BM_K : BM_V, r, 0, (int)Dh);
    e = upload_rows(m->w_xkv, map, m->V * 2, data, is_device != 0, s);
  } else {
    void* dst = nullptr;
    switch (kind) {
      case G_QUERY: dst = m->query; break;
      case G_A0W: dst = m->w_a0; break;
      case G_A0B: dst = m->b_a0; break;
      case G_A1W: dst = m->w_a1; break;
      case G_A1B: dst = m->b_a1; break;
      case G_FUSEW: dst = m->w_fuse; break;
      case G_FUSEB: dst = m->b_fuse; break;
      case G_FINAL: dst = m->final_norm; break;
      case G_CORRW: dst = m->w_corr; break;
      case G_CORRB: dst = m->b_corr; break;
      case G_CONFW: dst = m->w_conf; break;
      case G_CONFB: dst = m->b_conf; break;
    }
    e = hipMemcpyAsync(dst, data, bytes, ck, s);
  }
  if (e == hipSuccess) e = hipStreamSynchronize(s);
  if (e != hipSuccess) return cfail(m, JPI_ERR_HIP, std::string("jpi_corr_set_weight: ") + hipGetErrorString(e));
  m->have[blk >= 0 ? (size_t)blk * B_N + kind : (size_t)NBLK * B_N + kind] = 1;
  m->finalized = false;
  return JPI_OK;
}

jpi_status jpi_corr_finalize_weights(jpi_corr* m, void* stream) {
  (void)stream;
  if (!m) return JPI_ERR_ARG;
  for (int bl = 0; bl < NBLK; ++bl)
    for (int k = 0; k < B_N; ++k)
      if (!m->have[(size_t)bl * B_N + k])
        return cfail(m, JPI_ERR_STATE, std::string("missing tensor ") + block_prefix[bl] + bkind_suffix[k]);
  for (int k = 0; k < G_N; ++k)
    if (!m->have[(size_t)NBLK * B_N + k]) return cfail(m, JPI_ERR_STATE, std::string("missing tensor ") + gkind_name[k]);
  m->finalized = true;
  return JPI_OK;
}

jpi_status jpi_corr_compress(jpi_corr* m, const void* vlm_state, int batch, int n_tokens, float* state_out,
                             void* stream) {
  if (!m) return JPI_ERR_ARG;
  if (!vlm_state || !state_out) return cfail(m, JPI_ERR_ARG, "jpi_corr_compress: vlm_state or state_out is NULL");
  if (batch < 1 || batch > m->Bmax || n_tokens < 1 || n_tokens > m->Tmax)
    return cfail(m, JPI_ERR_ARG, "jpi_corr_compress: batch or n_tokens outside [1, max_batch] / [1, max_vlm_tokens]");
  if (!m->finalized) return cfail(m, JPI_ERR_STATE, "jpi_corr_compress: weights are not finalized");
  CCHK(m, hipSetDevice(m->device));
  hipStream_t s = (hipStream_t)stream;
  const int W = m->W, Dh = m->Dh, T = m->T;
  CCHK(m, launch_fill_i32(m->tlen, batch, n_tokens, s));
  // the VLM tokens' keys and values (no query heads, no rotation)
  GemmLaunch g{};
  g.A = vlm_state;
  g.W = m->w_xkv;
  g.M = batch * n_tokens;
  g.N = 2 * Dh;
  g.K = m->V;
  g.splitk = 1;
  g.n_cu = m->n_cu;
  g.epi = EPI_QKV;
  g.ep.q = nullptr;
  g.ep.ks = m->xk;
  g.ep.ks_bstride = (int64_t)m->Tmax * Dh;
  g.ep.vst = m->xvt;
  g.ep.vst_ld = m->Tpad;
  g.ep.rope = m->rope_id;
  g.ep.n_heads = 0;
  g.ep.head_dim = Dh;
  g.ep.horizon = n_tokens;
  CCHK(m, launch_gemm(JPI_BF16, g, s));
  // learned queries -> one block whose rows also see the VLM tokens
  CCHK(m, launch_bcast_rows(m->query, m->h, batch * T, T, W, s));
  CCHK(m, launch_norm_rows(m->h, m->norms, m->y, batch * T, W, m->cfg.rms_eps, s));
  BlockLaunch b = block_base(m, BLK_QF, batch, T);
  b.kp = m->xk;
  b.vpt = m->xvt;
  b.kp_bstride = (int64_t)m->Tmax * Dh;
  b.vpt_bstride = (int64_t)Dh * m->Tpad;
  b.vpt_dstride = m->Tpad;
  b.prefix_len = m->tlen;
  b.P = n_tokens;
  CCHK(m, enqueue_block(b, s));
  CCHK(m, hipMemcpyAsync(state_out, m->h, (size_t)batch * T * W * 4, hipMemcpyDeviceToDevice, s));
  return JPI_OK;
}

jpi_status jpi_corr_predict(jpi_corr* m, const float* state, const float* actions, int batch, int n_actions,
                            float* item_out, float* conf_out, void* stream) {
  if (!m) return JPI_ERR_ARG;
  if (!state || !actions || !item_out || !conf_out)
    return cfail(m, JPI_ERR_ARG, "jpi_corr_predict: NULL state, actions or output");
  if (batch < 1 || batch > m->Bmax || n_actions < 1 || n_actions > m->Nmax)
    return cfail(m, JPI_ERR_ARG, "jpi_corr_predict: batch or n_actions outside [1, max_batch] / [1, max_actions]");
  if (!m->finalized) return cfail(m, JPI_ERR_STATE, "jpi_corr_predict: weights are not finalized");
  CCHK(m, hipSetDevice(m->device));
  hipStream_t s = (hipStream_t)stream;
  const int W = m->W, Dh = m->Dh, T = m->T, n = n_actions, Ma = batch * n, Mq = batch * T;
  const float* nrm = m->norms;
  // action branch: MLP, then the block with RoPE at positions 0 .. n-1
  CCHK(m, launch_rope_table(m->zero_len, m->rope_act, batch, n, Dh, m->cfg.rope_base, s));
  hipLaunchKernelGGL(k_action_in, dim3(Ma), dim3(256), 0, s, actions, (const bf16*)m->w_a0, m->b_a0, (bf16*)m->u, W,
                     m->A);
  CCHK(m, hipGetLastError());
  CCHK(m, linear_norm(m, m->u, m->w_a1, m->b_a1, Ma, W, nrm + (size_t)2 * BLK_ACT * W, s));
  BlockLaunch b = block_base(m, BLK_ACT, batch, n);
  b.rope = m->rope_act;
  CCHK(m, enqueue_block(b, s));
  // [c_j ; s] -> fusion projection -> two blocks -> final norm
  hipLaunchKernelGGL(k_fuse_in, dim3(Mq), dim3(256), 0, s, state, m->h, (bf16*)m->xcat, T, n, W);
  CCHK(m, hipGetLastError());
  CCHK(m, linear_norm(m, m->xcat, m->w_fuse, m->b_fuse, Mq, 2 * W, nrm + (size_t)2 * BLK_J0 * W, s));
  b = block_base(m, BLK_J0, batch, T);
  b.next_norm = nrm + (size_t)2 * BLK_J1 * W;
  CCHK(m, enqueue_block(b, s));
  b = block_base(m, BLK_J1, batch, T);
  b.next_norm = m->final_norm;
  CCHK(m, enqueue_block(b, s));
  // heads
  GemmLaunch g{};
  g.A = m->y;
  g.W = m->w_corr;
  g.M = Mq;
  g.N = W;
  g.K = W;
  g.splitk = gemm_pick_splitk(JPI_BF16, Mq, W, W, m->n_cu);
  g.n_cu = m->n_cu;
  g.epi = EPI_STORE_F32;
  g.ep.out_f32 = m->partial;
  CCHK(m, launch_gemm(JPI_BF16, g, s));
  hipLaunchKernelGGL(k_conf, dim3(batch), dim3(256), 0, s, (const bf16*)m->y, (const bf16*)m->w_conf, m->b_conf,
                     conf_out, T, W);
  CCHK(m, hipGetLastError());
  hipLaunchKernelGGL(k_item, dim3(Mq), dim3(256), 0, s, m->partial, g.splitk, Mq, m->b_corr, item_out, W);
  CCHK(m, hipGetLastError());
  return JPI_OK;
}

const char* jpi_corr_last_error(const jpi_corr* m) { return m ? m->err.c_str() : "module is NULL"; }

}  // extern "C"
