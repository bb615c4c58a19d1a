// libjpi runtime: context, weight packing, resident buffers, the modulation
// table cache and the HIP-graph cache, behind the C ABI of include/jpi.h.
//
// Packed weight layout on the device (dtype = cfg.dtype, row-major [out][in]):
//   per layer, contiguous:  QKV [(nH+2)Dh][W] | O [W][nH Dh] | GU [2F][W] | D [W][F]
//   QKV rows: q heads then k then v.  Inside each q head and inside k, 32-row
//   group t holds original rows 16t..16t+15 followed by Dh/2+16t..Dh/2+16t+15,
//   so a GEMM output tile sees each RoPE pair (d, d + Dh/2) in one lane.
//   GU rows: 32-row group t holds gate rows 16t..16t+15 then up rows
//   16t..16t+15, so GeGLU pairs also land in one lane.
//   Modulation: all attn_mod / mlp_mod / final_mod rows stacked into one
//   [(6L+2)W][W] matrix; row block 2l is layer l's attention norm, 2l+1 its
//   MLP norm, 2L the final norm (scale | shift | gate, W rows each).
//
// Per denoise step k the modulation depends only on t_k = 1 - k/N, so the
// table [N + 1][(6L+2)W] of all (scale, shift, gate) is computed once per
// (weights, N) and read by the step kernels; row N is t = 0, the time of
// committed rows when they are treated as clean actions.
#include <hip/hip_runtime.h>

#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <map>
#include <string>
#include <tuple>
#include <vector>

#include "jpi_internal.h"

using namespace jpi;

namespace {

enum TensorKind {
  T_IN_W, T_IN_B, T_TIME0_W, T_TIME0_B, T_TIME1_W, T_TIME1_B, T_ATTN_MOD_W, T_ATTN_MOD_B, T_Q, T_K, T_V, T_O,
  T_MLP_MOD_W, T_MLP_MOD_B, T_GATE, T_UP, T_DOWN, T_FINAL_MOD_W, T_FINAL_MOD_B, T_OUT_W, T_OUT_B,
  // action-time variant
  T_ATM_IN_W, T_ATM_IN_B, T_ATM_OUT_W, T_ATM_OUT_B, T_STATE_W, T_STATE_B, T_FINAL_NORM, T_ATTN_NORM, T_MLP_NORM,
  T_NKINDS
};

const char* kind_suffix[T_NKINDS] = {"action_in.w", "action_in.b", "time_mlp.0.w", "time_mlp.0.b", "time_mlp.1.w",
                                     "time_mlp.1.b", "attn_mod.w", "attn_mod.b", "q.w", "k.w", "v.w", "o.w",
                                     "mlp_mod.w", "mlp_mod.b", "gate.w", "up.w", "down.w", "final_mod.w",
                                     "final_mod.b", "action_out.w", "action_out.b", "action_time_mlp_in.w",
                                     "action_time_mlp_in.b", "action_time_mlp_out.w", "action_time_mlp_out.b",
                                     "state_proj.w", "state_proj.b", "final_norm.w", "attn_norm.w", "mlp_norm.w"};

bool kind_is_layer(int k) { return (k >= T_ATTN_MOD_W && k <= T_DOWN) || k == T_ATTN_NORM || k == T_MLP_NORM; }
bool kind_is_matrix(int k) {
  return k == T_IN_W || k == T_TIME0_W || k == T_TIME1_W || k == T_ATTN_MOD_W || k == T_Q || k == T_K || k == T_V ||
         k == T_O || k == T_MLP_MOD_W || k == T_GATE || k == T_UP || k == T_DOWN || k == T_FINAL_MOD_W ||
         k == T_OUT_W || k == T_ATM_IN_W || k == T_ATM_OUT_W || k == T_STATE_W;
}
// tensors each variant takes
bool kind_in_variant(int k, int variant) {
  const bool adarms = k == T_TIME0_W || k == T_TIME0_B || k == T_TIME1_W || k == T_TIME1_B || k == T_ATTN_MOD_W ||
                      k == T_ATTN_MOD_B || k == T_MLP_MOD_W || k == T_MLP_MOD_B || k == T_FINAL_MOD_W ||
                      k == T_FINAL_MOD_B;
  const bool action_time = k >= T_ATM_IN_W && k <= T_MLP_NORM;
  return variant == JPI_VARIANT_ACTION_TIME ? !adarms : !action_time;
}

struct GraphKey {
  int batch, prefix, n_steps, n_fixed, n_corr;
  bool committed_t0;  // committed rows modulated at t = 0
  bool persist;       // the single-launch path and the multi-kernel path capture different graphs
  bool operator<(const GraphKey& o) const {
    return std::tie(batch, prefix, n_steps, n_fixed, n_corr, committed_t0, persist) <
           std::tie(o.batch, o.prefix, o.n_steps, o.n_fixed, o.n_corr, o.committed_t0, o.persist);
  }
};

__global__ void k_scatter_rows(const char* __restrict__ src, char* __restrict__ dst, const int* __restrict__ map,
                               int rows, int row_bytes) {
  const int r = blockIdx.x;
  if (r >= rows) return;
  const char* s = src + (size_t)r * row_bytes;
  char* d = dst + (size_t)map[r] * row_bytes;
  for (int i = threadIdx.x * 4; i < row_bytes; i += blockDim.x * 4) *reinterpret_cast<int*>(d + i) = *reinterpret_cast<const int*>(s + i);
}

}  // namespace

struct jpi_ctx {
  jpi_config cfg;
  int device = 0, n_cu = 0;
  std::string err;
  int L, W, nH, Dh, F, A, H, Bmax, Pmax, Mmax;
  int Cmax;  // correction tokens per rollout, upper bound
  jpi_dtype dt;
  size_t esz;
  int R;  // modulation rows (6L+2)W
  // packed weights
  void* w_layers = nullptr;
  size_t layer_elems = 0, off_o = 0, off_gu = 0, off_d = 0;
  void *w_in = nullptr, *w_t0 = nullptr, *w_t1 = nullptr, *w_mod = nullptr, *w_out = nullptr;
  float *b_in = nullptr, *b_t0 = nullptr, *b_t1 = nullptr, *b_mod = nullptr, *b_out = nullptr;
  std::vector<char> have;  // per (kind, layer)
  bool finalized = false;
  // prefix and state
  void *kp = nullptr, *vp = nullptr;  // [L][Bmax][Pmax][Dh] as bound
  void* vpt = nullptr;                 // [L][Bmax][Dh][Ppad] prefix V transposed at bind time
  int Ppad = 0;                        // Pmax + horizon rounded up to a multiple of 8
  int* d_prefix_len = nullptr;
  int* h_prefix_len = nullptr;  // pinned staging
  int batch = 0, prefix = 0;
  bool prefix_bound = false;
  float2* rope_tab = nullptr;  // [batch][n_corr + H][Dh/2] at positions prefix_len + r
  int rope_rows = 0;           // suffix rows per rollout the table was built for
  float* committed = nullptr;
  int n_fixed = 0;
  float* corr = nullptr;       // [Bmax][Cmax][W] correction tokens
  int n_corr = 0;
  bool committed_t0 = false;   // committed rows take the t = 0 modulation
  // action-time variant: weights, robot state and the state token's pass
  void *w_atm_a = nullptr, *w_atm_t = nullptr, *w_atm_out = nullptr, *w_state = nullptr;  // [W][W] x3, [W][state_dim]
  float *b_atm_in = nullptr, *b_atm_out = nullptr, *b_state = nullptr;
  float* norms = nullptr;      // [2L+1][W]: attention and MLP norm of each layer, then the final norm
  float *ones = nullptr, *zeros = nullptr;
  float* state = nullptr;      // [Bmax][state_dim]
  bool state_bound = false;
  int* d_plen1 = nullptr;      // prefix_len + 1: the action rows also see the state slot
  float2* rope_s = nullptr;    // [Bmax][Dh/2] the state token's rotation (position prefix_len)
  float* hs = nullptr;         // [Bmax][W] state token residual
  void *ys = nullptr, *ks_s = nullptr, *vst_s = nullptr, *u2 = nullptr;
  // activations
  float *x = nullptr, *h = nullptr;
  void *y = nullptr, *q = nullptr, *ks = nullptr, *vst = nullptr, *o = nullptr, *z = nullptr;
  float* partial = nullptr;  // split-K slices of the O / Down projections
  size_t partial_cap = 0;
  float* opart = nullptr;    // attention chunk partials (O, running max, running sum)
  size_t attn_cap = 0;
  // caches
  std::map<int, float*> tables;
  std::map<GraphKey, hipGraphExec_t> graphs;
  hipStream_t cap_stream = nullptr;
  // single-launch (persistent) path
  unsigned* pflags = nullptr;  // completion flag lines of the single-launch kernel (one per workgroup)
  unsigned persist_spin = 0;   // bound of the single-launch kernel's waits in polls (0: the default)
  unsigned* perr = nullptr;    // set when a wait for producers timed out
  unsigned long long* ptrace = nullptr;  // trace build only: [max grid][trace_slots] phase timestamps
  int trace_slots = 0, trace_grid = 0, trace_used = 0;
  int persist_occ = -1;        // workgroups per CU the persistent kernel fits (-1: not queried)
  void* w_frag = nullptr;      // layer weights with every matrix fragment-ordered
  bool frag_ready = false;     // w_frag matches w_layers
  void *ysw = nullptr, *osw = nullptr, *zsw = nullptr, *qsw = nullptr;  // fragment-ordered activations
  // measurement: events around every launch of one kernel kind
  int timed_kind = JPI_KERNEL_NONE;
  std::vector<hipEvent_t> ev;  // pairs (start, end)
  int ev_used = 0;
};

namespace {

thread_local std::string g_noctx_err;

jpi_status fail(jpi_ctx* c, jpi_status st, const std::string& msg) {
  if (c) c->err = msg;
  else g_noctx_err = msg;
  return st;
}

#define HIPCHK(c, expr)                                                                     \
  do {                                                                                      \
    hipError_t e_ = (expr);                                                                 \
    if (e_ != hipSuccess)                                                                   \
      return fail((c), e_ == hipErrorOutOfMemory ? JPI_ERR_OOM : JPI_ERR_HIP,               \
                  std::string(#expr) + ": " + hipGetErrorString(e_));                       \
  } while (0)

jpi_status dmalloc(jpi_ctx* c, void** p, size_t bytes) {
  *p = nullptr;
  if (bytes == 0) bytes = 256;
  hipError_t e = hipMalloc(p, bytes);
  if (e != hipSuccess) {
    *p = nullptr;
    (void)hipGetLastError();
    return fail(c, JPI_ERR_OOM, "hipMalloc of " + std::to_string(bytes) + " bytes failed: " + hipGetErrorString(e));
  }
  return JPI_OK;
}

#define TRY(expr)                    \
  do {                               \
    jpi_status st_ = (expr);         \
    if (st_ != JPI_OK) return st_;   \
  } while (0)

void drop_graphs(jpi_ctx* c) {
  for (auto& kv : c->graphs) (void)hipGraphExecDestroy(kv.second);
  c->graphs.clear();
}

void drop_events(jpi_ctx* c) {
  for (hipEvent_t e : c->ev) (void)hipEventDestroy(e);
  c->ev.clear();
  c->ev_used = 0;
}

void drop_tables(jpi_ctx* c) {
  for (auto& kv : c->tables) (void)hipFree(kv.second);
  c->tables.clear();
}

int64_t expected_elems(const jpi_ctx* c, int k) {
  const int64_t W = c->W, A = c->A, Dh = c->Dh, nH = c->nH, F = c->F;
  switch (k) {
    case T_IN_W: return W * A;
    case T_IN_B: return W;
    case T_TIME0_W: case T_TIME1_W: return W * W;
    case T_TIME0_B: case T_TIME1_B: return W;
    case T_ATTN_MOD_W: case T_MLP_MOD_W: return 3 * W * W;
    case T_ATTN_MOD_B: case T_MLP_MOD_B: return 3 * W;
    case T_Q: return nH * Dh * W;
    case T_K: case T_V: return Dh * W;
    case T_O: return W * nH * Dh;
    case T_GATE: case T_UP: return F * W;
    case T_DOWN: return W * F;
    case T_FINAL_MOD_W: return 2 * W * W;
    case T_FINAL_MOD_B: return 2 * W;
    case T_OUT_W: return A * W;
    case T_OUT_B: return A;
    case T_ATM_IN_W: return W * 2 * W;
    case T_ATM_OUT_W: return W * W;
    case T_ATM_IN_B: case T_ATM_OUT_B: case T_STATE_B: case T_FINAL_NORM: case T_ATTN_NORM: case T_MLP_NORM: return W;
    case T_STATE_W: return W * c->cfg.state_dim;
  }
  return -1;
}

// Parse "layers.{l}.<suffix>" or a global name.  Returns false if unknown.
bool parse_name(const jpi_ctx* c, const char* name, int* kind, int* layer) {
  *layer = -1;
  const char* pre = "layers.";
  if (strncmp(name, pre, 7) == 0) {
    const char* p = name + 7;
    if (*p < '0' || *p > '9') return false;
    char* end = nullptr;
    long l = strtol(p, &end, 10);
    if (!end || *end != '.' || l < 0 || l >= c->L) return false;
    for (int k = 0; k < T_NKINDS; ++k)
      if (kind_is_layer(k) && kind_in_variant(k, c->cfg.variant) && strcmp(end + 1, kind_suffix[k]) == 0) {
        *kind = k;
        *layer = (int)l;
        return true;
      }
    return false;
  }
  for (int k = 0; k < T_NKINDS; ++k)
    if (!kind_is_layer(k) && kind_in_variant(k, c->cfg.variant) && strcmp(name, kind_suffix[k]) == 0) {
      *kind = k;
      return true;
    }
  return false;
}

int have_index(const jpi_ctx* c, int kind, int layer) {
  return kind_is_layer(kind) ? T_NKINDS + layer * T_NKINDS + kind : kind;
}

// packed row of source row r for q / k (RoPE pairs (d, d + Dh/2) in one 32-row group)
int rope_pack_row(int r, int Dh) {
  const int half = Dh / 2;
  const int dd = r % Dh, head = r / Dh;
  const int hi = dd >= half ? 1 : 0;
  const int d = dd - hi * half;
  return head * Dh + (d / 16) * 32 + hi * 16 + (d % 16);
}

}  // namespace

extern "C" {

int jpi_abi_version(void) { return JPI_ABI_VERSION; }

const char* jpi_status_str(jpi_status s) {
  switch (s) {
    case JPI_OK: return "ok";
    case JPI_ERR_ARG: return "invalid argument";
    case JPI_ERR_SHAPE: return "shape mismatch";
    case JPI_ERR_DTYPE: return "dtype mismatch";
    case JPI_ERR_STATE: return "invalid call order";
    case JPI_ERR_OOM: return "device out of memory";
    case JPI_ERR_HIP: return "HIP runtime error";
    case JPI_ERR_UNSUPPORTED: return "unsupported";
  }
  return "unknown status";
}

const char* jpi_last_error(const jpi_ctx* ctx) { return ctx ? ctx->err.c_str() : g_noctx_err.c_str(); }

jpi_status jpi_destroy(jpi_ctx* c) {
  if (!c) return JPI_OK;
  (void)hipSetDevice(c->device);
  (void)hipDeviceSynchronize();
  drop_graphs(c);
  drop_tables(c);
  drop_events(c);
  void* bufs[] = {c->w_atm_a, c->w_atm_t, c->w_atm_out, c->w_state, c->b_atm_in, c->b_atm_out, c->b_state, c->norms,
                  c->ones, c->zeros, c->state, c->d_plen1, c->rope_s, c->hs, c->ys, c->ks_s, c->vst_s, c->u2,
                  c->w_layers, c->w_in, c->w_t0, c->w_t1, c->w_mod, c->w_out, c->b_in, c->b_t0, c->b_t1, c->b_mod,
                  c->b_out, c->kp, c->vp, c->vpt, c->d_prefix_len, c->rope_tab, c->committed, c->corr, c->x, c->h, c->y, c->q, c->ks,
                  c->vst, c->o, c->z, c->partial, c->opart, c->pflags, c->perr, c->w_frag, c->ysw, c->osw,
                  c->zsw, c->qsw, c->ptrace};
  for (void* p : bufs)
    if (p) (void)hipFree(p);
  if (c->h_prefix_len) (void)hipHostFree(c->h_prefix_len);
  if (c->cap_stream) (void)hipStreamDestroy(c->cap_stream);
  delete c;
  return JPI_OK;
}

jpi_status jpi_create(const jpi_config* cfg, int device, jpi_ctx** out) {
  if (!out) return fail(nullptr, JPI_ERR_ARG, "jpi_create: out is NULL");
  *out = nullptr;
  if (!cfg) return fail(nullptr, JPI_ERR_ARG, "jpi_create: cfg is NULL");
  const jpi_config& g = *cfg;
  if (g.n_layers < 1 || g.width < 1 || g.n_heads < 1 || g.n_kv_heads < 1 || g.head_dim < 1 || g.mlp_dim < 1 ||
      g.action_dim < 1 || g.horizon < 1 || g.max_batch < 1 || g.max_prefix < 0)
    return fail(nullptr, JPI_ERR_ARG, "jpi_create: every dimension must be positive");
  if (g.max_corr < 0 || g.max_corr > 64) return fail(nullptr, JPI_ERR_ARG, "jpi_create: max_corr outside [0, 64]");
  if (g.variant != JPI_VARIANT_ADARMS && g.variant != JPI_VARIANT_ACTION_TIME)
    return fail(nullptr, JPI_ERR_ARG, "jpi_create: unknown variant");
  if (g.variant == JPI_VARIANT_ACTION_TIME ? (g.state_dim < 1 || g.state_dim > 4096 || g.max_corr != 0 ||
                                              g.max_prefix < 1)
                                           : g.state_dim != 0)
    return fail(nullptr, JPI_ERR_ARG, "jpi_create: the action-time variant needs 1 <= state_dim <= 4096, max_corr 0 "
                                      "and max_prefix >= 1; the default variant state_dim 0");
  const int seq_max = g.horizon + g.max_corr;  // suffix rows per rollout
  if (g.n_kv_heads != 1 || g.n_heads % g.n_kv_heads != 0)
    return fail(nullptr, JPI_ERR_ARG, "jpi_create: this version implements exactly one shared KV head");
  if (g.head_dim != 64 && g.head_dim != 128 && g.head_dim != 256)
    return fail(nullptr, JPI_ERR_ARG, "jpi_create: head_dim must be 64, 128 or 256");
  if (g.width % 64 != 0 || g.mlp_dim % 64 != 0 || (g.n_heads * g.head_dim) % 64 != 0)
    return fail(nullptr, JPI_ERR_ARG, "jpi_create: width, mlp_dim and n_heads*head_dim must be multiples of 64");
  if (g.dtype != JPI_F32 && g.dtype != JPI_BF16) return fail(nullptr, JPI_ERR_ARG, "jpi_create: bad dtype");
  if (!(g.rms_eps > 0.f) || !(g.rope_base > 1.f))
    return fail(nullptr, JPI_ERR_ARG, "jpi_create: rms_eps must be > 0 and rope_base > 1");
  if ((long long)g.max_batch * seq_max > (1 << 20))
    return fail(nullptr, JPI_ERR_ARG, "jpi_create: max_batch*(horizon+max_corr) too large");
  if (g.max_prefix > attn_max_prefix(g.dtype, seq_max))
    return fail(nullptr, JPI_ERR_ARG, "jpi_create: max_prefix above " +
                                          std::to_string(attn_max_prefix(g.dtype, seq_max)));
  if (g.action_dim > 64) return fail(nullptr, JPI_ERR_ARG, "jpi_create: action_dim above 64");
  if (g.width > 4096) return fail(nullptr, JPI_ERR_ARG, "jpi_create: width above 4096");

  int ndev = 0;
  if (hipGetDeviceCount(&ndev) != hipSuccess || device < 0 || device >= ndev) {
    (void)hipGetLastError();
    return fail(nullptr, JPI_ERR_HIP, "jpi_create: no HIP device " + std::to_string(device));
  }
  jpi_ctx* c = new jpi_ctx();
  c->cfg = g;
  c->device = device;
  c->L = g.n_layers;
  c->W = g.width;
  c->nH = g.n_heads;
  c->Dh = g.head_dim;
  c->F = g.mlp_dim;
  c->A = g.action_dim;
  c->H = g.horizon;
  c->Bmax = g.max_batch;
  c->Pmax = g.max_prefix;
  c->Cmax = g.max_corr;
  c->Mmax = g.max_batch * seq_max;
  c->dt = g.dtype;
  c->esz = g.dtype == JPI_BF16 ? 2 : 4;
  c->R = (6 * c->L + 2) * c->W;
  c->have.assign(T_NKINDS + (size_t)c->L * T_NKINDS, 0);

  auto cleanup_fail = [&](jpi_status st) {
    std::string msg = c->err;
    jpi_destroy(c);
    return fail(nullptr, st, msg);
  };
  if (hipSetDevice(device) != hipSuccess) {
    (void)hipGetLastError();
    return cleanup_fail(fail(c, JPI_ERR_HIP, "hipSetDevice failed"));
  }
  hipDeviceProp_t prop;
  if (hipGetDeviceProperties(&prop, device) != hipSuccess) return cleanup_fail(fail(c, JPI_ERR_HIP, "props"));
  c->n_cu = prop.multiProcessorCount;
  if (hipStreamCreateWithFlags(&c->cap_stream, hipStreamNonBlocking) != hipSuccess)
    return cleanup_fail(fail(c, JPI_ERR_HIP, "stream create failed"));

  const size_t es = c->esz;
  const size_t W = c->W, Dh = c->Dh, nH = c->nH, F = c->F, A = c->A, M = c->Mmax;
  c->layer_elems = (nH + 2) * Dh * W + W * nH * Dh + 2 * F * W + W * F;
  c->off_o = (nH + 2) * Dh * W;
  c->off_gu = c->off_o + W * nH * Dh;
  c->off_d = c->off_gu + 2 * F * W;
  jpi_status st;
#define ALLOC(ptr, bytes)                                          \
  st = dmalloc(c, (void**)&(ptr), (bytes));                        \
  if (st != JPI_OK) return cleanup_fail(st);
  ALLOC(c->w_layers, c->layer_elems * c->L * es);
  ALLOC(c->w_in, W * A * es);
  ALLOC(c->b_in, W * 4);
  ALLOC(c->w_t0, W * W * es);
  ALLOC(c->w_t1, W * W * es);
  ALLOC(c->b_t0, W * 4);
  ALLOC(c->b_t1, W * 4);
  ALLOC(c->w_mod, (size_t)c->R * W * es);
  ALLOC(c->b_mod, (size_t)c->R * 4);
  ALLOC(c->w_out, A * W * es);
  ALLOC(c->b_out, A * 4);
  const size_t kv_elems = (size_t)c->L * c->Bmax * (size_t)c->Pmax * Dh;
  ALLOC(c->kp, kv_elems * es);
  ALLOC(c->vp, kv_elems * es);
  // room for the action keys after the longest prefix (the single-launch
  // path stores the action rows' V there), rounded to 16-byte rows
  c->Ppad = (c->Pmax + seq_max + 7) / 8 * 8;
  ALLOC(c->vpt, (size_t)c->L * c->Bmax * (size_t)c->Ppad * Dh * es);
  ALLOC(c->d_prefix_len, c->Bmax * 4);
  ALLOC(c->rope_tab, M * (Dh / 2) * sizeof(float2));
  ALLOC(c->committed, M * A * 4);
  ALLOC(c->corr, std::max<size_t>(1, (size_t)c->Bmax * c->Cmax * W) * 4);
  ALLOC(c->x, M * A * 4);
  ALLOC(c->h, M * W * 4);
  ALLOC(c->y, M * W * es);
  ALLOC(c->q, M * nH * Dh * es);
  ALLOC(c->ks, M * Dh * es);
  ALLOC(c->vst, (size_t)c->Bmax * Dh * ((seq_max + 7) / 8 * 8) * es);  // rows padded to 8 elements
  ALLOC(c->o, M * nH * Dh * es);
  ALLOC(c->z, M * F * es);
  ALLOC(c->pflags, (size_t)persist_flag_words() * sizeof(unsigned));
  ALLOC(c->perr, 256);
  if (persist_trace_build()) {  // room for 64 Euler steps of every layer's 8 phases, 3 stamps each
    c->trace_slots = 1 + 3 * 64 * c->L * 8;
    c->trace_grid = persist_max_grid();
    ALLOC(c->ptrace, (size_t)c->trace_grid * c->trace_slots * sizeof(unsigned long long));
  }
  if (g.variant == JPI_VARIANT_ACTION_TIME) {
    const size_t B = c->Bmax, SD = g.state_dim;
    ALLOC(c->w_atm_a, W * W * es);
    ALLOC(c->w_atm_t, W * W * es);
    ALLOC(c->w_atm_out, W * W * es);
    ALLOC(c->w_state, W * SD * es);
    ALLOC(c->b_atm_in, W * 4);
    ALLOC(c->b_atm_out, W * 4);
    ALLOC(c->b_state, W * 4);
    ALLOC(c->norms, (2 * (size_t)c->L + 1) * W * 4);
    ALLOC(c->ones, W * 4);
    ALLOC(c->zeros, W * 4);
    ALLOC(c->state, B * SD * 4);
    ALLOC(c->d_plen1, B * 4);
    ALLOC(c->rope_s, B * (Dh / 2) * sizeof(float2));
    ALLOC(c->hs, B * W * 4);
    ALLOC(c->ys, B * W * es);
    ALLOC(c->ks_s, B * Dh * es);
    ALLOC(c->vst_s, B * Dh * 8 * es);
    ALLOC(c->u2, M * W * es);
    if (launch_fill_f32(c->ones, (int)W, 1.0f, 0) != hipSuccess || launch_fill_f32(c->zeros, (int)W, 0.0f, 0) != hipSuccess ||
        hipDeviceSynchronize() != hipSuccess)
      return cleanup_fail(fail(c, JPI_ERR_HIP, "fill"));
  }
#undef ALLOC
  if (hipMemset(c->perr, 0, 256) != hipSuccess) return cleanup_fail(fail(c, JPI_ERR_HIP, "hipMemset"));
  if (hipHostMalloc((void**)&c->h_prefix_len, c->Bmax * sizeof(int)) != hipSuccess) {
    (void)hipGetLastError();
    c->h_prefix_len = nullptr;
    return cleanup_fail(fail(c, JPI_ERR_OOM, "pinned prefix_len staging"));
  }
  *out = c;
  return JPI_OK;
}

jpi_status jpi_set_weight(jpi_ctx* c, const char* name, const void* data, int64_t n_elems, jpi_dtype dt,
                          int is_device, void* stream) {
  if (!c) return fail(nullptr, JPI_ERR_ARG, "jpi_set_weight: ctx is NULL");
  if (!name || !data) return fail(c, JPI_ERR_ARG, "jpi_set_weight: name or data is NULL");
  int kind, layer;
  if (!parse_name(c, name, &kind, &layer)) return fail(c, JPI_ERR_ARG, std::string("unknown tensor name: ") + name);
  const int64_t want = expected_elems(c, kind);
  if (n_elems != want)
    return fail(c, JPI_ERR_SHAPE, std::string(name) + ": expected " + std::to_string(want) + " elements, got " +
                                       std::to_string(n_elems));
  const bool mat = kind_is_matrix(kind);
  const jpi_dtype want_dt = mat ? c->dt : JPI_F32;
  if (dt != want_dt)
    return fail(c, JPI_ERR_DTYPE, std::string(name) + (mat ? ": matrices must have the context dtype"
                                                           : ": vectors must be JPI_F32"));
  HIPCHK(c, hipSetDevice(c->device));
  hipStream_t s = (hipStream_t)stream;
  const size_t es = mat ? c->esz : 4;
  const size_t bytes = (size_t)n_elems * es;
  const size_t W = c->W, Dh = c->Dh, nH = c->nH;

  // destination base and row map (rows of length `cols`)
  char* base = nullptr;
  int rows = 0, cols = 0;
  std::vector<int> map;
  char* lay = layer >= 0 ? (char*)c->w_layers + (size_t)layer * c->layer_elems * c->esz : nullptr;
  auto identity = [&](char* dst, int r, int cl) {
    base = dst;
    rows = r;
    cols = cl;
  };
  switch (kind) {
    case T_IN_W: identity((char*)c->w_in, c->W, c->A); break;
    case T_IN_B: identity((char*)c->b_in, 1, c->W); break;
    case T_TIME0_W: identity((char*)c->w_t0, c->W, c->W); break;
    case T_TIME0_B: identity((char*)c->b_t0, 1, c->W); break;
    case T_TIME1_W: identity((char*)c->w_t1, c->W, c->W); break;
    case T_TIME1_B: identity((char*)c->b_t1, 1, c->W); break;
    case T_ATTN_MOD_W: identity((char*)c->w_mod + (size_t)(2 * layer) * 3 * W * W * c->esz, 3 * c->W, c->W); break;
    case T_ATTN_MOD_B: identity((char*)(c->b_mod + (size_t)(2 * layer) * 3 * W), 1, 3 * c->W); break;
    case T_MLP_MOD_W:
      identity((char*)c->w_mod + (size_t)(2 * layer + 1) * 3 * W * W * c->esz, 3 * c->W, c->W);
      break;
    case T_MLP_MOD_B: identity((char*)(c->b_mod + (size_t)(2 * layer + 1) * 3 * W), 1, 3 * c->W); break;
    case T_FINAL_MOD_W: identity((char*)c->w_mod + (size_t)(6 * c->L) * W * W * c->esz, 2 * c->W, c->W); break;
    case T_FINAL_MOD_B: identity((char*)(c->b_mod + (size_t)(6 * c->L) * W), 1, 2 * c->W); break;
    case T_OUT_W: identity((char*)c->w_out, c->A, c->W); break;
    case T_OUT_B: identity((char*)c->b_out, 1, c->A); break;
    case T_ATM_IN_B: identity((char*)c->b_atm_in, 1, c->W); break;
    case T_ATM_OUT_W: identity((char*)c->w_atm_out, c->W, c->W); break;
    case T_ATM_OUT_B: identity((char*)c->b_atm_out, 1, c->W); break;
    case T_STATE_W: identity((char*)c->w_state, c->W, c->cfg.state_dim); break;
    case T_STATE_B: identity((char*)c->b_state, 1, c->W); break;
    case T_FINAL_NORM: identity((char*)(c->norms + (size_t)2 * c->L * W), 1, c->W); break;
    case T_ATTN_NORM: identity((char*)(c->norms + (size_t)2 * layer * W), 1, c->W); break;
    case T_MLP_NORM: identity((char*)(c->norms + (size_t)(2 * layer + 1) * W), 1, c->W); break;
    case T_ATM_IN_W: break;  // split below
    case T_O: identity(lay + c->off_o * c->esz, c->W, (int)(nH * Dh)); break;
    case T_DOWN: identity(lay + c->off_d * c->esz, c->W, c->F); break;
    case T_Q:
    case T_K:
    case T_V: {
      base = lay;
      cols = c->W;
      const int r0 = kind == T_Q ? 0 : kind == T_K ? (int)(nH * Dh) : (int)((nH + 1) * Dh);
      rows = kind == T_Q ? (int)(nH * Dh) : (int)Dh;
      map.resize(rows);
      for (int r = 0; r < rows; ++r) map[r] = r0 + (kind == T_V ? r : rope_pack_row(r, (int)Dh));
      break;
    }
    case T_GATE:
    case T_UP: {
      base = lay + c->off_gu * c->esz;
      cols = c->W;
      rows = c->F;
      map.resize(rows);
      for (int f = 0; f < rows; ++f) map[f] = (f / 16) * 32 + (kind == T_UP ? 16 : 0) + (f % 16);
      break;
    }
  }
  if (kind == T_ATM_IN_W) {
    // [W][2W]: the action columns and the time columns go to two [W][W] matrices
    const hipMemcpyKind ck = is_device ? hipMemcpyDeviceToDevice : hipMemcpyHostToDevice;
    HIPCHK(c, hipMemcpy2DAsync(c->w_atm_a, W * es, data, 2 * W * es, W * es, W, ck, s));
    HIPCHK(c, hipMemcpy2DAsync(c->w_atm_t, W * es, (const char*)data + W * es, 2 * W * es, W * es, W, ck, s));
  } else if (map.empty()) {
    HIPCHK(c, hipMemcpyAsync(base, data, bytes, is_device ? hipMemcpyDeviceToDevice : hipMemcpyHostToDevice, s));
  } else {
    void* src = const_cast<void*>(data);
    void* tmp = nullptr;
    int* dmap = nullptr;
    TRY(dmalloc(c, (void**)&dmap, map.size() * sizeof(int)));
    if (!is_device) {
      jpi_status st2 = dmalloc(c, &tmp, bytes);
      if (st2 != JPI_OK) {
        (void)hipFree(dmap);
        return st2;
      }
      HIPCHK(c, hipMemcpyAsync(tmp, data, bytes, hipMemcpyHostToDevice, s));
      src = tmp;
    }
    HIPCHK(c, hipMemcpyAsync(dmap, map.data(), map.size() * sizeof(int), hipMemcpyHostToDevice, s));
    hipLaunchKernelGGL(k_scatter_rows, dim3(rows), dim3(256), 0, s, (const char*)src, base, (const int*)dmap, rows,
                       (int)(cols * es));
    HIPCHK(c, hipGetLastError());
    HIPCHK(c, hipStreamSynchronize(s));
    (void)hipFree(dmap);
    if (tmp) (void)hipFree(tmp);
  }
  HIPCHK(c, hipStreamSynchronize(s));
  c->have[have_index(c, kind, layer)] = 1;
  c->finalized = false;
  c->frag_ready = false;
  drop_graphs(c);
  drop_tables(c);
  return JPI_OK;
}

jpi_status jpi_finalize_weights(jpi_ctx* c, void* stream) {
  (void)stream;
  if (!c) return fail(nullptr, JPI_ERR_ARG, "jpi_finalize_weights: ctx is NULL");
  for (int k = 0; k < T_NKINDS; ++k) {
    if (!kind_in_variant(k, c->cfg.variant)) continue;
    if (kind_is_layer(k)) {
      for (int l = 0; l < c->L; ++l)
        if (!c->have[have_index(c, k, l)])
          return fail(c, JPI_ERR_STATE, "missing tensor layers." + std::to_string(l) + "." + kind_suffix[k]);
    } else if (!c->have[have_index(c, k, -1)]) {
      return fail(c, JPI_ERR_STATE, std::string("missing tensor ") + kind_suffix[k]);
    }
  }
  drop_graphs(c);
  drop_tables(c);
  c->finalized = true;
  c->frag_ready = false;
  return JPI_OK;
}

jpi_status jpi_prefix_buffers(jpi_ctx* c, void** k_out, void** v_out) {
  if (!c || !k_out || !v_out) return fail(c, JPI_ERR_ARG, "jpi_prefix_buffers: NULL argument");
  *k_out = c->kp;
  *v_out = c->vp;
  return JPI_OK;
}

jpi_status jpi_debug_persist_trace(jpi_ctx* c, uint64_t* host_out, int64_t cap, int* n_workgroups, int* n_slots,
                                   double* ticks_per_us) {
  if (!c || !n_workgroups || !n_slots || !ticks_per_us)
    return fail(c, JPI_ERR_ARG, "jpi_debug_persist_trace: NULL argument");
  if (!c->ptrace) return fail(c, JPI_ERR_UNSUPPORTED, "jpi_debug_persist_trace: library built without the trace mode");
  *n_workgroups = c->n_cu;
  *n_slots = c->trace_used;
  int khz = 0;
  HIPCHK(c, hipDeviceGetAttribute(&khz, hipDeviceAttributeWallClockRate, c->device));
  *ticks_per_us = khz / 1000.0;
  const int64_t need = (int64_t)c->n_cu * c->trace_used;
  if (!host_out || cap < need) return JPI_OK;  // sizes only
  HIPCHK(c, hipSetDevice(c->device));
  HIPCHK(c, hipDeviceSynchronize());
  HIPCHK(c, hipMemcpy2D(host_out, (size_t)c->trace_used * 8, c->ptrace, (size_t)c->trace_slots * 8,
                        (size_t)c->trace_used * 8, (size_t)c->n_cu, hipMemcpyDeviceToHost));
  return JPI_OK;
}

jpi_status jpi_debug_prefix_vt(jpi_ctx* c, void** vt_out, int* ld_out) {
  if (!c || !vt_out || !ld_out) return fail(c, JPI_ERR_ARG, "jpi_debug_prefix_vt: NULL argument");
  *vt_out = c->vpt;
  *ld_out = c->Ppad;
  return JPI_OK;
}

jpi_status jpi_bind_prefix(jpi_ctx* c, const void* k, const void* v, const int32_t* prefix_len_host, int batch,
                           int prefix, void* stream) {
  if (!c) return fail(nullptr, JPI_ERR_ARG, "jpi_bind_prefix: ctx is NULL");
  if ((!k || !v) && prefix > 0) return fail(c, JPI_ERR_ARG, "jpi_bind_prefix: k or v is NULL");
  if (batch < 1 || batch > c->Bmax)
    return fail(c, JPI_ERR_SHAPE, "jpi_bind_prefix: batch " + std::to_string(batch) + " outside [1, max_batch=" +
                                       std::to_string(c->Bmax) + "]");
  if (prefix < 0 || prefix > c->Pmax)
    return fail(c, JPI_ERR_SHAPE, "jpi_bind_prefix: prefix " + std::to_string(prefix) + " outside [0, max_prefix=" +
                                       std::to_string(c->Pmax) + "]");
  std::vector<int> lens(batch, prefix);
  if (prefix_len_host)
    for (int b = 0; b < batch; ++b) {
      if (prefix_len_host[b] < 0 || prefix_len_host[b] > prefix)
        return fail(c, JPI_ERR_SHAPE, "jpi_bind_prefix: prefix_len[" + std::to_string(b) + "] = " +
                                           std::to_string(prefix_len_host[b]) + " outside [0, prefix]");
      lens[b] = prefix_len_host[b];
    }
  if (c->cfg.variant == JPI_VARIANT_ACTION_TIME)
    for (int b = 0; b < batch; ++b)
      if (lens[b] >= c->Pmax)
        return fail(c, JPI_ERR_SHAPE, "jpi_bind_prefix: the action-time variant keeps prefix slot prefix_len free "
                                      "for the state token, so every prefix_len must be below max_prefix");
  HIPCHK(c, hipSetDevice(c->device));
  hipStream_t s = (hipStream_t)stream;
  HIPCHK(c, hipStreamSynchronize(s));  // staging buffer and resident KV are free to overwrite
  const size_t es = c->esz, Dh = c->Dh;
  const bool in_place = (k == c->kp && v == c->vp);
  if (in_place && prefix != c->Pmax)
    return fail(c, JPI_ERR_SHAPE, "jpi_bind_prefix: the resident buffers must be bound with prefix == max_prefix");
  if (!in_place && prefix > 0) {
    for (int l = 0; l < c->L; ++l) {
      const size_t dst_off = (size_t)l * c->Bmax * c->Pmax * Dh * es;
      const size_t src_off = (size_t)l * batch * prefix * Dh * es;
      HIPCHK(c, hipMemcpy2DAsync((char*)c->kp + dst_off, c->Pmax * Dh * es, (const char*)k + src_off, prefix * Dh * es,
                                 prefix * Dh * es, batch, hipMemcpyDeviceToDevice, s));
      HIPCHK(c, hipMemcpy2DAsync((char*)c->vp + dst_off, c->Pmax * Dh * es, (const char*)v + src_off, prefix * Dh * es,
                                 prefix * Dh * es, batch, hipMemcpyDeviceToDevice, s));
    }
  }
  // prefix V transposed ([Dh][key]) for the attention kernels' P.V operand
  for (int l = 0; l < c->L && prefix > 0; ++l) {
    const size_t src_off = (size_t)l * c->Bmax * c->Pmax * Dh * es;
    const size_t dst_off = (size_t)l * c->Bmax * c->Ppad * Dh * es;
    HIPCHK(c, launch_transpose(c->dt, (const char*)c->vp + src_off, (char*)c->vpt + dst_off, prefix, (int)Dh,
                               (int64_t)Dh, c->Ppad, (int64_t)c->Pmax * Dh, (int64_t)Dh * c->Ppad, batch, s));
  }
  memcpy(c->h_prefix_len, lens.data(), batch * sizeof(int));
  HIPCHK(c, hipMemcpyAsync(c->d_prefix_len, c->h_prefix_len, batch * sizeof(int), hipMemcpyHostToDevice, s));
  if (c->batch != batch) {  // state rows were bound for another batch
    c->n_fixed = c->n_corr = 0;
    c->state_bound = false;
  }
  HIPCHK(c, launch_rope_table(c->d_prefix_len, c->rope_tab, batch, c->H + c->n_corr, c->Dh, c->cfg.rope_base, s));
  c->rope_rows = c->H + c->n_corr;
  c->batch = batch;
  c->prefix = prefix;
  c->prefix_bound = true;
  return JPI_OK;
}

jpi_status jpi_bind_state(jpi_ctx* c, const float* committed_dev, int n_fixed, const void* corr_tokens, int n_corr,
                          void* stream) {
  if (!c) return fail(nullptr, JPI_ERR_ARG, "jpi_bind_state: ctx is NULL");
  if (!c->prefix_bound) return fail(c, JPI_ERR_STATE, "jpi_bind_state: bind the prefix first (it sets the batch)");
  if (n_fixed < 0 || n_fixed >= c->H)
    return fail(c, JPI_ERR_ARG, "jpi_bind_state: n_fixed must be in [0, horizon)");
  if (n_fixed > 0 && !committed_dev) return fail(c, JPI_ERR_ARG, "jpi_bind_state: committed is NULL");
  if (n_corr < 0 || n_corr > c->Cmax)
    return fail(c, JPI_ERR_ARG, "jpi_bind_state: n_corr must be in [0, max_corr=" + std::to_string(c->Cmax) + "]");
  if (n_corr > 0 && !corr_tokens) return fail(c, JPI_ERR_ARG, "jpi_bind_state: corr_tokens is NULL");
  if (n_corr > 0 && c->cfg.variant != JPI_VARIANT_ADARMS)
    return fail(c, JPI_ERR_UNSUPPORTED, "jpi_bind_state: correction tokens need the adaRMS variant");
  HIPCHK(c, hipSetDevice(c->device));
  hipStream_t s = (hipStream_t)stream;
  if (n_fixed > 0)
    HIPCHK(c, hipMemcpyAsync(c->committed, committed_dev, (size_t)c->batch * n_fixed * c->A * sizeof(float),
                             hipMemcpyDeviceToDevice, s));
  if (n_corr > 0)
    HIPCHK(c, hipMemcpyAsync(c->corr, corr_tokens, (size_t)c->batch * n_corr * c->W * sizeof(float),
                             hipMemcpyDeviceToDevice, s));
  c->n_fixed = n_fixed;
  c->n_corr = n_corr;
  return JPI_OK;
}

}  // extern "C"

namespace {

jpi_status ensure_table(jpi_ctx* c, int n_steps, hipStream_t s, float** out) {
  auto it = c->tables.find(n_steps);
  if (it != c->tables.end()) {
    *out = it->second;
    return JPI_OK;
  }
  const size_t W = c->W;
  const int rows = n_steps + 1;  // t_0 .. t_{N-1}, then t = 0
  float *tab = nullptr, *tmp = nullptr;
  TRY(dmalloc(c, (void**)&tab, (size_t)rows * (c->R + W) * sizeof(float)));  // + [rows][W] for the variant
  jpi_status st = dmalloc(c, (void**)&tmp, (size_t)3 * rows * W * sizeof(float));
  if (st != JPI_OK) {
    (void)hipFree(tab);
    return st;
  }
  float *emb = tmp, *c1 = tmp + rows * W, *cond = tmp + 2 * rows * W;
  hipError_t e = launch_time_embed(emb, rows, n_steps, c->W, s);
  if (c->cfg.variant == JPI_VARIANT_ACTION_TIME) {
    // plain RMSNorm layers: every row (scale, shift, gate) = (w, 0, 1); then, after the
    // table, the time half of the action-time MLP's first layer at each t: W_t e(t) + b_i
    if (e == hipSuccess) e = launch_const_table(tab, c->norms, rows, c->L, c->W, s);
    if (e == hipSuccess)
      e = launch_rowdot(c->dt, emb, c->w_atm_t, c->b_atm_in, tab + (size_t)rows * c->R, rows, c->W, c->W, 0, s);
  } else {
    if (e == hipSuccess) e = launch_rowdot(c->dt, emb, c->w_t0, c->b_t0, c1, rows, c->W, c->W, 1, s);
    if (e == hipSuccess) e = launch_rowdot(c->dt, c1, c->w_t1, c->b_t1, cond, rows, c->W, c->W, 1, s);
    if (e == hipSuccess) e = launch_rowdot(c->dt, cond, c->w_mod, c->b_mod, tab, rows, c->R, c->W, 0, s);
  }
  if (e == hipSuccess) e = hipStreamSynchronize(s);
  (void)hipFree(tmp);
  if (e != hipSuccess) {
    (void)hipFree(tab);
    return fail(c, JPI_ERR_HIP, std::string("modulation table: ") + hipGetErrorString(e));
  }
  c->tables[n_steps] = tab;
  *out = tab;
  return JPI_OK;
}

struct StepGemms {
  int M;
  int s_o, s_d;  // split-K of the O and Down projections (QKV and GateUp are not split)
  bool persist;  // single-launch path
  // action-time variant: split-K of the action-time MLP's two GEMMs, and of the
  // state token's O and Down projections (M = batch rows)
  int s_a = 1, s_so = 1, s_sd = 1;
};

bool use_persist(jpi_ctx* c, int batch) {
  const char* e = getenv("JPI_PERSIST");
  if (e && e[0] == '0') return false;
  const int S = c->H + c->n_corr;  // suffix rows per rollout
  if (!persist_supported(c->dt, batch * S, c->W, c->nH, c->Dh, c->F, S, c->A, c->Pmax)) return false;
  if (c->n_cu > persist_max_grid()) return false;
  if (c->persist_occ < 0) {
    int occ = 0;
    if (persist_occupancy(c->Dh, &occ) != hipSuccess) {
      (void)hipGetLastError();
      occ = 0;
    }
    c->persist_occ = occ;
  }
  return c->persist_occ >= 1;  // one workgroup per CU, grid = CU count: all co-resident
}

StepGemms plan_gemms(jpi_ctx* c, int batch) {
  StepGemms p;
  p.M = batch * (c->H + c->n_corr);
  p.persist = use_persist(c, batch);
  if (p.persist) {
    p.s_o = persist_pick_split(c->W / 32, c->nH * c->Dh, c->n_cu);
    p.s_d = persist_pick_split(c->W / 32, c->F, c->n_cu);
  } else {
    p.s_o = gemm_pick_splitk(c->dt, p.M, c->W, c->nH * c->Dh, c->n_cu);
    p.s_d = gemm_pick_splitk(c->dt, p.M, c->W, c->F, c->n_cu);
  }
  if (c->cfg.variant == JPI_VARIANT_ACTION_TIME) {
    p.s_a = gemm_pick_splitk(c->dt, p.M, c->W, c->W, c->n_cu);
    p.s_so = gemm_pick_splitk(c->dt, batch, c->W, c->nH * c->Dh, c->n_cu);
    p.s_sd = gemm_pick_splitk(c->dt, batch, c->W, c->F, c->n_cu);
  }
  return p;
}

jpi_status ensure_scratch(jpi_ctx* c, int batch, int prefix) {
  const StepGemms p = plan_gemms(c, batch);
  const size_t need = std::max((size_t)std::max(std::max(p.s_o, p.s_d), p.s_a) * p.M * c->W,
                               (size_t)std::max(p.s_so, p.s_sd) * batch * c->W);
  bool changed = false;
  if (need > c->partial_cap) {
    if (c->partial) (void)hipFree(c->partial);
    c->partial = nullptr;
    c->partial_cap = 0;
    TRY(dmalloc(c, (void**)&c->partial, need * sizeof(float)));
    c->partial_cap = need;
    changed = true;
  }
  const int S = c->H + c->n_corr;
  const size_t nch = p.persist ? (size_t)persist_chunks(prefix, S) : (size_t)attn_n_chunks(c->dt, prefix, S);
  const size_t attn = (size_t)batch * c->nH * nch * S * (c->Dh + 2);
  if (attn > c->attn_cap) {
    if (c->opart) (void)hipFree(c->opart);
    c->opart = nullptr;
    c->attn_cap = 0;
    TRY(dmalloc(c, (void**)&c->opart, attn * sizeof(float)));
    c->attn_cap = attn;
    changed = true;
  }
  if (p.persist && !c->ysw) {
    // fragment-ordered activations, 64 padded rows (the padding stays zero)
    const size_t es = c->esz, bq = std::max(1, 64 / c->H);
    TRY(dmalloc(c, &c->ysw, (size_t)64 * c->W * es));
    TRY(dmalloc(c, &c->osw, (size_t)64 * c->nH * c->Dh * es));
    TRY(dmalloc(c, &c->zsw, (size_t)64 * c->F * es));
    TRY(dmalloc(c, &c->qsw, bq * c->nH * 64 * c->Dh * es));
    HIPCHK(c, hipMemset(c->ysw, 0, (size_t)64 * c->W * es));
    HIPCHK(c, hipMemset(c->osw, 0, (size_t)64 * c->nH * c->Dh * es));
    HIPCHK(c, hipMemset(c->zsw, 0, (size_t)64 * c->F * es));
    HIPCHK(c, hipMemset(c->qsw, 0, bq * c->nH * 64 * c->Dh * es));
    HIPCHK(c, hipDeviceSynchronize());
    changed = true;
  }
  if (p.persist && !c->w_frag) {
    TRY(dmalloc(c, &c->w_frag, c->layer_elems * c->L * c->esz));
    c->frag_ready = false;
    changed = true;
  }
  if (changed) drop_graphs(c);  // captured graphs point at the old scratch
  return JPI_OK;
}

// Fragment-ordered copy of the layer weights for the single-launch path
// (enqueued on s before the kernel that reads it; redone after weight changes).
jpi_status ensure_frag(jpi_ctx* c, hipStream_t s) {
  if (c->frag_ready) return JPI_OK;
  const int W = c->W, HD = c->nH * c->Dh, F = c->F;
  const size_t es = c->esz;
  for (int l = 0; l < c->L; ++l) {
    const char* src = (const char*)c->w_layers + (size_t)l * c->layer_elems * es;
    char* dst = (char*)c->w_frag + (size_t)l * c->layer_elems * es;
    HIPCHK(c, launch_frag_order(src, dst, (c->nH + 2) * c->Dh, W, s));
    HIPCHK(c, launch_frag_order(src + c->off_o * es, dst + c->off_o * es, W, HD, s));
    HIPCHK(c, launch_frag_order(src + c->off_gu * es, dst + c->off_gu * es, 2 * F, W, s));
    HIPCHK(c, launch_frag_order(src + c->off_d * es, dst + c->off_d * es, W, F, s));
  }
  c->frag_ready = true;
  return JPI_OK;
}

// Enqueue the whole N-step loop on stream s (eagerly or under capture).
hipError_t enqueue_steps(jpi_ctx* c, const float* table, int n_steps, hipStream_t s) {
  const int batch = c->batch, prefix = c->prefix, H = c->H, C = c->n_corr;
  const int S = C + H;  // suffix rows per rollout: correction tokens, then action tokens
  const StepGemms p = plan_gemms(c, batch);
  const int M = p.M, W = c->W, Dh = c->Dh, nH = c->nH, F = c->F, L = c->L;
  const size_t es = c->esz;
  // action-time variant: the state token sits in prefix slot prefix_len, so the
  // action rows see prefix_len + 1 keys there and start at position prefix_len + 1
  const bool at = c->cfg.variant == JPI_VARIANT_ACTION_TIME;
  const int* plen_act = at ? c->d_plen1 : c->d_prefix_len;
  const int P_act = at ? prefix + 1 : prefix;
  const int nch = attn_n_chunks(c->dt, P_act, S);
  const float eps = c->cfg.rms_eps;
  const float dt_step = -1.0f / (float)n_steps;
  hipError_t e;
#define ENQ(x)                      \
  do {                              \
    e = (x);                        \
    if (e != hipSuccess) return e;  \
  } while (0)
  // optional event pairs around one kernel kind (measurement support)
  const int need_ev = c->timed_kind >= 0 ? 2 * n_steps * L : 0;
  while ((int)c->ev.size() < need_ev) {
    hipEvent_t ev;
    ENQ(hipEventCreate(&ev));
    c->ev.push_back(ev);
  }
  c->ev_used = 0;
  // events bracketing the timed kernel kind, taken on the dispatch itself
  auto timing = [&](int kind, hipEvent_t* start, hipEvent_t* stop) {
    *start = *stop = nullptr;
    if (kind != c->timed_kind) return;
    *start = c->ev[c->ev_used];
    *stop = c->ev[c->ev_used + 1];
    c->ev_used += 2;
  };
  if (at) {
    // the state token: W_s s + b_s, then every layer over it alone (it sees the prefix
    // and itself); each layer's key and value go into prefix slot prefix_len
    ENQ(launch_plus_one(c->d_prefix_len, c->d_plen1, batch, s));
    ENQ(launch_rope_table(c->d_plen1, c->rope_tab, batch, H, Dh, c->cfg.rope_base, s));
    ENQ(launch_rope_table(c->d_prefix_len, c->rope_s, batch, 1, Dh, c->cfg.rope_base, s));
    ENQ(launch_rowdot(c->dt, c->state, c->w_state, c->b_state, c->hs, batch, W, c->cfg.state_dim, 0, s));
    ENQ(launch_norm_rows(c->hs, c->norms, c->ys, batch, W, eps, s, c->dt == JPI_F32));
    BlockLaunch b{};
    b.B = batch;
    b.H = 1;
    b.W = W;
    b.nH = nH;
    b.Dh = Dh;
    b.F = F;
    b.n_cu = c->n_cu;
    b.off_o = c->off_o;
    b.off_gu = c->off_gu;
    b.off_d = c->off_d;
    b.h = c->hs;
    b.y = c->ys;
    b.q = c->q;
    b.o = c->o;
    b.z = c->z;
    b.partial = c->partial;
    b.s_o = p.s_so;
    b.s_d = p.s_sd;
    b.opart = c->opart;
    b.ks = c->ks_s;
    b.ks_bstride = 0;
    b.vst = c->vst_s;
    b.vst_ld = 8;
    b.kp_bstride = (int64_t)c->Pmax * Dh;
    b.vpt_bstride = (int64_t)c->Ppad * Dh;
    b.vpt_dstride = c->Ppad;
    b.prefix_len = c->d_prefix_len;
    b.P = prefix;
    b.rope = c->rope_s;
    b.ones = c->ones;
    b.zeros = c->zeros;
    b.eps = eps;
    b.f32 = c->dt == JPI_F32;
    for (int l = 0; l < L; ++l) {
      b.w = (const char*)c->w_layers + (size_t)l * c->layer_elems * es;
      char* kl = (char*)c->kp + (size_t)l * c->Bmax * c->Pmax * Dh * es;
      char* vl = (char*)c->vpt + (size_t)l * c->Bmax * c->Ppad * Dh * es;
      b.kp = kl;
      b.vpt = vl;
      b.mlp_norm = c->norms + (size_t)(2 * l + 1) * W;
      b.next_norm = c->norms + (size_t)(l + 1 < L ? 2 * (l + 1) : 2 * L) * W;
      ENQ(enqueue_block(b, s));
      ENQ(launch_put_state_kv(c->dt, c->ks_s, c->vst_s, 8, kl, b.kp_bstride, vl, b.vpt_bstride, b.vpt_dstride,
                              c->d_prefix_len, batch, Dh, s));
    }
  }
  // action-time variant, step k: h = W_o swish(W_i [W_a x + b_a ; e(t_k)] + b_i) + b_o (and its first norm)
  const float* ctab = table + (size_t)(n_steps + 1) * c->R;  // W_t e(t_k) + b_i rows after the table
#define ENQ_L(x)                    \
  do {                              \
    hipError_t e_ = (x);            \
    if (e_ != hipSuccess) return e_; \
  } while (0)
  auto action_time_inproj = [&](int k) -> hipError_t {
    const float* tk = table + (size_t)k * c->R;
    // h = W_o swish(W_i [W_a x + b_a ; e(t_k)] + b_i) + b_o, then the first norm
    ENQ_L(launch_action_embed(c->dt, c->x, c->w_in, c->b_in, c->y, M, W, c->A, s));
    GemmLaunch g{};
    g.M = M;
    g.A = c->y;
    g.W = c->w_atm_a;
    g.N = W;
    g.K = W;
    g.splitk = p.s_a;
    g.epi = EPI_STORE_F32;
    g.ep.out_f32 = c->partial;
    g.n_cu = c->n_cu;
    ENQ_L(launch_gemm(c->dt, g, s));
    ENQ_L(launch_swish_slices(c->dt, c->partial, p.s_a, M, ctab + (size_t)k * W, c->u2, W, s));
    g.A = c->u2;
    g.W = c->w_atm_out;
    ENQ_L(launch_gemm(c->dt, g, s));
    ENQ_L(launch_bcast_rows(c->b_atm_out, c->h, M, 1, W, s));
    RowLaunch r{};
    r.part = c->partial;
    r.S = p.s_a;
    r.M = M;
    r.W = W;
    r.h = c->h;
    r.gate = tk + 2 * W;  // ones in the plain-norm table
    r.scale = tk;
    r.shift = tk + W;
    r.y = c->y;
    r.eps = eps;
    r.horizon = H;
    ENQ_L(launch_resid_norm(c->dt, r, false, s));
    return hipSuccess;
  };
#undef ENQ_L
  const int n_t0 = c->committed_t0 && !at ? c->n_fixed : 0;
  if (p.persist) {
    PersistArgs pa{};
    pa.L = L;
    pa.W = W;
    pa.nH = nH;
    pa.Dh = Dh;
    pa.F = F;
    pa.A = c->A;
    pa.H = S;
    pa.n_corr = C;
    pa.corr = c->corr;
    pa.B = batch;
    pa.M = M;
    pa.C = persist_chunks(P_act, S);
    pa.n_steps = n_steps;
    pa.n_fixed = c->n_fixed;
    pa.n_t0 = c->committed_t0 ? c->n_fixed : 0;
    pa.s_o = p.s_o;
    pa.s_d = p.s_d;
    pa.R = c->R;
    pa.eps = eps;
    pa.dt = dt_step;
    pa.w_layers = c->w_layers;
    pa.w_frag = c->w_frag;
    pa.layer_elems = (int64_t)c->layer_elems;
    pa.off_o = (int64_t)c->off_o;
    pa.off_gu = (int64_t)c->off_gu;
    pa.off_d = (int64_t)c->off_d;
    pa.w_in = c->w_in;
    pa.b_in = c->b_in;
    pa.w_out = c->w_out;
    pa.b_out = c->b_out;
    pa.table = table;
    pa.kp = c->kp;
    pa.vpt = c->vpt;
    pa.kp_lstride = (int64_t)c->Bmax * c->Pmax * Dh;
    pa.kp_bstride = (int64_t)c->Pmax * Dh;
    pa.vpt_lstride = (int64_t)c->Bmax * c->Ppad * Dh;
    pa.vpt_bstride = (int64_t)c->Ppad * Dh;
    pa.vpt_dstride = c->Ppad;
    pa.prefix_len = plen_act;
    pa.rope = c->rope_tab;
    pa.x = c->x;
    pa.h = c->h;
    pa.y = c->ysw;
    pa.q = c->qsw;
    pa.ks = c->ks;
    pa.vst = c->vst;
    pa.opart = c->opart;
    pa.ml = c->opart + (size_t)batch * nH * pa.C * S * Dh;
    pa.o = c->osw;
    pa.part = c->partial;
    pa.z = c->zsw;
    pa.flags = c->pflags;
    pa.err = c->perr;
    pa.spin_limit = c->persist_spin ? c->persist_spin : persist_default_spin();
    pa.trace = c->ptrace;
    pa.trace_slots = c->trace_slots;
    c->trace_used = std::min(c->trace_slots, 1 + 3 * n_steps * L * 8);
    if (!at) {
      timing(JPI_KERNEL_PERSISTENT, &pa.ev_start, &pa.ev_stop);
      ENQ(launch_persist(pa, c->n_cu, s));
      return hipSuccess;
    }
    // action-time variant: per step the action-time MLP (multi-kernel), then one
    // single-launch step that starts its rows from that h
    pa.n_steps = 1;
    pa.n_t0 = 0;
    pa.h_in = c->h;
    for (int k = 0; k < n_steps; ++k) {
      ENQ(action_time_inproj(k));
      pa.table = table + (size_t)k * c->R;
      timing(JPI_KERNEL_PERSISTENT, &pa.ev_start, &pa.ev_stop);
      ENQ(launch_persist(pa, c->n_cu, s));
    }
    return hipSuccess;
  }
  for (int k = 0; k < n_steps; ++k) {
    const float* tk = table + (size_t)k * c->R;
    const float* fm = tk + (size_t)(6 * L) * W;
    const int64_t t0_delta = (int64_t)(n_steps - k) * c->R;  // to the t = 0 row
    if (at) {
      ENQ(action_time_inproj(k));
    } else {
      ENQ(launch_inproj_norm(c->dt, c->x, c->w_in, c->b_in, c->h, tk, tk + W, c->y, M, W, c->A, eps, c->corr, C, H,
                             n_t0, t0_delta, s));
    }
    for (int l = 0; l < L; ++l) {
      const char* lay = (const char*)c->w_layers + (size_t)l * c->layer_elems * es;
      const float* am = tk + (size_t)(2 * l) * 3 * W;
      const float* mm = tk + (size_t)(2 * l + 1) * 3 * W;
      // QKV + RoPE (y holds adaRMSNorm(h) with this layer's attention modulation)
      GemmLaunch g{};
      g.M = M;
      g.A = c->y;
      g.W = lay;
      g.N = (nH + 2) * Dh;
      g.K = W;
      g.splitk = 1;
      g.epi = EPI_QKV;
      g.ep.q = c->q;
      g.ep.ks = c->ks;
      g.ep.vst = c->vst;
      g.ep.vst_ld = (S + 7) / 8 * 8;
      g.ep.rope = c->rope_tab;
      g.ep.n_heads = nH;
      g.ep.head_dim = Dh;
      g.ep.horizon = S;
      timing(JPI_KERNEL_QKV, &g.ev_start, &g.ev_stop);
      g.n_cu = c->n_cu;
      ENQ(launch_gemm(c->dt, g, s));
      // attention
      AttnLaunch a{};
      a.q = c->q;
      a.ks = c->ks;
      a.vst = c->vst;
      a.vst_ld = (S + 7) / 8 * 8;
      a.kp = (const char*)c->kp + (size_t)l * c->Bmax * c->Pmax * Dh * es;
      a.vpt = (const char*)c->vpt + (size_t)l * c->Bmax * c->Ppad * Dh * es;
      a.kp_bstride = (int64_t)c->Pmax * Dh;
      a.vpt_bstride = (int64_t)c->Ppad * Dh;
      a.vpt_dstride = c->Ppad;
      a.prefix_len = plen_act;
      a.B = batch;
      a.nH = nH;
      a.H = S;
      a.P = P_act;
      a.Dh = Dh;
      a.opart = c->opart;
      a.mpart = c->opart + (size_t)batch * nH * nch * S * Dh;
      a.lpart = a.mpart + (size_t)batch * nH * nch * S;
      a.out = c->o;
      a.out_f32 = 0;
      a.n_cu = c->n_cu;
      timing(JPI_KERNEL_ATTENTION, &a.ev_start, &a.ev_stop);
      ENQ(launch_attention(c->dt, a, s));
      // O projection (split-K slices) -> gated residual + MLP adaRMSNorm
      g = GemmLaunch{};
      g.M = M;
      g.A = c->o;
      g.W = lay + c->off_o * es;
      g.N = W;
      g.K = nH * Dh;
      g.splitk = p.s_o;
      g.epi = EPI_STORE_F32;
      g.ep.out_f32 = c->partial;
      timing(JPI_KERNEL_OPROJ, &g.ev_start, &g.ev_stop);
      g.n_cu = c->n_cu;
      ENQ(launch_gemm(c->dt, g, s));
      RowLaunch r{};
      r.part = c->partial;
      r.S = p.s_o;
      r.M = M;
      r.W = W;
      r.h = c->h;
      r.gate = am + 2 * W;
      r.scale = mm;
      r.shift = mm + W;
      r.y = c->y;
      r.eps = eps;
      r.horizon = H;
      r.n_lead = C;
      r.n_t0 = n_t0;
      r.t0_delta = t0_delta;
      ENQ(launch_resid_norm(c->dt, r, false, s));
      // GateUp + GeGLU
      g = GemmLaunch{};
      g.M = M;
      g.A = c->y;
      g.W = lay + c->off_gu * es;
      g.N = 2 * F;
      g.K = W;
      g.splitk = 1;
      g.epi = EPI_GEGLU;
      g.ep.z = c->z;
      g.ep.mlp_dim = F;
      timing(JPI_KERNEL_GATEUP, &g.ev_start, &g.ev_stop);
      g.n_cu = c->n_cu;
      ENQ(launch_gemm(c->dt, g, s));
      // Down (split-K slices) -> gated residual + next norm (or final head + Euler)
      g = GemmLaunch{};
      g.M = M;
      g.A = c->z;
      g.W = lay + c->off_d * es;
      g.N = W;
      g.K = F;
      g.splitk = p.s_d;
      g.epi = EPI_STORE_F32;
      g.ep.out_f32 = c->partial;
      timing(JPI_KERNEL_DOWN, &g.ev_start, &g.ev_stop);
      g.n_cu = c->n_cu;
      ENQ(launch_gemm(c->dt, g, s));
      r.S = p.s_d;
      r.gate = mm + 2 * W;
      const bool last = l == L - 1;
      if (!last) {
        const float* an = tk + (size_t)(2 * (l + 1)) * 3 * W;
        r.scale = an;
        r.shift = an + W;
      } else {
        r.scale = fm;
        r.shift = fm + W;
        r.w_out = c->w_out;
        r.b_out = c->b_out;
        r.x = c->x;
        r.A = c->A;
        r.n_fixed = c->n_fixed;
        r.dt = dt_step;
      }
      ENQ(launch_resid_norm(c->dt, r, last, s));
    }
  }
#undef ENQ
  return hipSuccess;
}

bool eager_mode() {
  const char* e = getenv("JPI_EAGER");
  return e && e[0] == '1';
}

}  // namespace

extern "C" {

jpi_status jpi_denoise(jpi_ctx* c, const float* noise_dev, int n_steps, float* actions_dev, void* stream) {
  if (!c) return fail(nullptr, JPI_ERR_ARG, "jpi_denoise: ctx is NULL");
  if (!noise_dev || !actions_dev) return fail(c, JPI_ERR_ARG, "jpi_denoise: noise or actions is NULL");
  if (n_steps < 1) return fail(c, JPI_ERR_ARG, "jpi_denoise: n_steps must be >= 1");
  if (!c->finalized) return fail(c, JPI_ERR_STATE, "jpi_denoise: weights are not finalized");
  if (!c->prefix_bound) return fail(c, JPI_ERR_STATE, "jpi_denoise: no prefix bound");
  if (c->cfg.variant == JPI_VARIANT_ACTION_TIME && !c->state_bound)
    return fail(c, JPI_ERR_STATE, "jpi_denoise: the action-time variant needs jpi_bind_robot_state");
  HIPCHK(c, hipSetDevice(c->device));
  hipStream_t s = (hipStream_t)stream;
  float* table = nullptr;
  TRY(ensure_table(c, n_steps, s, &table));
  // the action-time variant's action rows also see the state token's prefix slot
  TRY(ensure_scratch(c, c->batch, c->prefix + (c->cfg.variant == JPI_VARIANT_ACTION_TIME ? 1 : 0)));
  if (use_persist(c, c->batch)) TRY(ensure_frag(c, s));
  HIPCHK(c, launch_init_x(noise_dev, c->committed, c->x, c->batch, c->H, c->A, c->n_fixed, s));
  if (c->rope_rows != c->H + c->n_corr) {  // the suffix length changed since the table was built
    HIPCHK(c, launch_rope_table(c->d_prefix_len, c->rope_tab, c->batch, c->H + c->n_corr, c->Dh, c->cfg.rope_base, s));
    c->rope_rows = c->H + c->n_corr;
  }
  if (eager_mode() || c->timed_kind >= 0) {
    HIPCHK(c, enqueue_steps(c, table, n_steps, s));
  } else {
    const GraphKey key{c->batch, c->prefix, n_steps, c->n_fixed, c->n_corr, c->committed_t0, use_persist(c, c->batch)};
    auto it = c->graphs.find(key);
    if (it == c->graphs.end()) {
      hipGraph_t graph = nullptr;
      HIPCHK(c, hipStreamBeginCapture(c->cap_stream, hipStreamCaptureModeThreadLocal));
      hipError_t e = enqueue_steps(c, table, n_steps, c->cap_stream);
      hipError_t e2 = hipStreamEndCapture(c->cap_stream, &graph);
      if (e != hipSuccess || e2 != hipSuccess) {
        if (graph) (void)hipGraphDestroy(graph);
        (void)hipGetLastError();
        return fail(c, JPI_ERR_HIP, std::string("graph capture: ") + hipGetErrorString(e != hipSuccess ? e : e2));
      }
      hipGraphExec_t exec = nullptr;
      hipError_t e3 = hipGraphInstantiate(&exec, graph, nullptr, nullptr, 0);
      (void)hipGraphDestroy(graph);
      if (e3 != hipSuccess) return fail(c, JPI_ERR_HIP, std::string("graph instantiate: ") + hipGetErrorString(e3));
      it = c->graphs.emplace(key, exec).first;
    }
    HIPCHK(c, hipGraphLaunch(it->second, s));
  }
  HIPCHK(c, hipMemcpyAsync(actions_dev, c->x, (size_t)c->batch * c->H * c->A * sizeof(float),
                           hipMemcpyDeviceToDevice, s));
  return JPI_OK;
}

jpi_status jpi_bind_robot_state(jpi_ctx* c, const float* state_dev, void* stream) {
  if (!c) return fail(nullptr, JPI_ERR_ARG, "jpi_bind_robot_state: ctx is NULL");
  if (c->cfg.variant != JPI_VARIANT_ACTION_TIME)
    return fail(c, JPI_ERR_UNSUPPORTED, "jpi_bind_robot_state: only the action-time variant takes a robot state");
  if (!state_dev) return fail(c, JPI_ERR_ARG, "jpi_bind_robot_state: state is NULL");
  if (!c->prefix_bound) return fail(c, JPI_ERR_STATE, "jpi_bind_robot_state: bind the prefix first (it sets the batch)");
  HIPCHK(c, hipSetDevice(c->device));
  HIPCHK(c, hipMemcpyAsync(c->state, state_dev, (size_t)c->batch * c->cfg.state_dim * sizeof(float),
                           hipMemcpyDeviceToDevice, (hipStream_t)stream));
  c->state_bound = true;
  return JPI_OK;
}

jpi_status jpi_set_committed_t0(jpi_ctx* c, int enable) {
  if (!c) return fail(nullptr, JPI_ERR_ARG, "jpi_set_committed_t0: ctx is NULL");
  c->committed_t0 = enable != 0;
  return JPI_OK;
}

jpi_status jpi_sync(jpi_ctx* c, void* stream) {
  if (!c) return fail(nullptr, JPI_ERR_ARG, "jpi_sync: ctx is NULL");
  HIPCHK(c, hipSetDevice(c->device));
  HIPCHK(c, hipStreamSynchronize((hipStream_t)stream));
  HIPCHK(c, hipGetLastError());
  unsigned perr = 0;
  HIPCHK(c, hipMemcpy(&perr, c->perr, sizeof(perr), hipMemcpyDeviceToHost));
  if (perr != 0) {
    HIPCHK(c, hipMemset(c->perr, 0, sizeof(perr)));
    return fail(c, JPI_ERR_HIP, "single-launch denoise: a wait for producer workgroups timed out; the output is invalid");
  }
  return JPI_OK;
}

jpi_status jpi_debug_set_spin_limit(jpi_ctx* c, uint32_t polls) {
  if (!c) return fail(nullptr, JPI_ERR_ARG, "jpi_debug_set_spin_limit: ctx is NULL");
  HIPCHK(c, hipSetDevice(c->device));
  HIPCHK(c, hipDeviceSynchronize());
  c->persist_spin = polls;
  drop_graphs(c);  // the bound is an argument of the captured launch
  return JPI_OK;
}

jpi_status jpi_debug_time_kernel(jpi_ctx* c, int kind) {
  if (!c) return fail(nullptr, JPI_ERR_ARG, "jpi_debug_time_kernel: ctx is NULL");
  if (kind < JPI_KERNEL_NONE || kind > JPI_KERNEL_PERSISTENT)
    return fail(c, JPI_ERR_ARG, "jpi_debug_time_kernel: bad kind");
  HIPCHK(c, hipSetDevice(c->device));
  HIPCHK(c, hipDeviceSynchronize());
  drop_graphs(c);
  c->timed_kind = kind;
  c->ev_used = 0;
  return JPI_OK;
}

jpi_status jpi_debug_kernel_time(jpi_ctx* c, float* total_ms, int* launches) {
  if (!c || !total_ms || !launches) return fail(c, JPI_ERR_ARG, "jpi_debug_kernel_time: NULL argument");
  if (c->timed_kind < 0) return fail(c, JPI_ERR_STATE, "jpi_debug_kernel_time: timing is off");
  HIPCHK(c, hipSetDevice(c->device));
  float tot = 0.f;
  for (int i = 0; i + 1 < c->ev_used; i += 2) {
    float ms = 0.f;
    HIPCHK(c, hipEventElapsedTime(&ms, c->ev[i], c->ev[i + 1]));
    tot += ms;
  }
  *total_ms = tot;
  *launches = c->ev_used / 2;
  return JPI_OK;
}

jpi_status jpi_debug_gemm(const void* A, const void* Wt, float* C, int M, int N, int K, jpi_dtype dt, int splitk,
                          void* stream) {
  if (!A || !Wt || !C) return fail(nullptr, JPI_ERR_ARG, "jpi_debug_gemm: NULL pointer");
  if (M < 1 || N < 1 || K < 1 || splitk < 1) return fail(nullptr, JPI_ERR_ARG, "jpi_debug_gemm: sizes must be >= 1");
  if (dt != JPI_F32 && dt != JPI_BF16) return fail(nullptr, JPI_ERR_ARG, "jpi_debug_gemm: bad dtype");
  const int q = gemm_k_quantum(dt, M);
  if (K % (q * splitk) != 0)
    return fail(nullptr, JPI_ERR_ARG, "jpi_debug_gemm: K must be a multiple of " + std::to_string(q) + "*splitk");
  hipStream_t s = (hipStream_t)stream;
  GemmLaunch g{};
  g.A = A;
  g.W = Wt;
  g.M = M;
  g.N = N;
  g.K = K;
  g.splitk = splitk;
  g.epi = EPI_STORE_F32;
  g.ep.out_f32 = C;
  float* part = nullptr;
  hipError_t e = hipSuccess;
  if (splitk > 1) {
    e = hipMalloc((void**)&part, (size_t)splitk * M * N * sizeof(float));
    g.ep.out_f32 = part;
  }
  if (e == hipSuccess) e = launch_gemm(dt, g, s);
  if (e == hipSuccess && splitk > 1) e = launch_sum_slices(part, C, splitk, (size_t)M * N, s);
  if (e == hipSuccess) e = hipStreamSynchronize(s);
  if (part) (void)hipFree(part);
  if (e != hipSuccess) {
    (void)hipGetLastError();
    return fail(nullptr, e == hipErrorOutOfMemory ? JPI_ERR_OOM : JPI_ERR_HIP,
                std::string("jpi_debug_gemm: ") + hipGetErrorString(e));
  }
  return JPI_OK;
}

jpi_status jpi_debug_attention(const void* q, const void* ks, const void* vs, const void* kp, const void* vp,
                               const int32_t* prefix_len_host, int batch, int n_heads, int H, int P, int Dh,
                               jpi_dtype dt, float* out, void* stream) {
  if (!q || !ks || !vs || !out || !prefix_len_host || ((!kp || !vp) && P > 0))
    return fail(nullptr, JPI_ERR_ARG, "jpi_debug_attention: NULL pointer");
  if (batch < 1 || n_heads < 1 || H < 1 || P < 0 || (Dh != 64 && Dh != 128 && Dh != 256))
    return fail(nullptr, JPI_ERR_ARG, "jpi_debug_attention: bad sizes");
  if (dt != JPI_F32 && dt != JPI_BF16) return fail(nullptr, JPI_ERR_ARG, "jpi_debug_attention: bad dtype");
  if (P > attn_max_prefix(dt, H)) return fail(nullptr, JPI_ERR_ARG, "jpi_debug_attention: prefix too long");
  for (int b = 0; b < batch; ++b)
    if (prefix_len_host[b] < 0 || prefix_len_host[b] > P)
      return fail(nullptr, JPI_ERR_ARG, "jpi_debug_attention: prefix_len out of range");
  hipStream_t s = (hipStream_t)stream;
  const size_t es = dt == JPI_BF16 ? 2 : 4;
  const int nch = attn_n_chunks(dt, P, H);
  const int Ppad = (P + 7) / 8 * 8 > 0 ? (P + 7) / 8 * 8 : 8;
  int* dlen = nullptr;
  float* part = nullptr;
  void *vpt = nullptr, *vst = nullptr;
  const size_t np = (size_t)batch * n_heads * nch * H * (Dh + 2);
  hipError_t ea = hipMalloc((void**)&dlen, batch * sizeof(int));
  if (ea == hipSuccess) ea = hipMalloc((void**)&part, np * sizeof(float));
  if (ea == hipSuccess) ea = hipMalloc(&vpt, (size_t)batch * Dh * Ppad * es);
  const int Hs = (H + 7) / 8 * 8;  // V^T rows padded to 8 elements
  if (ea == hipSuccess) ea = hipMalloc(&vst, (size_t)batch * Dh * Hs * es);
  auto cleanup = [&]() {
    if (dlen) (void)hipFree(dlen);
    if (part) (void)hipFree(part);
    if (vpt) (void)hipFree(vpt);
    if (vst) (void)hipFree(vst);
  };
  if (ea != hipSuccess) {
    (void)hipGetLastError();
    cleanup();
    return fail(nullptr, ea == hipErrorOutOfMemory ? JPI_ERR_OOM : JPI_ERR_HIP,
                std::string("jpi_debug_attention: scratch: ") + hipGetErrorString(ea));
  }
  AttnLaunch a{};
  a.q = q;
  a.ks = ks;
  a.vst = vst;
  a.vst_ld = Hs;
  a.kp = kp ? kp : ks;
  a.vpt = vpt;
  a.kp_bstride = (int64_t)P * Dh;
  a.vpt_bstride = (int64_t)Ppad * Dh;
  a.vpt_dstride = Ppad;
  a.prefix_len = dlen;
  a.B = batch;
  a.nH = n_heads;
  a.H = H;
  a.P = P;
  a.Dh = Dh;
  a.opart = part;
  a.mpart = part + (size_t)batch * n_heads * nch * H * Dh;
  a.lpart = a.mpart + (size_t)batch * n_heads * nch * H;
  a.out = out;
  a.out_f32 = 1;
  {
    int dev = 0, ncu = 0;
    if (hipGetDevice(&dev) == hipSuccess &&
        hipDeviceGetAttribute(&ncu, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess)
      a.n_cu = ncu;
  }
  hipError_t e = hipMemcpyAsync(dlen, prefix_len_host, batch * sizeof(int), hipMemcpyHostToDevice, s);
  if (e == hipSuccess && P > 0)
    e = launch_transpose(dt, vp, vpt, P, Dh, Dh, Ppad, (int64_t)P * Dh, (int64_t)Dh * Ppad, batch, s);
  if (e == hipSuccess) e = launch_transpose(dt, vs, vst, H, Dh, Dh, Hs, (int64_t)H * Dh, (int64_t)Dh * Hs, batch, s);
  if (e == hipSuccess) e = launch_attention(dt, a, s);
  if (e == hipSuccess) e = hipStreamSynchronize(s);
  cleanup();
  if (e != hipSuccess) return fail(nullptr, JPI_ERR_HIP, std::string("jpi_debug_attention: ") + hipGetErrorString(e));
  return JPI_OK;
}

}  // extern "C"

// ---------------------------------------------------------------------------
// resident prefix buffers for an in-place producer (the VLM prefill)
// ---------------------------------------------------------------------------
jpi_status jpi::ae_prefix_target(jpi_ctx* c, int L, int Dh, jpi_dtype dt, int batch, int prefix,
                                 AePrefixTarget* t, const char** why) {
  *why = nullptr;
  if (!c || !t) {
    *why = "action-expert context is NULL";
    return JPI_ERR_ARG;
  }
  if (c->L != L || c->Dh != Dh || c->dt != dt) {
    *why = "the action expert's layer count, head_dim or dtype differs from the producer's";
    return JPI_ERR_SHAPE;
  }
  if (batch < 1 || batch > c->Bmax || prefix < 1 || prefix > c->Pmax) {
    *why = "batch or prefix exceeds the action expert's max_batch / max_prefix";
    return JPI_ERR_SHAPE;
  }
  if (c->cfg.variant == JPI_VARIANT_ACTION_TIME && prefix >= c->Pmax) {
    *why = "the action-time variant keeps prefix slot prefix_len free for the state token (prefix < max_prefix)";
    return JPI_ERR_SHAPE;
  }
  t->kp = c->kp;
  t->vpt = c->vpt;
  t->kp_bstride = (int64_t)c->Pmax * Dh;
  t->kp_lstride = (int64_t)c->Bmax * t->kp_bstride;
  t->vpt_ld = c->Ppad;
  t->vpt_bstride = (int64_t)Dh * c->Ppad;
  t->vpt_lstride = (int64_t)c->Bmax * t->vpt_bstride;
  t->prefix_len = c->d_prefix_len;
  t->rope_tab = c->rope_tab;
  t->H = c->H + c->n_corr;
  t->rope_base = c->cfg.rope_base;
  return JPI_OK;
}

jpi_status jpi::ae_prefix_bound(jpi_ctx* c, int batch, int prefix, int rope_rows) {
  if (c->batch != batch) {  // state rows were bound for another batch
    c->n_fixed = c->n_corr = 0;
    c->state_bound = false;
  }
  c->rope_rows = rope_rows;  // jpi_denoise rebuilds the table if the suffix length differs
  c->batch = batch;
  c->prefix = prefix;
  c->prefix_bound = true;
  return JPI_OK;
}
