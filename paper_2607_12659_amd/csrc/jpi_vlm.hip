// VLM prefill (include/jpi_vlm.h): the LLM pass over the prefix tokens whose
// per-layer K and V condition the action expert (Appendix "Model
// Architecture of π series Models"), written straight into the expert's
// resident prefix buffers (Section "System Design": GPU-resident buffers).
//
// A pre-norm Gemma decoder layer is the action expert's layer with constant
// modulation: RMSNorm with (1 + w) scaling is the adaRMSNorm form with
// scale = w and shift = 0, and the plain residual is the gated one with
// gate = 1.  So the prefill runs the expert's kernels: the tiled GEMM with
// the QKV+RoPE, fp32 split-K and GeGLU epilogues, the batched attention
// (the prefix tokens are its query rows and its only keys), and the
// residual + norm row kernel.  The QKV epilogue writes K (rotated) into the
// expert's K buffer and V^T into its transposed-V buffer for the layer.
#include <cstring>
#include <string>
#include <vector>

#include "../../include/jpi_vlm.h"
#include "jpi_device.h"
#include "jpi_internal.h"

using namespace jpi;

namespace {

enum VKind { V_ATTN_NORM, V_Q, V_K, V_V, V_O, V_MLP_NORM, V_GATE, V_UP, V_DOWN, V_NLAYER, V_FINAL_NORM = V_NLAYER };
const char* vkind_suffix[V_NLAYER + 1] = {"attn_norm.w", "q.w", "k.w", "v.w", "o.w", "mlp_norm.w",
                                          "gate.w", "up.w", "down.w", "final_norm.w"};

}  // namespace

struct jpi_vlm {
  jpi_vlm_config cfg;
  int device = 0, n_cu = 0;
  std::string err;
  int L, W, nH, Dh, F, Bmax, Pmax, Mmax;
  // packed layer weights, the action expert's layout: [q|k|v rows (RoPE pack order) | O | gate/up interleaved | Down]
  void* w_layers = nullptr;
  size_t layer_elems = 0, off_o = 0, off_gu = 0, off_d = 0;
  float* norms = nullptr;  // [L][2][W] (attention, MLP) then the final [W]
  float *ones = nullptr, *zeros = nullptr;
  std::vector<char> have;
  bool finalized = false;
  // activations
  float* h = nullptr;
  void *y = nullptr, *q = nullptr, *o = nullptr, *z = nullptr;
  float* partial = nullptr;
  float* opart = nullptr;
  float2* rope = nullptr;
  int* zero_len = nullptr;  // [Bmax] zeros: the prefix tokens have no earlier keys
  int s_o = 1, s_d = 1;
};

namespace {

jpi_status vfail(jpi_vlm* v, jpi_status st, const std::string& msg) {
  if (v) v->err = msg;
  return st;
}

#define VCHK(v, expr)                                                                      \
  do {                                                                                     \
    hipError_t e_ = (expr);                                                                \
    if (e_ != hipSuccess) return vfail(v, JPI_ERR_HIP, std::string(#expr) + ": " + hipGetErrorString(e_)); \
  } while (0)

}  // namespace

extern "C" {

jpi_status jpi_vlm_destroy(jpi_vlm* v) {
  if (!v) return JPI_OK;
  (void)hipSetDevice(v->device);
  for (void* p : {(void*)v->w_layers, (void*)v->norms, (void*)v->ones, (void*)v->zeros, (void*)v->h, v->y, v->q, v->o,
                  v->z, (void*)v->partial, (void*)v->opart, (void*)v->rope, (void*)v->zero_len})
    if (p) (void)hipFree(p);
  delete v;
  return JPI_OK;
}

jpi_status jpi_vlm_create(const jpi_vlm_config* cfg, int device, jpi_vlm** out) {
  if (!cfg || !out) return JPI_ERR_ARG;
  *out = nullptr;
  const jpi_vlm_config& g = *cfg;
  if (g.n_layers < 1 || g.width < 256 || g.width % 256 || g.n_heads < 1 || g.n_kv_heads != 1 ||
      (g.head_dim != 64 && g.head_dim != 128 && g.head_dim != 256) || g.mlp_dim < 256 || g.mlp_dim % 256 ||
      (g.n_heads * g.head_dim) % 256 ||
      g.max_batch < 1 || g.max_prefix < 1 || !(g.rms_eps > 0.f) || !(g.rope_base > 1.f) ||
      g.width > 4096 || (size_t)g.max_batch * g.max_prefix > (1u << 20))
    return JPI_ERR_ARG;
  if (g.dtype != JPI_BF16) return JPI_ERR_UNSUPPORTED;
  jpi_vlm* v = new jpi_vlm();
  v->cfg = g;
  v->device = device;
  v->L = g.n_layers;
  v->W = g.width;
  v->nH = g.n_heads;
  v->Dh = g.head_dim;
  v->F = g.mlp_dim;
  v->Bmax = g.max_batch;
  v->Pmax = g.max_prefix;
  v->Mmax = g.max_batch * g.max_prefix;
  if (hipSetDevice(device) != hipSuccess) {
    jpi_vlm_destroy(v);
    return JPI_ERR_HIP;
  }
  hipDeviceProp_t prop;
  if (hipGetDeviceProperties(&prop, device) != hipSuccess) {
    jpi_vlm_destroy(v);
    return JPI_ERR_HIP;
  }
  v->n_cu = prop.multiProcessorCount;
  const size_t W = v->W, Dh = v->Dh, nH = v->nH, F = v->F, M = v->Mmax;
  v->off_o = (nH + 2) * Dh * W;
  v->off_gu = v->off_o + W * nH * Dh;
  v->off_d = v->off_gu + 2 * F * W;
  v->layer_elems = v->off_d + W * F;
  v->s_o = gemm_pick_splitk(JPI_BF16, (int)M, (int)W, (int)(nH * Dh), v->n_cu);
  v->s_d = gemm_pick_splitk(JPI_BF16, (int)M, (int)W, (int)F, v->n_cu);
  const size_t nch = (size_t)attn_n_chunks(JPI_BF16, 0, v->Pmax);
  bool ok = true;
  auto alloc = [&](void** p, size_t bytes) {
    if (ok && hipMalloc(p, bytes) != hipSuccess) ok = false;
  };
  alloc(&v->w_layers, (size_t)v->L * v->layer_elems * 2);
  alloc((void**)&v->norms, ((size_t)2 * v->L + 1) * W * 4);
  alloc((void**)&v->ones, W * 4);
  alloc((void**)&v->zeros, W * 4);
  alloc((void**)&v->h, M * W * 4);
  alloc(&v->y, M * W * 2);
  alloc(&v->q, M * nH * Dh * 2);
  alloc(&v->o, M * nH * Dh * 2);
  alloc(&v->z, M * F * 2);
  alloc((void**)&v->partial, (size_t)(v->s_o > v->s_d ? v->s_o : v->s_d) * M * W * 4);
  alloc((void**)&v->opart, M * nH * nch * (Dh + 2) * 4);
  alloc((void**)&v->rope, M * (Dh / 2) * sizeof(float2));
  alloc((void**)&v->zero_len, v->Bmax * 4);
  if (!ok) {
    (void)hipGetLastError();
    jpi_vlm_destroy(v);
    return JPI_ERR_OOM;
  }
  if (launch_fill_f32(v->ones, (int)W, 1.0f, 0) != hipSuccess || launch_fill_f32(v->zeros, (int)W, 0.0f, 0) != hipSuccess ||
      launch_fill_i32(v->zero_len, v->Bmax, 0, 0) != hipSuccess) {
    jpi_vlm_destroy(v);
    return JPI_ERR_HIP;
  }
  if (hipDeviceSynchronize() != hipSuccess) {
    jpi_vlm_destroy(v);
    return JPI_ERR_HIP;
  }
  v->have.assign((size_t)V_NLAYER * v->L + 1, 0);
  *out = v;
  return JPI_OK;
}

jpi_status jpi_vlm_set_weight(jpi_vlm* v, const char* name, const void* data, int64_t n_elems, jpi_dtype dt,
                              int is_device, void* stream) {
  if (!v) return JPI_ERR_ARG;
  if (!name || !data) return vfail(v, JPI_ERR_ARG, "jpi_vlm_set_weight: name or data is NULL");
  int kind = -1, layer = -1;
  if (strcmp(name, vkind_suffix[V_FINAL_NORM]) == 0) {
    kind = V_FINAL_NORM;
  } else if (strncmp(name, "layers.", 7) == 0 && name[7] >= '0' && name[7] <= '9') {
    char* end = nullptr;
    const long l = strtol(name + 7, &end, 10);
    if (end && *end == '.' && l >= 0 && l < v->L)
      for (int k = 0; k < V_NLAYER; ++k)
        if (strcmp(end + 1, vkind_suffix[k]) == 0) {
          kind = k;
          layer = (int)l;
        }
  }
  if (kind < 0) return vfail(v, JPI_ERR_ARG, std::string("unknown tensor name: ") + name);
  const int64_t W = v->W, Dh = v->Dh, nH = v->nH, F = v->F;
  const bool vec = kind == V_ATTN_NORM || kind == V_MLP_NORM || kind == V_FINAL_NORM;
  int64_t want = 0;
  switch (kind) {
    case V_ATTN_NORM: case V_MLP_NORM: case V_FINAL_NORM: want = W; break;
    case V_Q: want = nH * Dh * W; break;
    case V_K: case V_V: want = Dh * W; break;
    case V_O: want = W * nH * Dh; break;
    case V_GATE: case V_UP: want = F * W; break;
    case V_DOWN: want = W * F; break;
  }
  if (n_elems != want)
    return vfail(v, JPI_ERR_SHAPE, std::string(name) + ": expected " + std::to_string(want) + " elements, got " +
                                       std::to_string(n_elems));
  if (dt != (vec ? JPI_F32 : JPI_BF16))
    return vfail(v, JPI_ERR_DTYPE, std::string(name) + (vec ? ": norm weights must be JPI_F32" : ": matrices must be JPI_BF16"));
  VCHK(v, hipSetDevice(v->device));
  hipStream_t s = (hipStream_t)stream;
  const hipMemcpyKind ck = is_device ? hipMemcpyDeviceToDevice : hipMemcpyHostToDevice;
  char* lay = layer >= 0 ? (char*)v->w_layers + (size_t)layer * v->layer_elems * 2 : nullptr;
  if (vec) {
    float* dst = kind == V_FINAL_NORM ? v->norms + (size_t)2 * v->L * W
                                      : v->norms + ((size_t)2 * layer + (kind == V_MLP_NORM)) * W;
    VCHK(v, hipMemcpyAsync(dst, data, W * 4, ck, s));
  } else if (kind == V_O || kind == V_DOWN) {
    VCHK(v, hipMemcpyAsync(lay + (kind == V_O ? v->off_o : v->off_d) * 2, data, (size_t)n_elems * 2, ck, s));
  } else {
    // row-permuted copies: q/k rows in RoPE pack order after q heads, v rows
    // natural; gate/up rows interleaved in 32-row groups [gate 16 | up 16]
    char* base = kind == V_GATE || kind == V_UP ? lay + v->off_gu * 2 : lay;
    const BlockMatrix bm = kind == V_Q ? BM_Q : kind == V_K ? BM_K : kind == V_V ? BM_V : kind == V_GATE ? BM_GATE : BM_UP;
    std::vector<int> map((size_t)(n_elems / W));
    for (size_t r = 0; r < map.size(); ++r) map[r] = block_pack_row(bm, (int)r, (int)nH, (int)Dh);
    const hipError_t e = upload_rows(base, map, (int)(W * 2), data, is_device != 0, s);
    if (e != hipSuccess) return vfail(v, JPI_ERR_HIP, std::string("jpi_vlm_set_weight: ") + hipGetErrorString(e));
  }
  VCHK(v, hipStreamSynchronize(s));
  v->have[kind == V_FINAL_NORM ? (size_t)V_NLAYER * v->L : (size_t)layer * V_NLAYER + kind] = 1;
  v->finalized = false;
  return JPI_OK;
}

jpi_status jpi_vlm_finalize_weights(jpi_vlm* v, void* stream) {
  (void)stream;
  if (!v) return JPI_ERR_ARG;
  for (int l = 0; l < v->L; ++l)
    for (int k = 0; k < V_NLAYER; ++k)
      if (!v->have[(size_t)l * V_NLAYER + k])
        return vfail(v, JPI_ERR_STATE, "missing tensor layers." + std::to_string(l) + "." + vkind_suffix[k]);
  if (!v->have[(size_t)V_NLAYER * v->L]) return vfail(v, JPI_ERR_STATE, "missing tensor final_norm.w");
  v->finalized = true;
  return JPI_OK;
}

jpi_status jpi_vlm_prefill(jpi_vlm* v, const float* emb, int batch, int prefix, jpi_ctx* ae, void* hidden_out,
                           void* stream) {
  if (!v) return JPI_ERR_ARG;
  if (!emb || !ae) return vfail(v, JPI_ERR_ARG, "jpi_vlm_prefill: emb or ae is NULL");
  if (batch < 1 || batch > v->Bmax || prefix < 1 || prefix > v->Pmax)
    return vfail(v, JPI_ERR_ARG, "jpi_vlm_prefill: batch or prefix outside [1, max_batch] / [1, max_prefix]");
  if (!v->finalized) return vfail(v, JPI_ERR_STATE, "jpi_vlm_prefill: weights are not finalized");
  AePrefixTarget tg;
  const char* why = nullptr;
  const jpi_status ts = ae_prefix_target(ae, v->L, v->Dh, JPI_BF16, batch, prefix, &tg, &why);
  if (ts != JPI_OK) return vfail(v, ts, std::string("jpi_vlm_prefill: ") + (why ? why : "bad target"));
  VCHK(v, hipSetDevice(v->device));
  hipStream_t s = (hipStream_t)stream;
  const int W = v->W, nH = v->nH, Dh = v->Dh, F = v->F, L = v->L, M = batch * prefix;
  const float eps = v->cfg.rms_eps;
  const size_t lay_bytes = v->layer_elems * 2;
  const float* nrm = v->norms;

  VCHK(v, hipMemcpyAsync(v->h, emb, (size_t)M * W * 4, hipMemcpyDeviceToDevice, s));
  VCHK(v, launch_norm_rows(v->h, nrm, v->y, M, W, eps, s));
  VCHK(v, launch_rope_table(v->zero_len, v->rope, batch, prefix, Dh, v->cfg.rope_base, s));
  BlockLaunch b{};
  b.B = batch;
  b.H = prefix;
  b.W = W;
  b.nH = nH;
  b.Dh = Dh;
  b.F = F;
  b.n_cu = v->n_cu;
  b.off_o = v->off_o;
  b.off_gu = v->off_gu;
  b.off_d = v->off_d;
  b.h = v->h;
  b.y = v->y;
  b.q = v->q;
  b.o = v->o;
  b.z = v->z;
  b.partial = v->partial;
  b.s_o = v->s_o;
  b.s_d = v->s_d;
  b.opart = v->opart;
  b.ks_bstride = tg.kp_bstride;
  b.vst_ld = tg.vpt_ld;
  b.kp_bstride = tg.kp_bstride;
  b.vpt_bstride = tg.vpt_bstride;
  b.vpt_dstride = tg.vpt_ld;
  b.prefix_len = v->zero_len;  // the prefix tokens are the query rows and their own keys
  b.P = 0;
  b.rope = v->rope;
  b.ones = v->ones;
  b.zeros = v->zeros;
  b.eps = eps;
  for (int l = 0; l < L; ++l) {
    // K (rotated) and V^T go straight into the expert's buffers of layer l
    b.w = (const char*)v->w_layers + (size_t)l * lay_bytes;
    b.ks = (char*)tg.kp + (size_t)l * tg.kp_lstride * 2;
    b.vst = (char*)tg.vpt + (size_t)l * tg.vpt_lstride * 2;
    b.kp = b.ks;
    b.vpt = b.vst;
    b.mlp_norm = nrm + ((size_t)2 * l + 1) * W;
    b.next_norm = nrm + (l + 1 < L ? (size_t)2 * (l + 1) : (size_t)2 * L) * W;  // next layer's norm, else the final one
    VCHK(v, enqueue_block(b, s));
  }
  if (hidden_out) VCHK(v, hipMemcpyAsync(hidden_out, v->y, (size_t)M * W * 2, hipMemcpyDeviceToDevice, s));
  // bind: prefix_len = prefix for every rollout; the expert's own rows sit at positions prefix + i
  VCHK(v, launch_fill_i32(tg.prefix_len, batch, prefix, s));
  VCHK(v, launch_rope_table(tg.prefix_len, tg.rope_tab, batch, tg.H, Dh, tg.rope_base, s));
  return ae_prefix_bound(ae, batch, prefix, tg.H);
}

const char* jpi_vlm_last_error(const jpi_vlm* v) { return v ? v->err.c_str() : "vlm is NULL"; }

}  // extern "C"
