/* libjpi VLM prefill: the LLM pass that produces the action expert's prefix KV.
 *
 * The π-series VLA runs its LLM over the observation and instruction tokens
 * once per VLM refresh; the KV cache of each of its layers conditions the
 * action expert's layer of the same index (Appendix "Model Architecture of π
 * series Models"; Table "pi_architecture": 18 layers, width 2048, 8 heads of
 * dimension 256 sharing one KV head).  The paper keeps that cache resident on
 * the device instead of copying it between the two models (Section "System
 * Design", GPU-resident intermediate buffers); here the prefill writes every
 * layer's K (after RoPE) and V straight into the resident prefix buffers of
 * a jpi_ctx and marks them bound, so a jpi_denoise can follow at once.
 *
 * Layer (readings where the paper is silent): pre-norm Gemma decoder,
 * y = rms(h) * (1 + w) with eps = cfg.rms_eps, q/k/v projections without bias,
 * RoPE on q and k at positions 0 .. prefix-1 (half-split pairs, base
 * cfg.rope_base), attention over the whole prefix (no causal mask), output
 * projection and residual, then the same norm and a tanh-GeGLU MLP with
 * residual.  The input is the token embeddings; the final-layer hidden state
 * is rms(h) * (1 + w_final).
 *
 * Conventions as include/jpi.h: every call returns a jpi_status, device
 * pointers are plain addresses, streams are hipStream_t passed as void*.
 */
#ifndef JPI_VLM_H_
#define JPI_VLM_H_

#include <stdint.h>

#include "jpi.h"

#ifdef __cplusplus
extern "C" {
#endif

typedef struct jpi_vlm jpi_vlm;

typedef struct {
  int n_layers, width, n_heads, n_kv_heads, head_dim, mlp_dim;
  int max_batch, max_prefix;
  jpi_dtype dtype;   /* JPI_BF16 (the only type this version supports) */
  float rms_eps;     /* 1e-6 */
  float rope_base;   /* 1e4 */
} jpi_vlm_config;

/* Allocate the weights and the activation buffers for max_batch x max_prefix
 * tokens on `device`.  Errors: JPI_ERR_ARG (sizes <= 0, n_kv_heads != 1,
 * head_dim not in {64, 128, 256}, width, mlp_dim or n_heads * head_dim not a
 * multiple of 256, width > 4096), JPI_ERR_UNSUPPORTED (dtype other than bf16),
 * JPI_ERR_OOM, JPI_ERR_HIP. */
jpi_status jpi_vlm_create(const jpi_vlm_config* cfg, int device, jpi_vlm** out);
jpi_status jpi_vlm_destroy(jpi_vlm* vlm);  /* NULL is a no-op */

/* Copy one tensor in (host or device memory; the caller keeps ownership).
 * Names: layers.{l}.attn_norm.w [W], layers.{l}.q.w [heads*Dh][W],
 * layers.{l}.k.w and .v.w [Dh][W], layers.{l}.o.w [W][heads*Dh],
 * layers.{l}.mlp_norm.w [W], layers.{l}.gate.w and .up.w [F][W],
 * layers.{l}.down.w [W][F], final_norm.w [W].  Matrices in the config dtype,
 * norm weights fp32.  Errors: JPI_ERR_ARG, JPI_ERR_SHAPE, JPI_ERR_DTYPE. */
jpi_status jpi_vlm_set_weight(jpi_vlm* vlm, const char* name, const void* data, int64_t n_elems, jpi_dtype dt,
                              int is_device, void* stream);
jpi_status jpi_vlm_finalize_weights(jpi_vlm* vlm, void* stream);  /* JPI_ERR_STATE names a missing tensor */

/* Run the LLM over emb (device, fp32 [batch][prefix][width]) and write each
 * layer's K and V into ae's resident prefix buffers for rollouts 0..batch-1,
 * binding them with prefix_len = prefix for every rollout (as jpi_bind_prefix
 * would).  hidden_out (device, [batch][prefix][width] in the config dtype) gets
 * the final-layer hidden state, or is skipped when NULL.  Stream-ordered.
 * ae must have the same layer count and head_dim, one KV head, the same dtype,
 * max_batch >= batch and max_prefix >= prefix.  Errors: JPI_ERR_ARG (NULL,
 * batch or prefix out of range), JPI_ERR_SHAPE (ae mismatch), JPI_ERR_STATE
 * (weights not finalized), JPI_ERR_HIP. */
jpi_status jpi_vlm_prefill(jpi_vlm* vlm, const float* emb, int batch, int prefix, jpi_ctx* ae, void* hidden_out,
                           void* stream);

const char* jpi_vlm_last_error(const jpi_vlm* vlm);  /* text of the last failure of a call on vlm */

#ifdef __cplusplus
}
#endif

#endif /* JPI_VLM_H_ */
