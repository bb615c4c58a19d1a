/* libjpi future correction module: predicts the compressed VLM state at the
 * time the next chunk starts executing, from the actions committed until then.
 *
 * Section "Foresight-Aligned Asynchronous Correction" and Appendix
 * "Architecture of Future Correction Module": the committed actions pass an
 * MLP and a Transformer block whose last token is kept; the VLM final-layer
 * state is compressed to T' = 4 tokens of the action expert's width by a
 * Q-Former block; the two are concatenated, projected and passed through two
 * Transformer blocks; a correction head gives the correction item (T' tokens
 * for the action expert) and a confidence head a scalar confidence.  About
 * 40M parameters.  Algorithm 1 calls it on every scheduler iteration: after a
 * VLM refresh on the freshly compressed state, otherwise on its own previous
 * prediction (the hidden-state buffer B_h), which is why compression and
 * prediction are separate calls here.
 *
 * Readings where the paper is silent (also in the oracle's header):
 *   - every block is the VLM's pre-norm decoder layer at the expert's width
 *     (y = rms(h) (1 + w), one shared KV head, tanh-GeGLU MLP, no biases);
 *   - Q-Former: T' learned queries attend jointly to the VLM tokens' keys and
 *     values (their own two projections from d_VLM) and to their own; no
 *     positional rotation; the state is the block's residual output;
 *   - action branch: u_i = W2 gelu_tanh(W1 a_i + b1) + b2, one block with RoPE
 *     at positions 0..n-1 and no mask, s = the last token's residual output;
 *   - fusion along features with s repeated: z_j = W_f [c_j ; s] + b_f, then two
 *     blocks without positional rotation;
 *   - heads on y = rms(z) (1 + w_final): item_j = W_c y_j + b_c and
 *     confidence = w_conf . mean_j(y_j) + b_conf (unbounded).
 *
 * Conventions as include/jpi.h: every call returns a jpi_status, device
 * pointers are plain addresses on the module's device, streams are
 * hipStream_t passed as void*, bf16 data is raw 16-bit patterns.
 */
#ifndef JPI_CORR_H_
#define JPI_CORR_H_

#include <stdint.h>

#include "jpi.h"

#ifdef __cplusplus
extern "C" {
#endif

typedef struct jpi_corr jpi_corr;

typedef struct {
  int width;           /* d_AE: the action expert's width (1024) */
  int n_heads, n_kv_heads, head_dim, mlp_dim;  /* every block (8, 1, 128, 2048) */
  int action_dim;      /* A (32) */
  int vlm_width;       /* d_VLM (2048) */
  int n_query;         /* T': compressed tokens (4) */
  int max_batch;       /* rollouts per call, upper bound */
  int max_actions;     /* committed actions per call, upper bound (Delta) */
  int max_vlm_tokens;  /* T: VLM state tokens per rollout, upper bound */
  jpi_dtype dtype;     /* JPI_BF16 (the only type this version supports) */
  float rms_eps;       /* 1e-6 */
  float rope_base;     /* 1e4 */
} jpi_corr_config;

/* Allocate weights and activation buffers on `device`.  Errors: JPI_ERR_ARG
 * (sizes <= 0, n_kv_heads != 1, head_dim not in {64, 128, 256}, width, mlp_dim,
 * n_heads * head_dim or vlm_width not a multiple of 256, width > 4096,
 * action_dim > 256, n_query > 64), JPI_ERR_UNSUPPORTED (dtype other than
 * bf16), JPI_ERR_OOM, JPI_ERR_HIP. */
jpi_status jpi_corr_create(const jpi_corr_config* cfg, int device, jpi_corr** out);
jpi_status jpi_corr_destroy(jpi_corr* m);  /* NULL is a no-op */

/* Copy one tensor in (host or device memory; the caller keeps ownership;
 * complete when the call returns).  Names and shapes ([out][in]):
 *   qformer.query [T'][W] (fp32), qformer.xk.w [Dh][d_VLM], qformer.xv.w [Dh][d_VLM]
 *   action_mlp.0.w [W][A]  action_mlp.0.b [W]  action_mlp.1.w [W][W]  action_mlp.1.b [W]
 *   fuse.w [W][2W]  fuse.b [W]
 *   {qformer, action_block, blocks.0, blocks.1}.{attn_norm.w [W], q.w [heads*Dh][W],
 *     k.w [Dh][W], v.w [Dh][W], o.w [W][heads*Dh], mlp_norm.w [W], gate.w [F][W],
 *     up.w [F][W], down.w [W][F]}
 *   final_norm.w [W]  corr_head.w [W][W]  corr_head.b [W]  conf_head.w [1][W]  conf_head.b [1]
 * Matrices bf16; biases, norm weights and the queries fp32.  Errors:
 * JPI_ERR_ARG (unknown name, NULL), JPI_ERR_SHAPE, JPI_ERR_DTYPE, JPI_ERR_HIP. */
jpi_status jpi_corr_set_weight(jpi_corr* m, const char* name, const void* data, int64_t n_elems, jpi_dtype dt,
                               int is_device, void* stream);
jpi_status jpi_corr_finalize_weights(jpi_corr* m, void* stream);  /* JPI_ERR_STATE names a missing tensor */

/* Final-layer state compressor (the Q-Former): vlm_state (device, bf16
 * [batch][n_tokens][d_VLM], e.g. the hidden_out of jpi_vlm_prefill) ->
 * state_out (device, fp32 [batch][T'][W]).  Stream-ordered.  Errors:
 * JPI_ERR_ARG (NULL, batch or n_tokens outside [1, max]), JPI_ERR_STATE
 * (weights not finalized), JPI_ERR_HIP. */
jpi_status jpi_corr_compress(jpi_corr* m, const void* vlm_state, int batch, int n_tokens, float* state_out,
                             void* stream);

/* f_corr: from the compressed state (device, fp32 [batch][T'][W]: a
 * jpi_corr_compress output or the previous item) and the committed actions
 * (device, fp32 [batch][n_actions][A]) predict the correction item
 * (item_out, device fp32 [batch][T'][W], ready for jpi_bind_state's
 * corr_tokens) and the confidence (conf_out, device fp32 [batch]).  item_out
 * may alias state (the state is read before the item is written).
 * Stream-ordered.  Errors: JPI_ERR_ARG (NULL, batch or n_actions outside
 * [1, max]), JPI_ERR_STATE (weights not finalized), JPI_ERR_HIP. */
jpi_status jpi_corr_predict(jpi_corr* m, const float* state, const float* actions, int batch, int n_actions,
                            float* item_out, float* conf_out, void* stream);

const char* jpi_corr_last_error(const jpi_corr* m);  /* text of the last failure of a call on m */

#ifdef __cplusplus
}
#endif

#endif /* JPI_CORR_H_ */
