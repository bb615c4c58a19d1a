/*
 * libjpi — C ABI of an MI355X (gfx950) flow-matching action-expert denoiser.
 *
 * The operation (paper: "Jetson-PI: Towards Onboard Real-Time Robot Control
 * via Foresight-Aligned Asynchronous Inference"):
 *   - Background section and Appendix "Model Architecture of pi series
 *     Models": the VLM passes its per-layer KV cache to the action expert,
 *     a DiT whose input is random action noise; at each layer the action
 *     tokens attend with their own queries to keys/values formed by
 *     concatenating the LLM layer's KV cache with the action tokens' own;
 *     a fixed number of flow-matching denoising steps refines the noise
 *     into an action chunk.
 *   - Algorithm 1 ("confidence-based scheduling"): the call f_act(h, B_kv)
 *     is made on every scheduler iteration; it is what jpi_denoise runs.
 *   - Section "System Design": the computation graph is built once and
 *     reused (fixed token length), intermediates stay in fixed-size
 *     GPU-resident buffers, and all denoising steps are unrolled into one
 *     graph.  libjpi captures the whole N-step loop once per shape into a
 *     HIP graph over context-owned buffers.
 *
 * Semantics fixed where the paper is silent (also in the oracle's header):
 *   flow from noise at t=1 to actions at t=0, t_k = 1 - k/N, explicit Euler
 *   x <- x + dt v(x, t_k) with dt = -1/N; adaRMSNorm y = rms(h)(1+scale)+shift
 *   with (scale, shift, gate) = Linear(swish(T2 swish(T1 emb(t) + b1) + b2)),
 *   residual h += gate * sublayer(y); tanh-GELU GeGLU MLP; one KV head shared
 *   by all query heads; RoPE (base rope_base, half-split pairs) on action
 *   queries/keys at positions prefix_len + i; prefix K already rotated;
 *   each action query sees prefix slots j < prefix_len and all action keys;
 *   rows i < n_fixed are committed actions, never updated.
 *
 * Conventions
 *   - Every call returns a jpi_status; nothing throws or aborts.  The text of
 *     the last failure on a context is jpi_last_error(ctx).
 *   - "device" pointers are HIP device pointers on the context's device;
 *     "host" pointers are ordinary CPU memory.  The library never frees or
 *     keeps caller memory beyond the stream order of the call that used it.
 *   - Streams are hipStream_t values passed as void* (NULL = null stream).
 *     Work is enqueued asynchronously; synchronise the stream (or call
 *     jpi_sync) before reading outputs on the host.
 *   - A context is not thread-safe; use one context per stream.
 *   - Matrices are row-major [out][in] (y = x W^T); action chunks are
 *     [batch][horizon][A].  bf16 data is passed as raw 16-bit patterns.
 */
#ifndef JPI_H_
#define JPI_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define JPI_ABI_VERSION 4

typedef enum {
  JPI_OK = 0,
  JPI_ERR_ARG = 1,          /* NULL pointer, value out of range, unknown name */
  JPI_ERR_SHAPE = 2,        /* element count or size does not match the config */
  JPI_ERR_DTYPE = 3,        /* wrong element type for this tensor */
  JPI_ERR_STATE = 4,        /* call made in the wrong order (e.g. no weights yet) */
  JPI_ERR_OOM = 5,          /* device allocation failed */
  JPI_ERR_HIP = 6,          /* a HIP runtime call failed (text in jpi_last_error) */
  JPI_ERR_UNSUPPORTED = 7   /* valid request this version does not implement */
} jpi_status;

typedef enum { JPI_F32 = 0, JPI_BF16 = 1 } jpi_dtype;

/* Expert variants of the π series (Appendix "Model Architecture of π series
 * Models" lists one action expert for π0 and π0.5; the paper does not spell
 * out how time and state enter, so both forms here are readings):
 *   JPI_VARIANT_ADARMS: time conditions every norm (adaRMSNorm scale, shift
 *     and gate from a time MLP), the default described above.
 *   JPI_VARIANT_ACTION_TIME: π0 style -- plain RMSNorm (1 + w) and ungated
 *     residuals; time enters through an action-time MLP on each action token,
 *     h_i = W_o swish(W_i [W_a a_i + b_a ; e(t)] + b_i) + b_o; the robot state
 *     is one suffix token W_s s + b_s ahead of the actions (RoPE position
 *     prefix_len; actions at prefix_len + 1 + i) that attends to the prefix and
 *     itself only, so its keys and values are computed once per call and
 *     occupy prefix slot prefix_len of every layer. */
typedef enum { JPI_VARIANT_ADARMS = 0, JPI_VARIANT_ACTION_TIME = 1 } jpi_variant;

typedef struct {
  int n_layers;     /* L   (pi0.5 expert: 18, Table "pi_architecture") */
  int width;        /* W   (1024) */
  int n_heads;      /* query heads (8) */
  int n_kv_heads;   /* KV heads; this version requires 1 */
  int head_dim;     /* Dh  (256); 64, 128 or 256 */
  int mlp_dim;      /* F   GeGLU hidden width (4096) */
  int action_dim;   /* A   (32) */
  int horizon;      /* H   action tokens per chunk (50) */
  int max_batch;    /* rollouts per call, upper bound for resident buffers */
  int max_prefix;   /* prefix tokens per rollout, upper bound */
  jpi_dtype dtype;  /* storage type of matrices, prefix KV and activations */
  float rms_eps;    /* 1e-6 */
  float rope_base;  /* 1e4 */
  int max_corr;     /* correction tokens per rollout, upper bound (0: none; at most 64) */
  int variant;      /* jpi_variant (0: JPI_VARIANT_ADARMS) */
  int state_dim;    /* robot-state values per rollout (JPI_VARIANT_ACTION_TIME only; else 0) */
} jpi_config;

typedef struct jpi_ctx jpi_ctx;

/* ABI version of the loaded library (JPI_ABI_VERSION it was built with). */
int jpi_abi_version(void);

/* Static description of a status code.  Never NULL. */
const char* jpi_status_str(jpi_status s);

/* Text of the last failure on ctx ("" if none; a static message if ctx is NULL). */
const char* jpi_last_error(const jpi_ctx* ctx);

/* Create a context on HIP device `device`.  The config is validated on the
 * host before any HIP call: dims must be positive, n_kv_heads == 1,
 * n_heads % n_kv_heads == 0, head_dim 64, 128 or 256, width a multiple of
 * 64, mlp_dim a multiple of 64, max_corr in [0, 64], variant known, state_dim
 * in [1, 4096] for the action-time variant (which also needs max_corr 0 and
 * max_prefix >= 1) and 0 otherwise (JPI_ERR_ARG otherwise).  All resident buffers
 * (max_batch x max_prefix prefix KV, activations, partial sums, weights) are
 * allocated here and owned by the context (Section "System Design":
 * GPU-resident intermediate buffers).  On failure *out is NULL. */
jpi_status jpi_create(const jpi_config* cfg, int device, jpi_ctx** out);

/* Free everything the context owns.  NULL is accepted. */
jpi_status jpi_destroy(jpi_ctx* ctx);

/* Copy one named expert tensor into the context (packed for the kernels).
 * Names and shapes ([out][in] for matrices):
 *   action_in.w [W][A]  action_in.b [W]
 *   time_mlp.0.w [W][W] time_mlp.0.b [W]  time_mlp.1.w [W][W] time_mlp.1.b [W]
 *   layers.{l}.attn_mod.w [3W][W]  .attn_mod.b [3W]   (scale | shift | gate)
 *   layers.{l}.q.w [nH*Dh][W]  .k.w [Dh][W]  .v.w [Dh][W]  .o.w [W][nH*Dh]
 *   layers.{l}.mlp_mod.w [3W][W]  .mlp_mod.b [3W]
 *   layers.{l}.gate.w [F][W]  .up.w [F][W]  .down.w [W][F]
 *   final_mod.w [2W][W]  final_mod.b [2W]           (scale | shift)
 *   action_out.w [A][W]  action_out.b [A]
 * JPI_VARIANT_ACTION_TIME replaces the time MLP and every *_mod tensor by
 *   action_time_mlp_in.w [W][2W] (columns: action part, then time part)
 *   action_time_mlp_in.b [W]  action_time_mlp_out.w [W][W]  action_time_mlp_out.b [W]
 *   state_proj.w [W][state_dim]  state_proj.b [W]
 *   layers.{l}.attn_norm.w [W]  layers.{l}.mlp_norm.w [W]  final_norm.w [W]
 * Matrices must have dt == cfg.dtype, vectors dt == JPI_F32.  `data` is a
 * device pointer if is_device != 0, else a host pointer; the caller keeps
 * ownership.  The copy is complete when the call returns (the stream is
 * synchronised).  Errors: JPI_ERR_ARG (unknown name / NULL), JPI_ERR_SHAPE
 * (n_elems), JPI_ERR_DTYPE.  Setting a weight invalidates cached tables and
 * graphs. */
jpi_status jpi_set_weight(jpi_ctx* ctx, const char* name, const void* data, int64_t n_elems,
                          jpi_dtype dt, int is_device, void* stream);

/* Check that every tensor has been set (JPI_ERR_STATE names the first
 * missing one) and mark the weights ready. */
jpi_status jpi_finalize_weights(jpi_ctx* ctx, void* stream);

/* Zero-copy producer path: the context's resident prefix K and V buffers,
 * each [L][max_batch][max_prefix][Dh] of cfg.dtype.  A producer (the VLM
 * prefill) may write rollout b, layer l, token j at
 * ((l*max_batch + b)*max_prefix + j)*Dh and then call jpi_bind_prefix with
 * k == *k_out, v == *v_out and prefix == max_prefix (no copy is made). */
jpi_status jpi_prefix_buffers(jpi_ctx* ctx, void** k_out, void** v_out);

/* Bind the per-layer prefix KV cache (Appendix: keys/values of the LLM layer).
 * k, v: device pointers, [L][batch][prefix][Dh] of cfg.dtype, prefix K already
 * rotated.  They are copied (stream-ordered) into the resident buffers unless
 * they are those buffers.  prefix_len_host: host array [batch] of valid
 * lengths in [0, prefix] (NULL = all `prefix`); slots j >= prefix_len are
 * never read.  Errors: JPI_ERR_ARG (NULL), JPI_ERR_SHAPE (batch outside
 * [1, max_batch], prefix outside [0, max_prefix], prefix_len out of range). */
jpi_status jpi_bind_prefix(jpi_ctx* ctx, const void* k, const void* v, const int32_t* prefix_len_host,
                           int batch, int prefix, void* stream);

/* Bind the per-call state besides the prefix (Algorithm 1: f_act(h, B_kv)).
 *   - n_fixed committed action rows: actions already committed for execution
 *     while the next chunk is inferred.  committed_dev: device
 *     [batch][n_fixed][A] fp32 (may be NULL if n_fixed == 0).  n_fixed in
 *     [0, horizon).
 *   - n_corr correction tokens h (Section "Foresight-Aligned Asynchronous
 *     Correction": the correction item the future correction module hands to
 *     the action expert).  corr_tokens: device [batch][n_corr][W] fp32 (may
 *     be NULL if n_corr == 0), n_corr in [0, max_corr].  They enter every
 *     step as extra suffix tokens ahead of the action tokens: token j at RoPE
 *     position prefix_len + j, action token i at prefix_len + n_corr + i; they
 *     skip the action in-projection, go through every layer with the step's
 *     modulation, attend to and are attended by all suffix tokens, restart
 *     from the given values at every step and are never Euler-updated.
 * Both are copied stream-ordered into context buffers.  Must follow
 * jpi_bind_prefix, which sets the batch (binding a prefix with a different
 * batch clears both).  Correction rows run on both paths (the single-launch
 * kernel while batch * (n_corr + horizon) <= 64).  Errors: JPI_ERR_ARG
 * (NULL ctx or data, counts out of range), JPI_ERR_STATE (no prefix bound). */
jpi_status jpi_bind_state(jpi_ctx* ctx, const float* committed_dev, int n_fixed, const void* corr_tokens,
                          int n_corr, void* stream);

/* Robot state for JPI_VARIANT_ACTION_TIME: state_dev, device fp32
 * [batch][state_dim], copied stream-ordered; required before jpi_denoise.
 * Must follow jpi_bind_prefix (batch).  With this variant every prefix_len
 * must stay below max_prefix (the state token takes slot prefix_len), and
 * correction tokens are not supported.  Errors: JPI_ERR_ARG (NULL),
 * JPI_ERR_STATE (no prefix bound), JPI_ERR_UNSUPPORTED (other variant). */
jpi_status jpi_bind_robot_state(jpi_ctx* ctx, const float* state_dev, void* stream);

/* Flow time of the committed rows (a variant; Algorithm 1 commits actions
 * that are already final, while the paper does not say at which flow time
 * the expert sees them).  enable = 0 (default): committed rows share the
 * step's t_k with every other row.  enable != 0: committed rows carry t = 0
 * (clean actions) at every step, so their adaRMSNorm scale, shift and gate
 * come from the time conditioning at t = 0 while the other rows use t_k; the
 * correction tokens keep t_k.  Takes effect at the next jpi_denoise.  The
 * action-time variant ignores it (its time enters through the action-time
 * MLP, at the step's t for every action row).
 * Errors: JPI_ERR_ARG (NULL ctx). */
jpi_status jpi_set_committed_t0(jpi_ctx* ctx, int enable);

/* Denoise one action chunk per rollout: x starts at noise (rows < n_fixed
 * take the committed values), then n_steps Euler steps of the velocity field
 * run, and x is written to actions_dev.  noise_dev, actions_dev: device
 * [batch][H][A] fp32 (may alias).  Stream-ordered and asynchronous.  The first
 * call per (batch, prefix, n_steps, n_fixed, n_corr) builds the
 * modulation tables for the N step times and captures the N-step loop into a
 * HIP graph; later calls replay it.  Errors: JPI_ERR_STATE (weights not
 * finalized or no prefix bound), JPI_ERR_ARG (NULL, n_steps < 1).
 *
 * Co-residency: on the single-launch path (bf16, batch * (n_corr + H) <= 64)
 * the whole loop is one kernel of one workgroup per compute unit whose
 * workgroups wait for each other through memory.  That needs every
 * workgroup resident at once: do not let other device work (another stream,
 * another context or process on the same GPU) run concurrently with it.  If
 * some workgroups cannot start, the others wait a bounded number of polls,
 * then stop; the launch still terminates, the actions are invalid, and the
 * next jpi_sync returns JPI_ERR_HIP.  A caller that reads actions_dev
 * therefore checks the status of jpi_sync (not only of a stream
 * synchronisation) before using them. */
jpi_status jpi_denoise(jpi_ctx* ctx, const float* noise_dev, int n_steps, float* actions_dev, void* stream);

/* Synchronise `stream` and report asynchronous HIP errors as JPI_ERR_HIP,
 * including a wait of the single-launch denoise kernel for its producer
 * workgroups that timed out (its output is then invalid). */
jpi_status jpi_sync(jpi_ctx* ctx, void* stream);

/* ---- kernel-level entry points used by the parity tests ------------------ */

/* C[M][N] (fp32) = A[M][K] . W[N][K]^T with the library's GEMM kernel.
 * A, W: device, dtype dt (JPI_BF16 -> bf16 MFMA with fp32 accumulation,
 * JPI_F32 -> fp32 MFMA).  splitk >= 1 splits K across workgroups with a
 * fixed-order reduction.  Errors: JPI_ERR_ARG (NULL, sizes < 1, K not a
 * multiple of 32*splitk). */
jpi_status jpi_debug_gemm(const void* A, const void* W, float* C, int M, int N, int K, jpi_dtype dt,
                          int splitk, void* stream);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): the GEMM of
 * jpi_debug_gemm -- same arguments, same kernels, same fixed-order split-K
 * reduction, bitwise the same result -- without any allocation and without
 * synchronising the stream (the result is ready in stream order).  The
 * split-K partial slices (splitk * M * N fp32; none when splitk == 1) live in
 * a static device array of jpi_gemm_noalloc_scratch_bytes() bytes (16 MiB)
 * that each GPU holds from the library's load until the process ends; larger
 * requests fail with JPI_ERR_ARG before anything is enqueued.  Every call on
 * one GPU shares that array: calls whose execution overlaps on one GPU
 * (different streams, or host threads) race on it and must be ordered by the
 * caller.  The array keeps the last call's contents; nothing in it needs to
 * start at zero.  Errors: JPI_ERR_ARG (as jpi_debug_gemm, plus the size
 * limit), JPI_ERR_HIP (a launch failed); the text of the last failure on the
 * calling thread is jpi_gemm_noalloc_last_error(). */
jpi_status jpi_gemm_noalloc(const void* A, const void* W, float* C, int M, int N, int K, jpi_dtype dt, int splitk,
                            void* stream);
size_t jpi_gemm_noalloc_scratch_bytes(void);
const char* jpi_gemm_noalloc_last_error(void);

/* Prefix+self attention of one layer for `batch` rollouts with one shared KV
 * head, as used inside jpi_denoise (queries already rotated):
 *   q  [batch][n_heads][H][Dh], ks/vs [batch][H][Dh], kp/vp [batch][P][Dh]
 *   (all dtype dt, device), prefix_len_host [batch] host,
 *   out [batch*H][n_heads*Dh] fp32 device.
 * Errors: JPI_ERR_ARG. */
jpi_status jpi_debug_attention(const void* q, const void* ks, const void* vs, const void* kp, const void* vp,
                               const int32_t* prefix_len_host, int batch, int n_heads, int H, int P,
                               int Dh, jpi_dtype dt, float* out, void* stream);

/* The context's transposed prefix V, the attention kernels' P.V operand:
 * [L][max_batch][Dh][ld] of cfg.dtype, value j of rollout b, layer l at
 * ((l*max_batch + b)*Dh + d)*ld + j.  jpi_bind_prefix fills it from the bound
 * V; the VLM prefill's in-place hand-off writes it directly (and not the V
 * buffer of jpi_prefix_buffers).  Read-only for callers (tests inspect it).
 * Errors: JPI_ERR_ARG (NULL). */
jpi_status jpi_debug_prefix_vt(jpi_ctx* ctx, void** vt_out, int* ld_out);

/* ---- measurement support (used by the benchmark) ---------------------------- */

/* Phase timestamps of the last single-launch denoise (a library built with
 * the kernel's trace mode, -DJPI_PERSIST_TRACE=1, by
 * paper_2607_12659_amd/trace_links.py; the normal build returns
 * JPI_ERR_UNSUPPORTED).  Sets *n_workgroups (the launch's grid), *n_slots
 * (1 + 3 x phases of the call, 8 phases per layer: slot 0 is each
 * workgroup's start; phase p has slots 1 + 3p + {0: the flags of its
 * producers were seen, 1: its operands were loaded, 2: its end}) and
 * *ticks_per_us of the counter;
 * when host_out holds cap >= n_workgroups * n_slots entries it also
 * synchronises the device and copies the stamps, [workgroup][slot].
 * Errors: JPI_ERR_ARG (NULL), JPI_ERR_UNSUPPORTED, JPI_ERR_HIP. */
jpi_status jpi_debug_persist_trace(jpi_ctx* ctx, uint64_t* host_out, int64_t cap, int* n_workgroups, int* n_slots,
                                   double* ticks_per_us);

/* Test hook for the single-launch kernel's failure path.  That kernel's waits
 * for its producers' completion flags give up after `polls` unsuccessful
 * polls (its waits for split-K slice data keep the default bound and stop as
 * soon as their workgroup gave up elsewhere); a workgroup that gave up
 * records an error word and waits no more, so a launch always ends, jpi_sync
 * reports JPI_ERR_HIP ("... timed out") and the call's output is invalid.
 * polls = 0 restores the default bound (2^21 polls, seconds).  A tiny bound
 * forces the failure from the host while every kernel still exits normally.
 * Synchronises the device and drops the captured graphs (the bound is a
 * launch argument).
 * Errors: JPI_ERR_ARG (NULL ctx), JPI_ERR_HIP. */
jpi_status jpi_debug_set_spin_limit(jpi_ctx* ctx, uint32_t polls);

/* Kernel kinds of one denoise step, in launch order per layer. */
typedef enum {
  JPI_KERNEL_NONE = -1,
  JPI_KERNEL_QKV = 0,        /* adaRMSNorm'd activations x [q|k|v] weights, RoPE epilogue */
  JPI_KERNEL_ATTENTION = 1,  /* prefix+self attention (chunk pass and combine) */
  JPI_KERNEL_OPROJ = 2,      /* attention output x W_o, gated residual */
  JPI_KERNEL_GATEUP = 3,     /* activations x [gate|up], GeGLU epilogue */
  JPI_KERNEL_DOWN = 4,       /* GeGLU output x W_down, gated residual */
  JPI_KERNEL_PERSISTENT = 5  /* the single-launch denoise kernel (batch*horizon <= 64, bf16) */
} jpi_kernel_kind;

/* Ask jpi_denoise to record a pair of HIP events around every launch of
 * `kind` (JPI_KERNEL_NONE switches it off).  While it is on, jpi_denoise
 * enqueues the same kernels directly on the stream instead of replaying the
 * captured graph (events recorded inside a graph cannot be timed). */
jpi_status jpi_debug_time_kernel(jpi_ctx* ctx, int kind);

/* After the stream of the last jpi_denoise has been synchronised: the sum of
 * the recorded launch durations (ms) and the number of launches. */
jpi_status jpi_debug_kernel_time(jpi_ctx* ctx, float* total_ms, int* launches);

#ifdef __cplusplus
}
#endif
#endif /* JPI_H_ */
