/* libjpi scheduler: confidence-based scheduling of asynchronous VLA inference.
 *
 * The host loop of Algorithm 1 (Appendix "Algorithm Details of
 * Confidence-based Scheduling Optimization"; Section "Confidence-based
 * Scheduling Optimization").  The robot executes actions from the action
 * buffer B_a continuously while the loop predicts the next chunk.  Each
 * iteration either skips the VLM (confidence above the threshold: the future
 * correction module predicts the VLM state Delta_ae actions ahead from its
 * own previous prediction) or refreshes the environment (the VLM observes
 * now, and the correction module predicts Delta actions ahead from that
 * observation); either way the action expert then predicts a new chunk.
 *
 * The three models are caller hooks, so the same loop drives simulated
 * latencies (jpi_sched_sim_hooks) or real kernels (for instance an action
 * expert hook that calls jpi_denoise and times it).  Host code only: no call
 * touches a GPU unless a hook does.
 *
 * Conventions: every call returns a jpi_status (include/jpi.h); nothing
 * throws.  Times are milliseconds (double).  A hook returns 0 on success;
 * any other value stops the loop with JPI_ERR_STATE.
 */
#ifndef JPI_SCHED_H_
#define JPI_SCHED_H_

#include <stdint.h>

#include "jpi.h"

#ifdef __cplusplus
extern "C" {
#endif

typedef struct {
  double theta;        /* confidence threshold theta: the VLM is skipped while the last
                          confidence is > theta (the paper uses theta < 0) */
  int delta;           /* Delta: latency of the whole VLA in executed actions; the
                          actions committed while the VLM, correction and expert run */
  int delta_ae;        /* Delta_ae: the same for the correction module + action expert */
  int chunk_len;       /* actions per predicted chunk (the action buffer's size) */
  double action_ms;    /* execution time of one action (the robot's control period) */
  int64_t iterations;  /* iterations of the loop to run (>= 1) */
} jpi_sched_config;

/* Model hooks.  Each reports the time it took (measured or simulated) in *ms.
 * Action indices are absolute: action j is the j-th action the robot
 * executes.  Chunks are placed on that timeline: the chunk predicted by the
 * iteration that starts at action t, with n_committed actions committed to
 * its prediction, covers actions [t + n_committed, t + n_committed +
 * chunk_len) and replaces whatever an older chunk held there; the first
 * chunk (before the loop) covers [0, chunk_len).
 *   vlm(t):  observe at action index t and run the VLM (refreshes the prefix
 *            KV buffer B_kv and the hidden state h_t); also called once at start.
 *   corr(t, n_committed, from_vlm, chunk_start): predict the compressed VLM
 *            state n_committed actions ahead from h_t (from_vlm = 1) or from the
 *            hidden-state buffer B_h (from_vlm = 0), given the committed actions
 *            a_t .. a_{t+n_committed-1} (Algorithm 1).  chunk_start is the
 *            first action index of the latest chunk: a_j is that chunk's action
 *            j - chunk_start when j >= chunk_start and an older chunk's action
 *            otherwise (the loop can run ahead of the robot, so t may be below
 *            chunk_start).  Writes its confidence to *conf.
 *   act(t, have_corr, chunk_start): the action expert predicts the chunk that
 *            starts at action index chunk_start, from the prediction
 *            (have_corr = 1) or, at start, from h_0 (have_corr = 0, t = 0,
 *            chunk_start = 0). */
typedef struct {
  int (*vlm)(void* user, int64_t t, double* ms);
  int (*corr)(void* user, int64_t t, int n_committed, int from_vlm, int64_t chunk_start, double* conf, double* ms);
  int (*act)(void* user, int64_t t, int have_corr, int64_t chunk_start, double* ms);
  void* user;
} jpi_sched_hooks;

/* One loop iteration. */
typedef struct {
  int64_t t;           /* action index when the iteration started */
  int vlm;             /* 1 if the VLM ran (confidence was <= theta) */
  int n_committed;     /* actions handed to the correction module (delta or delta_ae) */
  double conf_in;      /* confidence that chose the branch */
  double conf_out;     /* confidence returned by the correction module */
  double ms;           /* wall time of the iteration (sum of its hooks): its reaction time */
  int64_t executed;    /* actions executed while it ran */
  int64_t starved;     /* of those, actions the buffer did not hold (the robot paused) */
} jpi_sched_event;

typedef struct {
  int64_t iterations, vlm_calls;   /* vlm_calls counts loop iterations that ran the VLM */
  double startup_ms;               /* initial VLM + action expert (before the loop) */
  double total_ms;                 /* loop time, startup excluded */
  double reaction_ms;              /* mean iteration time: from an observation (or a
                                      prediction of it) to the chunk that reacts to it */
  double control_hz;               /* new chunks per second: 1000 / reaction_ms */
  double vlm_fraction;             /* vlm_calls / iterations */
  int64_t actions_executed, actions_starved;
} jpi_sched_stats;

/* Run Algorithm 1 for cfg->iterations iterations.  trace (may be NULL) gets
 * the first trace_cap events.  Errors: JPI_ERR_ARG (NULL cfg/hooks/stats or a
 * missing hook, delta_ae < 0, delta < delta_ae, chunk_len < 1, action_ms <= 0,
 * iterations < 1), JPI_ERR_STATE (a hook failed). */
jpi_status jpi_sched_run(const jpi_sched_config* cfg, const jpi_sched_hooks* hooks, jpi_sched_stats* stats,
                         jpi_sched_event* trace, int64_t trace_cap);

/* Simulated models for the loop: fixed latencies per component and a forced
 * confidence trace (the correction module's i-th call returns conf[i % n_conf]).
 * The state must outlive the run; jpi_sched_sim_hooks fills hooks to use it. */
typedef struct {
  double vit_ms, llm_ms;   /* the VLM hook takes vit_ms + llm_ms */
  double corr_ms, ae_ms;   /* correction module, action expert */
  const double* conf;      /* forced confidences (caller-owned) */
  int64_t n_conf;
  int64_t corr_calls;      /* updated by the hooks */
  int64_t vlm_calls, act_calls;
} jpi_sched_sim;

jpi_status jpi_sched_sim_hooks(jpi_sched_sim* sim, jpi_sched_hooks* hooks);

#ifdef __cplusplus
}
#endif

#endif /* JPI_SCHED_H_ */
