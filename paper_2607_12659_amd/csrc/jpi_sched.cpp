// Confidence-based scheduling of asynchronous VLA inference: the host loop
// of Algorithm 1 (Appendix "Algorithm Details of Confidence-based Scheduling
// Optimization") over caller hooks for the VLM, the future correction module
// and the action expert, with the execution of the action buffer simulated on
// a clock.  Host code only.
#include <math.h>
#include <stddef.h>

#include "../../include/jpi_sched.h"

namespace {

// Actions the robot executes from the buffer while `ms` elapse.  `clock` is
// the time since the loop started, `ticks` the whole action periods in it
// so far; the buffer holds actions up to (not including) `end`, and the robot
// pauses at the end of the buffer until a new chunk arrives.
void execute(double ms, double action_ms, double* clock, int64_t* ticks, int64_t* t, int64_t end,
             int64_t* executed, int64_t* starved) {
  *clock += ms;
  const int64_t now = (int64_t)floor(*clock / action_ms);
  const int64_t n = now - *ticks;
  *ticks = now;
  const int64_t room = end > *t ? end - *t : 0;
  *executed = n < room ? n : room;
  *starved = n - *executed;
  *t += *executed;
}

int sim_vlm(void* user, int64_t, double* ms) {
  jpi_sched_sim* s = static_cast<jpi_sched_sim*>(user);
  ++s->vlm_calls;
  *ms = s->vit_ms + s->llm_ms;
  return 0;
}

int sim_corr(void* user, int64_t, int, int, int64_t, double* conf, double* ms) {
  jpi_sched_sim* s = static_cast<jpi_sched_sim*>(user);
  *conf = s->n_conf > 0 ? s->conf[s->corr_calls % s->n_conf] : 0.0;
  ++s->corr_calls;
  *ms = s->corr_ms;
  return 0;
}

int sim_act(void* user, int64_t, int, int64_t, double* ms) {
  jpi_sched_sim* s = static_cast<jpi_sched_sim*>(user);
  ++s->act_calls;
  *ms = s->ae_ms;
  return 0;
}

}  // namespace

extern "C" {

jpi_status jpi_sched_run(const jpi_sched_config* cfg, const jpi_sched_hooks* hooks, jpi_sched_stats* stats,
                         jpi_sched_event* trace, int64_t trace_cap) {
  if (!cfg || !hooks || !stats || !hooks->vlm || !hooks->corr || !hooks->act) return JPI_ERR_ARG;
  if (cfg->delta_ae < 0 || cfg->delta < cfg->delta_ae || cfg->chunk_len < 1 || !(cfg->action_ms > 0.0) ||
      cfg->iterations < 1 || (trace_cap > 0 && !trace))
    return JPI_ERR_ARG;
  jpi_sched_stats st = {};

  // B_kv, B_h <- f_vlm(o_0, l); B_a <- f_act(h_0, KV_0).  The robot has no
  // actions yet, so nothing executes during this.
  double ms_vlm = 0.0, ms_act = 0.0;
  if (hooks->vlm(hooks->user, 0, &ms_vlm) != 0) return JPI_ERR_STATE;
  if (hooks->act(hooks->user, 0, 0, 0, &ms_act) != 0) return JPI_ERR_STATE;
  st.startup_ms = ms_vlm + ms_act;

  double conf = 0.0;  // above any threshold theta < 0: the first iteration skips the VLM
  double clock = 0.0;
  int64_t ticks = 0, t = 0, buf_end = cfg->chunk_len;
  for (int64_t it = 0; it < cfg->iterations; ++it) {
    jpi_sched_event ev = {};
    ev.t = t;
    ev.conf_in = conf;
    ev.vlm = !(conf > cfg->theta);
    double ms = 0.0, part = 0.0;
    if (ev.vlm) {
      // observe now, refresh B_kv; predict Delta actions ahead from h_t
      if (hooks->vlm(hooks->user, t, &part) != 0) return JPI_ERR_STATE;
      ms += part;
      ev.n_committed = cfg->delta;
    } else {
      // predict Delta_ae actions ahead from the hidden-state buffer B_h
      ev.n_committed = cfg->delta_ae;
    }
    // a_t .. a_{t+n-1}: the latest chunk starts at buf_end - chunk_len
    if (hooks->corr(hooks->user, t, ev.n_committed, ev.vlm, buf_end - cfg->chunk_len, &conf, &part) != 0)
      return JPI_ERR_STATE;
    ms += part;
    if (hooks->act(hooks->user, t, 1, ev.t + ev.n_committed, &part) != 0) return JPI_ERR_STATE;
    ms += part;
    ev.conf_out = conf;
    ev.ms = ms;
    // the committed actions (and any after them still in the old chunk) run
    // while the models work; the new chunk starts after the committed ones
    execute(ms, cfg->action_ms, &clock, &ticks, &t, buf_end, &ev.executed, &ev.starved);
    buf_end = ev.t + ev.n_committed + cfg->chunk_len;
    if (it < trace_cap) trace[it] = ev;
    st.iterations += 1;
    st.vlm_calls += ev.vlm;
    st.total_ms += ms;
    st.actions_executed += ev.executed;
    st.actions_starved += ev.starved;
  }
  st.reaction_ms = st.total_ms / (double)st.iterations;
  st.control_hz = st.reaction_ms > 0.0 ? 1000.0 / st.reaction_ms : 0.0;
  st.vlm_fraction = (double)st.vlm_calls / (double)st.iterations;
  *stats = st;
  return JPI_OK;
}

jpi_status jpi_sched_sim_hooks(jpi_sched_sim* sim, jpi_sched_hooks* hooks) {
  if (!sim || !hooks || (sim->n_conf > 0 && !sim->conf) || sim->n_conf < 0) return JPI_ERR_ARG;
  sim->corr_calls = sim->vlm_calls = sim->act_calls = 0;
  hooks->vlm = sim_vlm;
  hooks->corr = sim_corr;
  hooks->act = sim_act;
  hooks->user = sim;
  return JPI_OK;
}

}  // extern "C"
