"""The scheduling loop of Algorithm 1 (confidence-based scheduling) on the
host, with simulated model latencies and forced confidence traces.

Pins: the branch rule and buffer updates of Algorithm 1 (first iteration skips
the VLM because the confidence starts at 0 > theta; each branch uses the
confidence of the previous correction call; committed actions are Delta_ae
without the VLM and Delta with it), action-accounting invariants, and the
reaction-time / control-frequency columns of the paper's latency table
(Table 'latency_breakdown', fixture tests/golden/latency_table.json): with the
VLM invoked on one iteration in seven, reaction = AE + (total - AE) / 7 lands
within 2% of every scheduled row, and control frequency = 1000 / reaction.
"""
import ctypes
import json
import math
import os

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _j():
    from paper_2607_12659_amd import jpi
    return jpi


def _run(conf, theta=-0.2, delta=9, delta_ae=3, chunk=50, action_ms=66.7, iters=700, vit=80.0, llm=210.0,
         corr=0.0, ae=120.0, trace=0):
    j = _j()
    arr = (ctypes.c_double * max(1, len(conf)))(*conf)
    sim = j.jpi_sched_sim(vit_ms=vit, llm_ms=llm, corr_ms=corr, ae_ms=ae, conf=arr, n_conf=len(conf))
    hooks = j.jpi_sched_hooks()
    assert j.jpi_sched_sim_hooks(sim, hooks) == j.JPI_OK
    cfg = j.jpi_sched_config(theta=theta, delta=delta, delta_ae=delta_ae, chunk_len=chunk, action_ms=action_ms,
                             iterations=iters)
    st, stats, ev = j.jpi_sched_run(cfg, hooks, trace)
    assert st == j.JPI_OK
    return stats, ev, sim, arr


def test_high_confidence_never_calls_the_vlm_after_start():
    stats, ev, sim, _ = _run([0.0], trace=20)
    assert stats.vlm_calls == 0 and sim.vlm_calls == 1          # only the initial observation
    assert all(e.vlm == 0 and e.n_committed == 3 for e in ev)   # Delta_ae committed actions each time
    assert stats.reaction_ms == pytest.approx(120.0)
    assert stats.startup_ms == pytest.approx(80.0 + 210.0 + 120.0)


def test_low_confidence_calls_the_vlm_from_the_second_iteration():
    stats, ev, sim, _ = _run([-1.0], iters=50, trace=50)
    assert ev[0].vlm == 0 and ev[0].conf_in == 0.0              # the confidence starts at 0 > theta
    assert all(e.vlm == 1 and e.n_committed == 9 for e in ev[1:])
    assert stats.vlm_calls == 49 and sim.vlm_calls == 50
    assert stats.reaction_ms == pytest.approx((120.0 + 49 * 410.0) / 50)


def test_branch_uses_the_previous_correction_confidence():
    conf = [0.5, -0.3, -0.1, -0.25, 0.0, -0.2, -0.21]
    _, ev, _, _ = _run(conf, iters=40, trace=40)
    for i in range(1, 40):
        assert ev[i].conf_in == ev[i - 1].conf_out
        assert ev[i].vlm == (not ev[i].conf_in > -0.2)         # strict: c == theta invokes the VLM
        assert ev[i].conf_out == conf[i % len(conf)]


def test_action_accounting():
    stats, ev, _, _ = _run([0.0] * 6 + [-1.0], iters=300, trace=300)
    ticks = math.floor(stats.total_ms / 66.7)
    assert stats.actions_executed + stats.actions_starved == ticks
    assert stats.actions_starved == 0                            # a 50-action chunk covers every latency here
    for a, b in zip(ev, ev[1:]):
        assert b.t == a.t + a.executed
    # a one-action chunk cannot cover a 120 ms expert call at 66.7 ms per action
    st2, _, _, _ = _run([0.0], chunk=1, iters=100, delta_ae=1, delta=1)
    assert st2.actions_starved > 0


def _table():
    with open(os.path.join(ROOT, "tests", "golden", "latency_table.json")) as f:
        return json.load(f)


def test_latency_table_columns_are_consistent():
    for dev, rows in _table()["devices"].items():
        for name, vit, llm, ae, total, reaction, hz in rows:
            assert 1000.0 / reaction == pytest.approx(hz, abs=0.01), (dev, name)
            if not (dev == "Jetson Orin" and name in ("Naive PI05", "+Schedule opt.")):
                assert vit + llm + ae == pytest.approx(total, abs=0.051), (dev, name)


@pytest.mark.parametrize("dev", ["Jetson Orin", "Jetson Thor"])
def test_reaction_time_matches_the_latency_table(dev):
    rows = _table()["devices"][dev]
    naive = rows[0]
    # no scheduling: the VLM runs every iteration (threshold above any confidence)
    stats, _, _, _ = _run([0.0], theta=1e30, vit=naive[1], llm=naive[4] - naive[1] - naive[3], ae=naive[3], iters=100)
    assert stats.reaction_ms == pytest.approx(naive[5], rel=1e-9)
    assert stats.control_hz == pytest.approx(naive[6], abs=0.01)
    for name, vit, llm, ae, total, reaction, hz in rows[1:]:
        # one low-confidence correction call in seven
        stats, _, _, _ = _run([0.0] * 6 + [-1.0], vit=vit, llm=total - vit - ae, ae=ae, iters=7001)
        assert stats.vlm_fraction == pytest.approx(1 / 7, abs=1e-3)
        assert stats.reaction_ms == pytest.approx(reaction, rel=0.02), (dev, name)
        assert stats.control_hz == pytest.approx(1000.0 / stats.reaction_ms)


def test_rejects_bad_arguments():
    j = _j()
    hooks = j.jpi_sched_hooks()
    sim = j.jpi_sched_sim()
    assert j.jpi_sched_sim_hooks(sim, hooks) == j.JPI_OK
    good = dict(theta=-0.2, delta=9, delta_ae=3, chunk_len=50, action_ms=66.7, iterations=10)
    for bad in (dict(delta=2), dict(delta_ae=-1), dict(chunk_len=0), dict(action_ms=0.0), dict(iterations=0)):
        cfg = j.jpi_sched_config(**{**good, **bad})
        st, _, _ = j.jpi_sched_run(cfg, hooks, 0)
        assert st == j.JPI_ERR_ARG, bad
    st, _, _ = j.jpi_sched_run(j.jpi_sched_config(**good), j.jpi_sched_hooks(), 0)   # hooks missing
    assert st == j.JPI_ERR_ARG


def test_python_hooks_drive_the_same_loop():
    j = _j()
    calls = []

    def vlm(user, t, ms):
        calls.append(("vlm", t))
        ms[0] = 300.0
        return 0

    def corr(user, t, n, from_vlm, start, conf, ms):
        calls.append(("corr", t, n, from_vlm))
        conf[0] = -1.0 if len(calls) % 5 == 0 else 0.0
        ms[0] = 2.0
        return 0

    def act(user, t, have_corr, start, ms):
        calls.append(("act", t, have_corr))
        ms[0] = 100.0
        return 0

    hooks = j.jpi_sched_hooks(j.SCHED_VLM_FN(vlm), j.SCHED_CORR_FN(corr), j.SCHED_ACT_FN(act), None)
    cfg = j.jpi_sched_config(theta=-0.2, delta=6, delta_ae=2, chunk_len=50, action_ms=50.0, iterations=12)
    st, stats, ev = j.jpi_sched_run(cfg, hooks, 12)
    assert st == j.JPI_OK
    assert calls[0] == ("vlm", 0) and calls[1] == ("act", 0, 0)
    for e in ev:
        assert e.ms == pytest.approx(102.0 + (300.0 if e.vlm else 0.0))
    # a failing hook stops the loop
    hooks2 = j.jpi_sched_hooks(j.SCHED_VLM_FN(vlm), j.SCHED_CORR_FN(corr), j.SCHED_ACT_FN(lambda u, t, h, c, ms: 1),
                               None)
    st, _, _ = j.jpi_sched_run(cfg, hooks2, 0)
    assert st == j.JPI_ERR_STATE


@pytest.mark.parametrize("model_ms", [12.0, 37.0, 260.0])
def test_hooks_get_the_committed_actions_from_the_timeline(model_ms):
    """Chunks are placed on the absolute action timeline: act(t, .., start)
    writes actions [start, start + chunk_len), and corr(t, n, .., start) must
    find a_t .. a_{t+n-1} there -- from the latest chunk where j >= start,
    from an older one below it (a loop faster than the robot runs ahead of
    the execution, so t < start happens).  Checked for a fast, a medium and a
    slow model against a 20 ms control period."""
    j = _j()
    chunk = 10
    timeline = {}        # action index -> (chunk id, position in the chunk)
    starts, seen = [], {"behind": 0, "ahead": 0}

    def vlm(user, t, ms):
        ms[0] = model_ms
        return 0

    def corr(user, t, n, from_vlm, start, conf, ms):
        assert start == starts[-1]                        # the latest chunk
        for a in range(t, t + n):
            cid, pos = timeline[a]                        # every committed action exists
            if a >= start:
                assert cid == len(starts) - 1 and pos == a - start
            else:
                assert cid < len(starts) - 1
        seen["behind" if t < start else "ahead"] += 1
        conf[0] = 1.0
        ms[0] = model_ms
        return 0

    def act(user, t, have_corr, start, ms):
        if not starts:
            assert (t, have_corr, start) == (0, 0, 0)
        else:
            assert start >= t
        starts.append(start)
        for p in range(chunk):
            timeline[start + p] = (len(starts) - 1, p)
        ms[0] = model_ms
        return 0

    hooks = j.jpi_sched_hooks(j.SCHED_VLM_FN(vlm), j.SCHED_CORR_FN(corr), j.SCHED_ACT_FN(act), None)
    cfg = j.jpi_sched_config(theta=-0.5, delta=4, delta_ae=4, chunk_len=chunk, action_ms=20.0, iterations=40)
    st, stats, ev = j.jpi_sched_run(cfg, hooks, 40)
    assert st == j.JPI_OK
    assert [e.t + e.n_committed for e in ev] == starts[1:]
    if model_ms < 20.0 * 4 / 2:
        assert seen["behind"] > 0        # the loop ran ahead of the robot
