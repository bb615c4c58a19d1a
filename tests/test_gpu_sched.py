"""Algorithm 1's loop driving the real action expert on the GPU.

The action-expert hook runs jpi_denoise (pi0.5 shape, batch 1) and reports
its time from HIP events; the VLM hook re-binds the prefix KV (the hand-off a
VLM refresh makes) and the correction hook replays a forced confidence trace.
Checks: every chunk the loop produced equals the stored oracle output for
these inputs (within the bf16 bar), and the loop's reaction time is the
measured expert time plus the measured prefix hand-offs it made.
"""
import ctypes

import numpy as np
import pytest

import synth
from gpu_util import assert_bf16, load_golden, make_expert, rel_l2_per_rollout, torch_cuda

pytestmark = pytest.mark.gpu


def test_schedule_loop_with_the_gpu_action_expert():
    torch = torch_cuda()
    from paper_2607_12659_amd import jpi
    from paper_2607_12659_amd.expert import to_device
    wl = synth.WORKLOADS["pi05-b1"]
    print("case scheduler + pi05-b1 expert", flush=True)
    ae = make_expert(wl, synth.make_weights(wl), max_batch=1, max_prefix=816)
    try:
        K, V = synth.make_prefix(wl)
        kd, vd = to_device(K), to_device(V)
        noise = to_device(np.ascontiguousarray(synth.make_noise(wl), np.float32))
        ref, _ = load_golden("pi05-b1")
        conf = [0.0, 0.0, -1.0]
        outs, t_act, t_vlm = [], [], []

        def timed(fn):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            torch.cuda.synchronize()
            e0.record()
            r = fn()
            e1.record()
            torch.cuda.synchronize()
            return r, e0.elapsed_time(e1)

        def vlm(user, t, ms):
            _, dt = timed(lambda: ae.bind_prefix(kd, vd, None))
            t_vlm.append(dt)
            ms[0] = dt
            return 0

        def corr(user, t, n, from_vlm, start, c, ms):
            c[0] = conf[len(outs) % len(conf)]
            ms[0] = 0.0
            return 0

        def act(user, t, have_corr, start, ms):
            out, dt = timed(lambda: ae.denoise(noise, wl.n_steps))
            ae.sync()   # the single-launch kernel's status: a timed-out wait invalidates the chunk
            outs.append(out.cpu().numpy().astype(np.float64))
            t_act.append(dt)
            ms[0] = dt
            return 0

        hooks = jpi.jpi_sched_hooks(jpi.SCHED_VLM_FN(vlm), jpi.SCHED_CORR_FN(corr), jpi.SCHED_ACT_FN(act), None)
        cfg = jpi.jpi_sched_config(theta=-0.2, delta=3, delta_ae=1, chunk_len=wl.dims.horizon, action_ms=66.7,
                                   iterations=9)
        st, stats, ev = jpi.jpi_sched_run(cfg, hooks, 9)
        assert st == jpi.JPI_OK
        assert len(outs) == 10                          # the initial chunk + one per iteration
        for o in outs:
            assert_bf16(o, ref, reg_rel=2e-3, reg_abs=1e-2)
        assert stats.vlm_calls == sum(e.vlm for e in ev) and stats.vlm_calls >= 2
        loop_act = sum(t_act[1:])
        loop_vlm = sum(t_vlm[1:])
        assert stats.total_ms == pytest.approx(loop_act + loop_vlm, rel=1e-9)
        print("scheduler: %d iterations, %d VLM refreshes, reaction %.2f ms (expert %.2f ms per chunk)"
              % (stats.iterations, stats.vlm_calls, stats.reaction_ms, loop_act / 9), flush=True)
    finally:
        ae.close()
