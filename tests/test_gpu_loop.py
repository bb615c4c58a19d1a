"""Algorithm 1 with every model on the GPU, at tiny shapes: the scheduling
loop drives the VLM prefill (+ compression), the correction module and the
action expert with the predicted item.  Every hook's output is checked
against the fp64 oracle given that hook's GPU inputs, so the test covers the
plumbing between the models: the prefix written in place, fresh state after
a refresh versus the hidden-state buffer otherwise, and the item bound into
the expert."""
import numpy as np
import pytest

import oracle
import synth
import synth.vlm as sv
from gpu_util import (BF16_ELEM, Corr, Vlm, bf16_bits_to_f64, elem_err_per_rollout, make_expert,
                      rel_l2_per_rollout, torch_cuda)
from oracle import correction as oc
from synth import correction as sc

pytestmark = pytest.mark.gpu

BF16_TOL = 2e-2


def test_schedule_loop_with_all_models_tiny():
    torch = torch_cuda()
    from paper_2607_12659_amd import jpi
    from paper_2607_12659_amd.expert import to_device
    vwl = sv.VLM_WORKLOADS["vlm-tiny"]
    awl = synth.WORKLOADS["tiny-fp32"].with_(dtype="bf16", name="tiny-bf16-loop")
    cwl = sc.CORR_WORKLOADS["corr-tiny"]
    cd = cwl.dims
    assert cd.width == awl.dims.width and cd.vlm_width == vwl.dims.width and cd.action_dim == awl.dims.action_dim
    print("case Algorithm 1 loop: vlm-tiny + corr-tiny + tiny bf16 expert", flush=True)
    vw = sv.make_vlm_weights(vwl)
    cw = sc.make_corr_weights(cwl, std=0.08)
    aw = synth.make_weights(awl)
    emb = sv.make_embeddings(vwl)
    noise = synth.make_noise(awl)
    vlm = Vlm(vwl.dims, vw, 1, vwl.prefix)
    corr = Corr(cd, cw, 1, awl.dims.horizon, vwl.prefix)
    ae = make_expert(awl, aw, max_batch=1, max_prefix=vwl.prefix, max_corr=cd.n_query)
    e_d = to_device(emb.astype(np.float32))
    n_d = to_device(noise.astype(np.float32))
    hidden = torch.empty((1, vwl.prefix, vwl.dims.width), dtype=torch.int16, device="cuda")
    item = torch.empty((1, cd.n_query, cd.width), device="cuda")   # the hidden-state buffer B_h
    chunk = torch.empty_like(n_d)
    forced = [1.0, -1.0, 1.0, 1.0, 1.0]
    log = []                          # (kind, inputs, outputs) on the host, in call order
    timeline, starts = {}, []         # the action buffer B_a on the absolute action index

    def host(t):
        return t.cpu().numpy()

    def vlm_hook(user, t, ms):
        vlm.prefill(e_d, 1, vwl.prefix, ae, hidden)
        st = jpi.jpi_corr_compress(corr.ctx, hidden, 1, vwl.prefix, item)   # B_h <- compressed h_t
        assert st == jpi.JPI_OK
        torch.cuda.synchronize()
        log.append(("vlm", host(hidden), host(item)))
        ms[0] = 1.0
        return 0

    def corr_hook(user, t, n, from_vlm, start, c, ms):
        n = max(1, min(n, awl.dims.horizon))
        src = host(item).copy()       # B_h: the fresh compression after a refresh, else the last item
        # a_t .. a_{t+n-1} from the action timeline (older chunks below `start`)
        assert start == starts[-1] and all(j in timeline for j in range(t, t + n))
        acts = np.stack([timeline[j] for j in range(t, t + n)])[None].astype(np.float32)
        corr.predict(item, to_device(acts), 1, n, item=item)
        torch.cuda.synchronize()
        log.append(("corr", (src, acts), host(item).copy()))
        c[0] = forced[sum(1 for k in log if k[0] == "corr") - 1]
        ms[0] = 0.1
        return 0

    def act_hook(user, t, have_corr, start, ms):
        ae.bind_state(None, 0, item if have_corr else None)
        ae.denoise(n_d, awl.n_steps, out=chunk)
        ae.sync()
        torch.cuda.synchronize()
        starts.append(start)
        for p, a in enumerate(host(chunk)[0]):
            timeline[start + p] = a
        log.append(("act", host(item).copy() if have_corr else None, host(chunk).copy()))
        ms[0] = 2.0
        return 0

    hooks = jpi.jpi_sched_hooks(jpi.SCHED_VLM_FN(vlm_hook), jpi.SCHED_CORR_FN(corr_hook), jpi.SCHED_ACT_FN(act_hook),
                                None)
    cfg = jpi.jpi_sched_config(theta=-0.5, delta=3, delta_ae=1, chunk_len=awl.dims.horizon, action_ms=1.0,
                               iterations=4)
    try:
        st, stats, ev = jpi.jpi_sched_run(cfg, hooks, 4)
        assert st == jpi.JPI_OK
    finally:
        ae.close()
        corr.close()
        vlm.close()
    assert [e.vlm for e in ev] == [0, 0, 1, 0] and stats.vlm_calls == 1
    assert [k[0] for k in log] == ["vlm", "act"] + ["corr", "act"] * 2 + ["vlm", "corr", "act", "corr", "act"]
    # the VLM output: the oracle prefill's KV (for the expert) and hidden state (for the compression)
    Kr, Vr, hid = oracle.vlm_prefill(vwl.dims, vw, emb[0])
    ex = oracle.Expert(awl.dims, aw)
    worst = {"vlm": 0.0, "corr": 0.0, "act": 0.0}
    worst_elem = dict(worst)

    def track(kind, got, ref):
        worst[kind] = max(worst[kind], rel_l2_per_rollout(got, ref))
        worst_elem[kind] = max(worst_elem[kind], elem_err_per_rollout(got, ref))

    for kind, inp, out in log:
        if kind == "vlm":
            got_hidden = bf16_bits_to_f64(inp)[0]
            track("vlm", got_hidden[None], hid[None])
            ref_c = oc.compress(cwl.dims, cw, inp[0].view(np.uint16))   # compression of the GPU's hidden state
            track("vlm", out.astype(np.float64), ref_c[None])
        elif kind == "corr":
            src, acts = inp
            ref_item, _ = oc.forward(cwl.dims, cw, acts.astype(np.float64), state=src.astype(np.float64))
            track("corr", out.astype(np.float64), ref_item)
        else:
            ref = oracle.denoise(ex, noise, Kr[:, None], Vr[:, None], [vwl.prefix], awl.n_steps,
                                 corr=None if inp is None else inp.astype(np.float64))
            track("act", out.astype(np.float64), ref)
    print("worst rel-L2 per hook kind: %s; element-wise %s" % ({k: "%.2e" % v for k, v in worst.items()},
                                                               {k: "%.2e" % v for k, v in worst_elem.items()}),
          flush=True)
    assert max(worst.values()) <= BF16_TOL
    assert max(worst_elem.values()) <= BF16_ELEM
