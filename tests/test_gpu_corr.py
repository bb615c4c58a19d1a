"""The correction item in the action expert (jpi_bind_state with correction
tokens) and the future correction module (include/jpi_corr.h) against the
fp64 oracle.  Same bars as the denoise parity: fp32 max-abs <= 1e-4, bf16
per-rollout relative L2 <= 2e-2."""
import numpy as np
import pytest

import oracle
import synth
from gpu_util import assert_bf16, load_golden, make_expert, rel_l2_per_rollout, run, run_env, torch_cuda
from oracle import correction as oc
from synth import correction as sc

pytestmark = pytest.mark.gpu

BF16_TOL = 2e-2
F32_TOL = 1e-4


def _inputs(wl, n_corr, lens):
    w = synth.make_weights(wl)
    K, V = synth.make_prefix(wl)
    noise = synth.make_noise(wl)
    corr = sc.make_item(wl.seed, wl.batch, n_corr, wl.dims.width)
    return w, K, V, noise, corr


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_tiny_expert_with_correction_tokens(dtype):
    torch_cuda()
    wl = synth.WORKLOADS["tiny-fp32"].with_(dtype=dtype, batch=3, n_fixed=2, name="tiny-corr")
    lens = [wl.prefix, 5, 0]
    print("case tiny expert + 4 correction tokens, %s, prefix_len %s" % (dtype, lens), flush=True)
    w, K, V, noise, corr = _inputs(wl, 4, lens)
    com = synth.make_committed(wl)
    ae = make_expert(wl, w, max_batch=4, max_prefix=wl.prefix, max_corr=6)
    try:
        got = run(ae, K, V, noise, wl.n_steps, prefix_len=lens, committed=com, n_fixed=2, corr=corr)
        ref = oracle.denoise(oracle.Expert(wl.dims, w), noise, K, V, lens, wl.n_steps, committed=com, n_fixed=2,
                             corr=corr)
        err = np.abs(got - ref).max()
        rel = rel_l2_per_rollout(got, ref)
        print("max-abs %.3e rel-L2 %.3e" % (err, rel), flush=True)
        if dtype == "f32":
            assert err <= F32_TOL
        else:
            assert_bf16(got, ref, "tiny bf16 with correction tokens")
        assert np.array_equal(got[:, :2].astype(np.float32), com)
        # the tokens matter, and unbinding them gives the expert without them
        plain = run(ae, K, V, noise, wl.n_steps, prefix_len=lens, committed=com, n_fixed=2)
        ref0 = oracle.denoise(oracle.Expert(wl.dims, w), noise, K, V, lens, wl.n_steps, committed=com, n_fixed=2)
        assert np.abs(ref - ref0).max() > 50 * max(err, 1e-6)
        if dtype == "f32":
            assert np.abs(plain - ref0).max() <= F32_TOL
        # a different token count on the same context (new graph, new RoPE rows)
        got1 = run(ae, K, V, noise, wl.n_steps, prefix_len=lens, committed=com, n_fixed=2, corr=corr[:, :1])
        ref1 = oracle.denoise(oracle.Expert(wl.dims, w), noise, K, V, lens, wl.n_steps, committed=com, n_fixed=2,
                              corr=corr[:, :1])
        if dtype == "f32":
            assert np.abs(got1 - ref1).max() <= F32_TOL
        else:
            assert_bf16(got1, ref1, "tiny bf16 with one correction token")
    finally:
        ae.close()


def test_tiny_expert_rejects_too_many_correction_tokens():
    torch = torch_cuda()
    from paper_2607_12659_amd import jpi
    from paper_2607_12659_amd.expert import to_device
    wl = synth.WORKLOADS["tiny-fp32"]
    w, K, V, noise, corr = _inputs(wl, 3, None)
    ae = make_expert(wl, w, max_corr=2)
    try:
        ae.bind_prefix(to_device(K), to_device(V))
        c = to_device(corr.astype(np.float32))
        assert jpi.jpi_bind_state(ae.ctx, None, 0, c, 3, None) == jpi.JPI_ERR_ARG
        assert jpi.jpi_bind_state(ae.ctx, None, 0, None, 2, None) == jpi.JPI_ERR_ARG
        assert jpi.jpi_bind_state(ae.ctx, None, 0, c, 2, None) == jpi.JPI_OK
        torch.cuda.synchronize()
    finally:
        ae.close()


def test_pi05_committed10_with_correction_item():
    """The pi0.5 expert at full size with the 4-token correction item and the
    10 committed rows of one scheduler iteration (54 suffix rows: the
    single-launch kernel), against the stored oracle output and the
    multi-kernel path; the call without the item is unchanged after."""
    torch_cuda()
    wl = synth.WORKLOADS["pi05-b1-committed10"]
    print("case pi05-b1-committed10-corr4", flush=True)
    w = synth.make_weights(wl)
    K, V = synth.make_prefix(wl)
    noise = synth.make_noise(wl)
    com = synth.make_committed(wl)
    corr = sc.make_item(wl.seed, 1, 4, wl.dims.width)
    ae = make_expert(wl, w, max_batch=1, max_prefix=816, max_corr=4)
    try:
        before = run(ae, K, V, noise, wl.n_steps, committed=com, n_fixed=10)
        got = run(ae, K, V, noise, wl.n_steps, committed=com, n_fixed=10, corr=corr)
        multi = run_env(ae, "0", K, V, noise, wl.n_steps, committed=com, n_fixed=10, corr=corr)
        ref, meta = load_golden("pi05-b1-committed10-corr4")
        assert meta["n_corr"] == 4
        plain, _ = load_golden("pi05-b1-committed10")
        effect = rel_l2_per_rollout(plain, ref)
        for label, out in (("single-launch", got), ("multi-kernel", multi)):
            rel = rel_l2_per_rollout(out, ref)
            print("%s: rel-L2 %.3e max-abs %.3e; the item moves the actions by %.3e"
                  % (label, rel, np.abs(out - ref).max(), effect), flush=True)
            assert_bf16(out, ref, label, reg_rel=2e-3, reg_abs=1e-2)
            assert effect > 10 * rel
            assert np.array_equal(out[:, :10].astype(np.float32), com)
        assert np.array_equal(got, run(ae, K, V, noise, wl.n_steps, committed=com, n_fixed=10, corr=corr))
        after = run(ae, K, V, noise, wl.n_steps, committed=com, n_fixed=10)
        assert np.array_equal(before, after)
    finally:
        ae.close()


def test_persistent_tiny_bf16_correction_rows_batched():
    """Two rollouts of 4 correction + horizon action rows in the single-launch
    kernel (ragged prefixes, committed rows) against the oracle and the
    multi-kernel path, and bitwise repeatable."""
    torch_cuda()
    wl = synth.WORKLOADS["tiny-fp32"].with_(dtype="bf16", batch=2, n_fixed=2, name="tiny-bf16-corr-b2")
    lens = [wl.prefix, 17]
    assert 2 * (wl.dims.horizon + 4) <= 64
    print("case tiny bf16 b2 + 4 correction rows, single-launch, prefix_len %s" % lens, flush=True)
    w, K, V, noise, corr = _inputs(wl, 4, lens)
    com = synth.make_committed(wl)
    ae = make_expert(wl, w, max_batch=2, max_prefix=wl.prefix, max_corr=4)
    try:
        kw = dict(prefix_len=lens, committed=com, n_fixed=2, corr=corr)
        got = run_env(ae, None, K, V, noise, wl.n_steps, **kw)
        multi = run_env(ae, "0", K, V, noise, wl.n_steps, **kw)
        again = run_env(ae, None, K, V, noise, wl.n_steps, **kw)
    finally:
        ae.close()
    ref = oracle.denoise(oracle.Expert(wl.dims, w), noise, K, V, lens, wl.n_steps, committed=com, n_fixed=2,
                         corr=corr)
    rel = rel_l2_per_rollout(got, ref)
    print("single-launch rel-L2 %.3e, vs multi-kernel %.3e" % (rel, rel_l2_per_rollout(got, multi)), flush=True)
    assert_bf16(got, ref, "single-launch")
    assert rel_l2_per_rollout(got, multi) <= 5e-3
    assert np.array_equal(got, again)
    assert np.array_equal(got[:, :2].astype(np.float32), com)


# ---------------------------------------------------------------------------
# the future correction module
# ---------------------------------------------------------------------------
def _conf_bound(w, y_mean):
    """Error allowed on a confidence: the bf16 bar applied to every term of
    its dot product, sum_k |w_conf[k] * mean_j y[j][k]| * 2e-2."""
    return BF16_TOL * float(np.abs(oracle.widen(w["conf_head.w"])[0] * y_mean).sum())


def _oracle_heads_input(d, w, state, acts):
    """mean_j of the final-normalised tokens (the confidence head's input), per rollout."""
    ww = {k: oracle.widen(v) for k, v in w.items()}
    out = []
    for b in range(len(acts)):
        s = oc.action_summary(d, w, acts[b])
        cat = np.concatenate([state[b], np.broadcast_to(s, state[b].shape)], axis=1)
        z = cat @ ww["fuse.w"].T + ww["fuse.b"]
        for p in ("blocks.0.", "blocks.1."):
            z = oc.block(ww, p, d.n_heads, z)
        y = oracle.rms_normalize(z) * (1.0 + ww["final_norm.w"])
        out.append(y.mean(axis=0))
    return out



def _check_corr(d, w, state_ref, acts, item, conf, label):
    ref_item, ref_conf = oc.forward(d, w, acts, state=state_ref)
    rel = rel_l2_per_rollout(item, ref_item)
    ym = _oracle_heads_input(d, w, state_ref, acts)
    dconf = [abs(conf[b] - ref_conf[b]) for b in range(len(acts))]
    bounds = [_conf_bound(w, ym[b]) for b in range(len(acts))]
    print("%s: item rel-L2 %.3e max-abs %.3e; confidence err %s bound %s" %
          (label, rel, np.abs(item - ref_item).max(), ["%.2e" % x for x in dconf], ["%.2e" % x for x in bounds]),
          flush=True)
    assert_bf16(item, ref_item, label + " item")
    assert all(dc <= bd for dc, bd in zip(dconf, bounds))
    return ref_item, ref_conf


def _corr_case(name, std):
    wl = sc.CORR_WORKLOADS[name]
    w = sc.make_corr_weights(wl, std=std)
    return wl, w, sc.make_vlm_state(wl), sc.make_actions(wl), sc.make_state(wl)


@pytest.mark.parametrize("name,std", [("corr-tiny", 0.08), ("corr40m-p816", 0.02)])
def test_correction_module_matches_oracle(name, std):
    torch = torch_cuda()
    from paper_2607_12659_amd.expert import to_device
    from gpu_util import Corr
    wl, w, vs, acts, state = _corr_case(name, std)
    d = wl.dims
    print("case %s: batch %d, %d actions, %d VLM tokens" % (name, wl.batch, wl.n_actions, wl.vlm_tokens), flush=True)
    m = Corr(d, w, max_batch=wl.batch + 1, max_actions=wl.n_actions + 2, max_vlm_tokens=wl.vlm_tokens + 9)
    try:
        # VLM refresh: compress the fresh state, then predict from it
        c = m.compress(to_device(vs), wl.batch, wl.vlm_tokens)
        acts_d = to_device(acts.astype(np.float32))
        item, conf = m.predict(c, acts_d, wl.batch, wl.n_actions)
        torch.cuda.synchronize()
        c_ref = np.stack([oc.compress(d, w, vs[b]) for b in range(wl.batch)])
        c_got = c.cpu().numpy().astype(np.float64)
        rel_c = rel_l2_per_rollout(c_got, c_ref)
        print("compressed state rel-L2 %.3e" % rel_c, flush=True)
        assert_bf16(c_got, c_ref, name + " compressed state")
        # the item is checked against the oracle run on the oracle's own state
        ref_item, _ = _check_corr(d, w, c_ref, acts, item.cpu().numpy().astype(np.float64),
                                  conf.cpu().numpy().astype(np.float64), name + " refresh")
        # VLM skipped: predict from the hidden-state buffer, in place
        st = to_device(state.astype(np.float32))
        item2, conf2 = m.predict(st, acts_d, wl.batch, wl.n_actions, item=st)
        torch.cuda.synchronize()
        _check_corr(d, w, state, acts, item2.cpu().numpy().astype(np.float64), conf2.cpu().numpy().astype(np.float64),
                    name + " from state (in place)")
        # fewer actions (Delta_ae < Delta) on the same module
        k = max(1, wl.n_actions - 3)
        st = to_device(state.astype(np.float32))
        item3, conf3 = m.predict(st, to_device(np.ascontiguousarray(acts[:, :k]).astype(np.float32)), wl.batch, k)
        torch.cuda.synchronize()
        _check_corr(d, w, state, acts[:, :k], item3.cpu().numpy().astype(np.float64),
                    conf3.cpu().numpy().astype(np.float64), name + " %d actions" % k)
        # sensitivity: the committed actions move the item far more than the GPU error
        got = item.cpu().numpy().astype(np.float64)
        moved, _ = oc.forward(d, w, acts * -1.0, state=c_ref)
        effect = rel_l2_per_rollout(moved, ref_item)
        err = rel_l2_per_rollout(got, ref_item)
        print("sensitivity: negated actions move the item by %.3e, GPU error %.3e" % (effect, err), flush=True)
        assert effect > 5 * err
    finally:
        m.close()


def test_correction_item_into_the_expert():
    """Algorithm 1's skip branch on the device, zero-copy: the module's item
    goes straight into jpi_bind_state and the expert denoises with it."""
    torch = torch_cuda()
    from paper_2607_12659_amd.expert import to_device
    from gpu_util import Corr
    cwl, w, vs, acts, state = _corr_case("corr-tiny", 0.08)
    awl = synth.WORKLOADS["tiny-fp32"].with_(dtype="bf16", batch=2, n_fixed=3, name="tiny-bf16-corr")
    assert awl.dims.width == cwl.dims.width
    print("case corr-tiny item -> tiny bf16 expert", flush=True)
    aw = synth.make_weights(awl)
    K, V = synth.make_prefix(awl)
    noise = synth.make_noise(awl)
    com = synth.make_committed(awl)
    m = Corr(cwl.dims, w, max_batch=2, max_actions=8, max_vlm_tokens=64)
    ae = make_expert(awl, aw, max_corr=cwl.dims.n_query)
    try:
        st = to_device(state.astype(np.float32))
        item, conf = m.predict(st, to_device(acts.astype(np.float32)), 2, cwl.n_actions)
        ae.bind_prefix(to_device(K), to_device(V))
        ae.bind_state(to_device(com.astype(np.float32)), 3, item)
        out = ae.denoise(to_device(noise.astype(np.float32)), awl.n_steps)
        ae.sync()
        got = out.cpu().numpy().astype(np.float64)
        ref_item, _ = oc.forward(cwl.dims, w, acts, state=state)
        ref = oracle.denoise(oracle.Expert(awl.dims, aw), noise, K, V, [awl.prefix] * 2, awl.n_steps, committed=com,
                             n_fixed=3, corr=ref_item)
        rel = rel_l2_per_rollout(got, ref)
        print("chained rel-L2 %.3e" % rel, flush=True)
        assert_bf16(got, ref, "chained")
        torch.cuda.synchronize()
    finally:
        ae.close()
        m.close()


def test_tiny_bf16_batch8_correction_rows_multikernel():
    """Eight rollouts of 4 correction + 10 action rows (112 rows: the
    multi-kernel path with several query tiles per rollout group), ragged
    prefixes including an empty one, committed rows, against the oracle."""
    torch_cuda()
    wl = synth.WORKLOADS["tiny-fp32"].with_(dtype="bf16", batch=8, n_fixed=1, name="tiny-bf16-corr-b8")
    lens = [64, 0, 17, 64, 1, 33, 63, 8]
    print("case tiny bf16 b8 + 4 correction rows, prefix_len %s" % lens, flush=True)
    w, K, V, noise, corr = _inputs(wl, 4, lens)
    com = synth.make_committed(wl)
    ae = make_expert(wl, w, max_batch=8, max_prefix=wl.prefix, max_corr=4)
    try:
        got = run(ae, K, V, noise, wl.n_steps, prefix_len=lens, committed=com, n_fixed=1, corr=corr)
    finally:
        ae.close()
    ref = oracle.denoise(oracle.Expert(wl.dims, w), noise, K, V, lens, wl.n_steps, committed=com, n_fixed=1,
                         corr=corr)
    rel = rel_l2_per_rollout(got, ref)
    print("rel-L2 %.3e max-abs %.3e" % (rel, np.abs(got - ref).max()), flush=True)
    assert_bf16(got, ref, "tiny bf16 b8 with correction rows")
    assert np.array_equal(got[:, :1].astype(np.float32), com)


def test_vlm_prefill_with_correction_tokens_bound():
    """The VLM prefill's in-place hand-off builds the expert's RoPE table for
    the suffix rows it sees; binding correction tokens before or after the
    prefill must give the same actions as the oracle on the prefill's KV."""
    torch = torch_cuda()
    from paper_2607_12659_amd.expert import to_device
    from gpu_util import Vlm
    import synth.vlm as sv
    vwl = sv.VLM_WORKLOADS["vlm-tiny"]
    awl = synth.WORKLOADS["tiny-fp32"].with_(dtype="bf16", name="tiny-bf16-vlm-corr")
    assert awl.dims.n_layers == vwl.dims.n_layers and awl.dims.head_dim == vwl.dims.head_dim
    print("case vlm-tiny prefill -> tiny bf16 expert with 3 correction tokens", flush=True)
    vw = sv.make_vlm_weights(vwl)
    emb = sv.make_embeddings(vwl)
    aw = synth.make_weights(awl)
    noise = synth.make_noise(awl)
    corr = sc.make_item(awl.seed, 1, 3, awl.dims.width)
    vlm = Vlm(vwl.dims, vw, 1, vwl.prefix)
    ae = make_expert(awl, aw, max_batch=1, max_prefix=vwl.prefix, max_corr=3)
    try:
        e_d = to_device(emb.astype(np.float32))
        c_d = to_device(corr.astype(np.float32))
        n_d = to_device(noise.astype(np.float32))
        vlm.prefill(e_d, 1, vwl.prefix, ae)          # tokens bound after the prefill
        ae.bind_state(None, 0, c_d)
        a = ae.denoise(n_d, awl.n_steps).cpu().numpy().astype(np.float64)
        vlm.prefill(e_d, 1, vwl.prefix, ae)          # tokens already bound during the prefill
        b = ae.denoise(n_d, awl.n_steps).cpu().numpy().astype(np.float64)
        ae.sync()
        torch.cuda.synchronize()
    finally:
        ae.close()
        vlm.close()
    Kr, Vr, _ = oracle.vlm_prefill(vwl.dims, vw, emb[0])
    ref = oracle.denoise(oracle.Expert(awl.dims, aw), noise, Kr[:, None], Vr[:, None], [vwl.prefix], awl.n_steps,
                         corr=corr)
    print("after-prefill binding rel-L2 %.3e, during-prefill binding %.3e"
          % (rel_l2_per_rollout(a, ref), rel_l2_per_rollout(b, ref)), flush=True)
    assert_bf16(a, ref, "after-prefill binding")
    assert_bf16(b, ref, "during-prefill binding")
    assert np.array_equal(a, b)
