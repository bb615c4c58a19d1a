"""The committed-rows-at-t=0 variant (jpi_set_committed_t0) against the fp64
oracle, on both denoise paths.  Same bars as the denoise parity."""
import numpy as np
import pytest

import oracle
import synth
from gpu_util import Inputs, load_golden, make_expert, rel_l2_per_rollout, run_env, torch_cuda
from synth import correction as sc

pytestmark = pytest.mark.gpu

BF16_TOL = 2e-2
F32_TOL = 1e-4


@pytest.mark.parametrize("dtype,n_corr", [("f32", 0), ("f32", 3), ("bf16", 0), ("bf16", 3)])
def test_tiny_committed_rows_at_t0(dtype, n_corr):
    torch_cuda()
    wl = synth.WORKLOADS["tiny-fp32"].with_(dtype=dtype, batch=2, n_fixed=3, prefix_len=(64, 9),
                                            name="tiny-t0-%s" % dtype)
    inp = Inputs(wl)
    # a time MLP ten times stronger than the N(0, 0.02) default, so that the
    # flow time of the committed rows moves the result well above the error bars
    for k in ("time_mlp.0.w", "time_mlp.1.w"):
        a = inp.weights[k]
        inp.weights[k] = (synth.f32_to_bf16_bits(synth.bf16_bits_to_f32(a) * np.float32(10)) if a.dtype == np.uint16
                          else (a * np.float32(10)).astype(np.float32))
    corr = sc.make_item(wl.seed, 2, n_corr, wl.dims.width) if n_corr else None
    print("case tiny %s committed rows at t=0, %d correction tokens" % (dtype, n_corr), flush=True)
    ae = make_expert(wl, inp.weights, max_corr=4)
    kw = dict(prefix_len=inp.prefix_len, committed=inp.committed, n_fixed=3, corr=corr)
    try:
        base = run_env(ae, None, inp.K, inp.V, inp.noise, wl.n_steps, **kw)
        ae.set_committed_t0(True)
        got = run_env(ae, None, inp.K, inp.V, inp.noise, wl.n_steps, **kw)
        multi = run_env(ae, "0", inp.K, inp.V, inp.noise, wl.n_steps, **kw)
        ae.set_committed_t0(False)
        back = run_env(ae, None, inp.K, inp.V, inp.noise, wl.n_steps, **kw)
    finally:
        ae.close()
    ex = oracle.Expert(wl.dims, inp.weights)
    ref = oracle.denoise(ex, inp.noise, inp.K, inp.V, inp.prefix_len, wl.n_steps, committed=inp.committed, n_fixed=3,
                         corr=corr, committed_t0=True)
    ref0 = oracle.denoise(ex, inp.noise, inp.K, inp.V, inp.prefix_len, wl.n_steps, committed=inp.committed,
                          n_fixed=3, corr=corr)
    err, rel = np.abs(got - ref).max(), rel_l2_per_rollout(got, ref)
    print("max-abs %.3e rel-L2 %.3e; multi-kernel vs oracle %.3e; the variant moves the actions by %.3e"
          % (err, rel, rel_l2_per_rollout(multi, ref), np.abs(ref - ref0).max()), flush=True)
    if dtype == "f32":
        assert err <= F32_TOL
    else:
        assert rel <= BF16_TOL and rel_l2_per_rollout(multi, ref) <= BF16_TOL
        assert rel_l2_per_rollout(got, multi) <= 5e-3
    assert np.abs(ref - ref0).max() > 20 * max(err, 1e-6)  # the variant is far outside the error
    assert np.array_equal(got[:, :3].astype(np.float32), inp.committed.astype(np.float32))
    assert np.array_equal(base, back)


def test_pi05_committed10_at_t0():
    """pi0.5, one rollout, 10 committed rows at t = 0, against the stored
    oracle output on the single-launch and the multi-kernel path.  (With the
    N(0, 0.02) time MLP the variant moves these actions by only ~6e-4, so the
    tiny tests carry the discrimination.)"""
    torch_cuda()
    wl = synth.WORKLOADS["pi05-b1-committed10"]
    print("case pi05-b1-committed10-t0", flush=True)
    w = synth.make_weights(wl)
    K, V = synth.make_prefix(wl)
    noise = synth.make_noise(wl)
    com = synth.make_committed(wl)
    ae = make_expert(wl, w, max_batch=1, max_prefix=816)
    try:
        ae.set_committed_t0(True)
        got = run_env(ae, None, K, V, noise, wl.n_steps, committed=com, n_fixed=10)
        multi = run_env(ae, "0", K, V, noise, wl.n_steps, committed=com, n_fixed=10)
        again = run_env(ae, None, K, V, noise, wl.n_steps, committed=com, n_fixed=10)
    finally:
        ae.close()
    ref, meta = load_golden("pi05-b1-committed10-t0")
    assert meta["committed_t0"] is True
    plain, _ = load_golden("pi05-b1-committed10")
    effect = rel_l2_per_rollout(plain, ref)
    for label, out in (("single-launch", got), ("multi-kernel", multi)):
        rel = rel_l2_per_rollout(out, ref)
        print("%s: rel-L2 %.3e max-abs %.3e; the variant moves the actions by %.3e"
              % (label, rel, np.abs(out - ref).max(), effect), flush=True)
        assert rel <= BF16_TOL
        assert np.array_equal(out[:, :10].astype(np.float32), com)
    assert np.array_equal(got, again)
