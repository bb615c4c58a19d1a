"""Benchmark of the flow-matching action-expert denoise on one MI355X.

One "step" of this benchmark is one jpi_denoise call: the whole hot path
(n_steps Euler steps of the action expert over one action chunk per rollout,
every layer attending to the resident prefix KV), on inputs already resident
in HBM.  Prints one JSON line:

  value      action chunks/s = batch * steps / timed seconds
  roofline   the dominant kernel's algorithmic bytes per launch / its average
             launch duration (start/stop HIP events tied to every dispatch of
             that kernel on the stream it runs on, in a timing pass right after
             the timed region), against MI355X's 8 TB/s HBM peak.  With
             batch * horizon <= 64 the whole call is one persistent kernel;
             otherwise the largest GEMM kind.  "kernels" lists every kind that
             ran.  "traffic" is the HBM bytes per launch measured with the
             FETCH_SIZE / WRITE_SIZE counters (scaled by a plain copy of known
             size, see --calibrate-copy) when the counters were taken on the
             current kernel source, else null
  measured_peaks  second denominators from the same run: a plain device copy
             (read + write GB/s) and a large bf16 GEMM (TFLOP/s) on this GPU
  cpu_baseline  the fp64 CPU oracle timed on the host cores, repeating the
                denoise of rollout 0 for at least 10 s (a bounded sample)

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME] [--no-cpu]
       python bench.py --calibrate-copy MIB   (a plain device copy, for counter scaling)
       python bench.py --workload NAME --calls-only N   (N calls and nothing else: a profiler's target)
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
BF16_MFMA_PEAK_TFLOPS = 2500.0
FP32_MFMA_PEAK_TFLOPS = 157.3

METRIC = "action chunks/sec (10-step flow denoise, pi0.5 shape, B=1); % HBM roofline"

# HBM traffic per launch of the persistent kernel from the FETCH_SIZE and
# WRITE_SIZE counters (rocprofv3 --pmc, one counter per run), keyed by the
# sha256 of the kernel source they were measured on; the byte counts are the
# counter readings times the copy calibration factor.
MEASURED_TRAFFIC = {
    # pi0.5 shape, batch 1: FETCH_SIZE 5213836.7 KiB x 1.99980 (a 256 MiB copy
    # reads back 131085.1875 KiB) + WRITE_SIZE 2469905.2 KiB x 1.00000 (the copy's
    # 262144 KiB), mean over 4 dispatches
    ("56f8be3ce3d539a631ccde8da1389902a25e5adb47a067af137615c17ce43316", "pi05-b1"):
        round(5213836.671875 * 1024 * 1.9997987949630083 + 2469905.1875 * 1024),
}


def kernel_source_hash():
    """sha256 of the single-launch kernel's code: its source and the device
    headers it includes, with comments and whitespace removed, so that the
    recorded traffic stays attached to the code it was measured on and nothing
    else."""
    import hashlib
    import re
    src = ""
    for name in ("jpi_persist.hip", "jpi_device.h", "jpi_internal.h"):
        with open(os.path.join(ROOT, "paper_2607_12659_amd", "csrc", name)) as f:
            src += f.read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    src = re.sub(r"//[^\n]*", "", src)
    return hashlib.sha256("".join(src.split()).encode()).hexdigest()


def calibrate_copy(mib):
    """A plain device-to-device copy of known size (for scaling the counters)."""
    import torch
    n = mib * (1 << 20) // 4
    src = torch.ones(n, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_bytes_read": n * 4, "copy_bytes_written": n * 4, "launches": 3}), flush=True)


def measured_peaks():
    """Second denominators measured on this GPU in the same run: a plain device
    copy of 1 GiB (read + write bytes per second) and a large plain bf16 GEMM
    (8192^3, contiguous operands)."""
    import torch
    x = torch.ones(1 << 29, dtype=torch.bfloat16, device="cuda")
    y = torch.empty_like(x)
    a = torch.randn(8192, 8192, dtype=torch.bfloat16, device="cuda")
    b = torch.randn(8192, 8192, dtype=torch.bfloat16, device="cuda")

    def timed(fn, reps):
        fn()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(reps):
            fn()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / reps * 1e-3

    t_copy = timed(lambda: y.copy_(x), 5)
    t_gemm = timed(lambda: torch.matmul(a, b), 5)
    del x, y, a, b
    torch.cuda.empty_cache()
    return {"copy_GBs": round(2.0 * (1 << 30) / t_copy / 1e9, 1),
            "bf16_gemm_TFLOPs": round(2.0 * 8192 ** 3 / t_gemm / 1e12, 1),
            "method": "torch copy of 1 GiB (read + write bytes); torch.matmul 8192^3 bf16"}


def algorithmic_counts(wl):
    """Bytes and flops one denoise call must move / compute.

    Weights are read once per Euler step (shared by the batch); each rollout's
    valid prefix KV once per step; the modulation rows used per step are
    counted; activations (cache-resident) and the once-per-(weights, N) time
    MLP / modulation precompute are not.
    """
    d = wl.dims
    es = 2 if wl.dtype == "bf16" else 4
    W, F, Dh, nH, A, L, H = d.width, d.mlp_dim, d.head_dim, d.n_heads, d.action_dim, d.n_layers, d.horizon
    per_layer = {"qkv": (nH + 2) * Dh * W, "oproj": W * nH * Dh, "gateup": 2 * F * W, "down": W * F}
    w_layer = sum(per_layer.values()) * es
    w_step = L * w_layer + (2 * W * A) * es
    kv_step = sum(2 * L * pl * Dh * es for pl in wl.valid_lengths())
    mod_step = (6 * L + 2) * W * 4
    M = wl.batch * H
    keys = [pl + H for pl in wl.valid_lengths()]
    gemm_flops = 2 * M * (L * sum(per_layer.values()) + 2 * W * A)
    attn_flops = sum(4 * L * nH * H * k * Dh for k in keys)
    return {
        "bytes_per_call": (w_step + kv_step + mod_step) * wl.n_steps,
        "flops_per_call": (gemm_flops + attn_flops) * wl.n_steps,
        "kernel_bytes": dict({k: v * es for k, v in per_layer.items()},
                             persistent=(w_step + kv_step + mod_step) * wl.n_steps),
        "kernel_flops": {k: 2 * M * v for k, v in per_layer.items()},
    }


def host_cpu():
    """The host's CPU model and the core counts the oracle could use."""
    model = ""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:  # pragma: no cover
        pass
    try:
        usable = len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        usable = os.cpu_count()
    return {"cpu_model": model, "nproc": os.cpu_count(), "usable_cores": usable}


def check_output(got, ref, dtype):
    """The timed output of rollout 0 against the oracle's, at the contract bars:
    fp32 max-abs <= 1e-4; bf16 relative L2 <= 2e-2 and every element within
    2e-2 of the largest reference magnitude."""
    import numpy as np
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    err = np.abs(got - ref)
    rel = float(np.linalg.norm(got - ref) / np.linalg.norm(ref))
    elem = float(err.max() / np.abs(ref).max())
    if dtype == "f32":
        ok = bool(np.isfinite(got).all() and err.max() <= 1e-4)
        bar = "max-abs <= 1e-4"
    else:
        ok = bool(np.isfinite(got).all() and rel <= 2e-2 and elem <= 2e-2)
        bar = "relative L2 <= 2e-2 and max|err| <= 2e-2 max|ref|"
    return {"checked": "rollout 0 of the last timed call vs the fp64 oracle on the same inputs",
            "rel_l2": rel, "elem_rel": elem, "max_abs": float(err.max()), "bar": bar, "ok": ok}


def blas_threads():
    """Threads numpy's BLAS uses on this host (what the fp64 oracle runs on)."""
    try:
        from threadpoolctl import threadpool_info
        return max([t.get("num_threads", 1) for t in threadpool_info()] or [1])
    except Exception:  # pragma: no cover
        return os.cpu_count()


def cpu_baseline(wl, weights, K, V, noise, committed=None, committed_t0=False):
    """Times the oracle on rollout 0 (a bounded sample) and returns
    (baseline entry, the oracle's actions for rollout 0)."""
    import oracle
    threads = blas_threads()
    host = host_cpu()
    ex = oracle.Expert(wl.dims, weights)
    lens = wl.valid_lengths()[:1]
    com = None if committed is None else committed[:1]
    # Bounded sample: repeat the denoise of rollout 0 until at least 10 s of host time
    # has passed (and at most 16 calls), then report calls per second.
    calls, t0, ref = 0, time.perf_counter(), None
    while True:
        out = oracle.denoise(ex, noise[:1], K[:, :1], V[:, :1], lens, wl.n_steps, committed=com,
                             n_fixed=wl.n_fixed, committed_t0=committed_t0)
        ref = out if ref is None else ref
        calls += 1
        dt = time.perf_counter() - t0
        if dt >= 10.0 or calls >= 16:
            break
    entry = {"value": round(calls / dt, 4), "unit": "chunks/s", "cores": int(threads), "kind": "oracle",
             "blas_threads": int(threads), "nproc": host["nproc"], "usable_cores": host["usable_cores"],
             "cpu_model": host["cpu_model"],
             "sample": "%d repeated %d-step denoise calls on rollout 0 of %s (fp64 numpy, BLAS threads=%d), "
                       "%.1f s in total" % (calls, wl.n_steps, wl.name, threads, dt)}
    return entry, ref[0]


def prefill_flops(vd, batch, prefix):
    """Matrix and attention flops of one VLM prefill (every layer)."""
    W, nH, Dh, F, M = vd.width, vd.n_heads, vd.head_dim, vd.mlp_dim, batch * prefix
    per_layer = 2.0 * M * W * (nH + 2) * Dh + 4.0 * batch * nH * prefix * prefix * Dh + 2.0 * M * nH * Dh * W \
        + 2.0 * M * W * 2 * F + 2.0 * M * F * W
    return vd.n_layers * per_layer


def bench_prefill(args, vwl):
    """VLM prefill (Gemma-2B shape) writing its KV in place into a pi0.5 expert
    context: one step = one prefill of every layer over the whole prefix."""
    import numpy as np
    import torch

    import synth
    import synth.vlm as synth_vlm
    from paper_2607_12659_amd import jpi
    from paper_2607_12659_amd.expert import ActionExpert, to_device

    vd = vwl.dims
    print("bench: workload %s, generating %.2f B synthetic parameters" % (
        vwl.name, sum(int(np.prod(s)) for _, s, _ in synth_vlm.vlm_weight_specs(vd)) / 1e9), file=sys.stderr, flush=True)
    vw = synth_vlm.make_vlm_weights(vwl)
    emb = synth_vlm.make_embeddings(vwl)
    torch.cuda.set_device(0)
    stream = torch.cuda.current_stream()
    cfg = jpi.jpi_vlm_config(n_layers=vd.n_layers, width=vd.width, n_heads=vd.n_heads, n_kv_heads=vd.n_kv_heads,
                             head_dim=vd.head_dim, mlp_dim=vd.mlp_dim, max_batch=vwl.batch, max_prefix=vwl.prefix,
                             dtype=jpi.JPI_BF16, rms_eps=1e-6, rope_base=1e4)
    st, vlm = jpi.jpi_vlm_create(cfg)
    jpi.check(st)
    for name, arr in vw.items():
        arr = np.ascontiguousarray(arr)
        st = jpi.jpi_vlm_set_weight(vlm, name, arr, arr.size, jpi.JPI_BF16 if arr.dtype == np.uint16 else jpi.JPI_F32, 0)
        if st != jpi.JPI_OK:
            raise RuntimeError(jpi.jpi_vlm_last_error(vlm))
    del vw
    if jpi.jpi_vlm_finalize_weights(vlm) != jpi.JPI_OK:
        raise RuntimeError(jpi.jpi_vlm_last_error(vlm))
    ewl = synth.WORKLOADS["pi05-b1"]
    ae = ActionExpert(ewl.dims, ewl.dtype, vwl.batch, vwl.prefix)
    ae.load_weights(synth.make_weights(ewl))
    e_dev = to_device(np.ascontiguousarray(emb, np.float32))

    def once():
        st = jpi.jpi_vlm_prefill(vlm, e_dev, vwl.batch, vwl.prefix, ae.ctx, None, stream)
        if st != jpi.JPI_OK:
            raise RuntimeError(jpi.jpi_vlm_last_error(vlm))

    for _ in range(args.warmup):
        once()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(args.steps):
        once()
    e1.record(stream)
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / args.steps
    fl = prefill_flops(vd, vwl.batch, vwl.prefix)
    tflops = fl / (ms * 1e-3) / 1e12
    # the expert consumes the KV in place: one denoise right after the prefill
    noise = to_device(np.ascontiguousarray(synth.make_noise(ewl), np.float32))
    out = ae.denoise(noise, ewl.n_steps)
    ae.sync()
    finite = bool(torch.isfinite(out).all().item())
    cpu = None
    if not args.no_cpu:
        import oracle
        vd1 = synth_vlm.VlmDims(**{**vd.__dict__, "n_layers": 1})
        w1 = synth_vlm.make_vlm_weights(vwl, n_layers=1)
        t0 = time.time()
        oracle.vlm_prefill(vd1, w1, emb[0])
        dt = time.time() - t0
        cpu = {"value": vwl.prefix / (dt * vd.n_layers), "unit": "tokens/s", "cores": blas_threads(),
               "kind": "oracle", "sample": "one of the %d layers of the fp64 oracle prefill over %d tokens "
               "(%.1f s), scaled to the whole stack" % (vd.n_layers, vwl.prefix, dt)}
    result = {
        "metric": "VLM prefill tokens/sec (Gemma-2B shape, prefix KV written in place into the action expert)",
        "value": round(vwl.batch * vwl.prefix / (ms * 1e-3), 1), "unit": "tokens/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms, 4), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": vwl.name, "batch": vwl.batch, "prefix_tokens": vwl.prefix, "layers": vd.n_layers,
                   "width": vd.width, "heads": vd.n_heads, "kv_heads": vd.n_kv_heads, "head_dim": vd.head_dim,
                   "mlp_dim": vd.mlp_dim},
        "roofline": {"bound": "mfma", "achieved": round(tflops, 2), "peak": BF16_MFMA_PEAK_TFLOPS, "unit": "TFLOP/s",
                     "frac": round(tflops / BF16_MFMA_PEAK_TFLOPS, 4), "traffic": None,
                     "flops_per_launch": fl, "avg_launch_us": round(ms * 1e3, 1)},
        "cpu_baseline": cpu, "expert_after_handoff_finite": finite,
    }
    ae.close()
    jpi.jpi_vlm_destroy(vlm)
    print(json.dumps(result), flush=True)


def corr_bytes(cd, wl):
    """Algorithmic HBM bytes of one VLM-refresh call of the correction module
    (compress + predict): every weight once, the VLM state, actions, item and
    confidence."""
    import numpy as np
    import synth.correction as synth_corr
    wbytes = sum(int(np.prod(s)) * (2 if mat else 4) for _, s, mat in synth_corr.corr_weight_specs(cd))
    io = wl.batch * (wl.vlm_tokens * cd.vlm_width * 2 + wl.n_actions * cd.action_dim * 4
                     + 2 * cd.n_query * cd.width * 4 + 4)
    return wbytes + io


def bench_corr(args, cwl):
    """Future correction module (about 40M parameters): one step = the
    VLM-refresh branch of Algorithm 1 (compress the VLM final-layer state,
    then predict the correction item and confidence from the committed
    actions).  Also timed: the skip branch alone (predict from the previous
    item) and a whole skip iteration (predict, then the pi0.5 expert denoise
    with the 4-token item and the committed rows)."""
    import numpy as np
    import torch

    import synth
    import synth.correction as synth_corr
    from paper_2607_12659_amd import jpi
    from paper_2607_12659_amd.expert import ActionExpert, to_device

    cd = cwl.dims
    print("bench: workload %s" % cwl.name, file=sys.stderr, flush=True)
    w = synth_corr.make_corr_weights(cwl)
    vs = synth_corr.make_vlm_state(cwl)
    acts = synth_corr.make_actions(cwl)
    torch.cuda.set_device(0)
    stream = torch.cuda.current_stream()
    cfg = jpi.jpi_corr_config(width=cd.width, n_heads=cd.n_heads, n_kv_heads=1, head_dim=cd.head_dim,
                              mlp_dim=cd.mlp_dim, action_dim=cd.action_dim, vlm_width=cd.vlm_width,
                              n_query=cd.n_query, max_batch=cwl.batch, max_actions=cwl.n_actions,
                              max_vlm_tokens=cwl.vlm_tokens, dtype=jpi.JPI_BF16, rms_eps=1e-6, rope_base=1e4)
    st, m = jpi.jpi_corr_create(cfg)
    jpi.check(st)
    for name, arr in w.items():
        arr = np.ascontiguousarray(arr)
        st = jpi.jpi_corr_set_weight(m, name, arr, arr.size, jpi.JPI_BF16 if arr.dtype == np.uint16 else jpi.JPI_F32, 0)
        if st != jpi.JPI_OK:
            raise RuntimeError(jpi.jpi_corr_last_error(m))
    if jpi.jpi_corr_finalize_weights(m) != jpi.JPI_OK:
        raise RuntimeError(jpi.jpi_corr_last_error(m))
    vs_d = to_device(vs)
    a_d = to_device(acts.astype(np.float32))
    state = torch.empty((cwl.batch, cd.n_query, cd.width), device="cuda")
    item = torch.empty_like(state)
    conf = torch.empty((cwl.batch,), device="cuda")

    def refresh():
        jpi.check(jpi.jpi_corr_compress(m, vs_d, cwl.batch, cwl.vlm_tokens, state, stream))
        jpi.check(jpi.jpi_corr_predict(m, state, a_d, cwl.batch, cwl.n_actions, item, conf, stream))

    def skip():
        jpi.check(jpi.jpi_corr_predict(m, item, a_d, cwl.batch, cwl.n_actions, item, conf, stream))

    def timed(fn, steps, warmup):
        for _ in range(warmup):
            fn()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(steps):
            fn()
        e1.record(stream)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / steps

    ms = timed(refresh, args.steps, args.warmup)
    ms_skip = timed(skip, args.steps, args.warmup)
    # a whole skip iteration: the item goes straight into the expert
    ewl = synth.WORKLOADS["pi05-b1-committed10"]
    ae = ActionExpert(ewl.dims, ewl.dtype, 1, ewl.prefix, max_corr=cd.n_query)
    ae.load_weights(synth.make_weights(ewl))
    K, V = synth.make_prefix(ewl)
    ae.bind_prefix(to_device(K), to_device(V), stream=stream)
    com = to_device(np.ascontiguousarray(synth.make_committed(ewl), np.float32))
    noise = to_device(np.ascontiguousarray(synth.make_noise(ewl), np.float32))
    out = torch.empty_like(noise)

    def iteration():
        skip()
        ae.bind_state(com, ewl.n_fixed, item, stream=stream)
        ae.denoise(noise, ewl.n_steps, out=out, stream=stream)

    ms_iter = timed(iteration, max(5, args.steps // 5), 2)
    ae.sync()
    finite = bool(torch.isfinite(out).all().item()) and bool(torch.isfinite(conf).all().item())
    ae.close()
    jpi.jpi_corr_destroy(m)
    byts = corr_bytes(cd, cwl)
    gbs = byts / (ms * 1e-3) / 1e9
    cpu = None
    if not args.no_cpu:
        import oracle
        calls, t0 = 0, time.time()
        while True:
            oracle.correction.forward(cd, w, acts[:1], vlm_state=vs[:1])
            calls += 1
            if time.time() - t0 >= 10.0:
                break
        dt = time.time() - t0
        cpu = {"value": round(calls / dt, 3), "unit": "refresh calls/s", "cores": blas_threads(), "kind": "oracle",
               "sample": "%d repeated fp64 oracle calls (compress + predict, rollout 0), %.1f s" % (calls, dt)}
    result = {
        "metric": "future correction module calls/sec (VLM-refresh branch: compress + predict, ~40M parameters)",
        "value": round(cwl.batch / (ms * 1e-3), 1), "unit": "calls/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(ms, 4), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": cwl.name, "batch": cwl.batch, "committed_actions": cwl.n_actions,
                   "vlm_tokens": cwl.vlm_tokens, "width": cd.width, "heads": cd.n_heads, "head_dim": cd.head_dim,
                   "mlp_dim": cd.mlp_dim, "vlm_width": cd.vlm_width, "n_query": cd.n_query},
        "roofline": {"bound": "hbm", "achieved": round(gbs, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(gbs / HBM_PEAK_GBS, 4), "traffic": None, "bytes_per_launch": byts,
                     "avg_launch_us": round(ms * 1e3, 1), "note": "whole call (about 40 launches), not one kernel"},
        "skip_branch_ms": round(ms_skip, 4),
        "skip_iteration_ms": round(ms_iter, 4),
        "cpu_baseline": cpu, "outputs_finite": finite,
    }
    print(json.dumps(result), flush=True)


def pi0_bytes(d, wl):
    """Algorithmic HBM bytes of one call of the action-time (pi0-style) expert:
    per Euler step every layer matrix and the action-time MLP once plus each
    rollout's valid prefix KV (and the state slot); once per call the state
    token's pass over every layer matrix and the prefix KV."""
    import numpy as np
    import synth.pi0 as synth_pi0
    es = 2 if wl.dtype == "bf16" else 4
    layer = sum(int(np.prod(s)) * es for n, s, mat in synth_pi0.pi0_weight_specs(d) if mat and n.startswith("layers."))
    mlp = sum(int(np.prod(s)) * es for n, s, mat in synth_pi0.pi0_weight_specs(d)
              if mat and n.startswith("action_time_mlp"))
    kv = sum(wl.valid_lengths()) * d.n_layers * d.head_dim * 2 * es
    return wl.n_steps * (layer + mlp + kv + wl.batch * d.n_layers * d.head_dim * 2 * es) + layer + kv


def bench_pi0(args, wl):
    """The action-time (pi0-style) expert: one step = one jpi_denoise call
    (the state token's pass, then N Euler steps) at the pi0.5 shape."""
    import numpy as np
    import torch

    import synth
    import synth.pi0 as synth_pi0
    from paper_2607_12659_amd import jpi
    from paper_2607_12659_amd.expert import ActionExpert, to_device

    d = wl.dims
    print("bench: workload %s" % wl.name, file=sys.stderr, flush=True)
    w = synth_pi0.make_pi0_weights(wl)
    K, V = synth.make_prefix(wl)
    noise = synth.make_noise(wl)
    st = synth_pi0.make_state(wl)
    torch.cuda.set_device(0)
    stream = torch.cuda.current_stream()
    ae = ActionExpert(d, wl.dtype, wl.batch, wl.prefix + 1, variant=jpi.JPI_VARIANT_ACTION_TIME,
                      state_dim=synth_pi0.STATE_DIM)
    ae.load_weights(w)
    ae.bind_prefix(to_device(K), to_device(V), wl.valid_lengths(), stream=stream)
    ae.bind_state(None, 0, stream=stream)
    ae.bind_robot_state(to_device(st.astype(np.float32)), stream=stream)
    nd = to_device(noise.astype(np.float32))
    out = torch.empty_like(nd)
    for _ in range(args.warmup):
        ae.denoise(nd, wl.n_steps, out=out, stream=stream)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(args.steps):
        ae.denoise(nd, wl.n_steps, out=out, stream=stream)
    e1.record(stream)
    torch.cuda.synchronize()
    ae.sync()
    ms = e0.elapsed_time(e1) / args.steps
    finite = bool(torch.isfinite(out).all().item())
    ae.close()
    byts = pi0_bytes(d, wl)
    gbs = byts / (ms * 1e-3) / 1e9
    cpu = None
    if not args.no_cpu:
        import oracle
        calls, t0 = 0, time.time()
        while True:
            oracle.pi0.denoise(d, w, noise[:1], K[:, :1], V[:, :1], wl.valid_lengths()[:1], wl.n_steps, st[:1])
            calls += 1
            if time.time() - t0 >= 10.0:
                break
        dt = time.time() - t0
        cpu = {"value": round(calls / dt, 4), "unit": "chunks/s", "cores": blas_threads(), "kind": "oracle",
               "sample": "%d repeated %d-step fp64 oracle denoise calls of rollout 0 (%.1f s)" % (calls, wl.n_steps, dt)}
    result = {
        "metric": "action chunks/sec (10-step flow denoise, action-time pi0-style expert, pi0.5 shape, B=1)",
        "value": round(wl.batch / (ms * 1e-3), 3), "unit": "chunks/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(ms, 4), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": wl.dtype, "data": "synthetic",
        "config": {"workload": wl.name, "batch": wl.batch, "prefix_tokens": wl.valid_lengths(), "horizon": d.horizon,
                   "layers": d.n_layers, "width": d.width, "n_steps": wl.n_steps, "variant": "action_time",
                   "state_dim": synth_pi0.STATE_DIM},
        "roofline": {"bound": "hbm", "achieved": round(gbs, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(gbs / HBM_PEAK_GBS, 4), "traffic": None, "bytes_per_launch": byts,
                     "avg_launch_us": round(ms * 1e3, 1), "note": "whole call on the multi-kernel graph"},
        "cpu_baseline": cpu, "outputs_finite": finite,
    }
    print(json.dumps(result), flush=True)


PI0_WORKLOADS = ("pi0-b1",)
LOOP_WORKLOADS = ("loop-pi05-gemma2b",)


def bench_loop(args):
    """Algorithm 1 on one MI355X with every model on the GPU: the VLM hook is
    the Gemma-2B-shape prefill (816 tokens, KV in place into the expert) plus
    the correction module's compression of its final hidden state; the
    correction hook is the module's prediction from the committed actions;
    the action hook binds the predicted item and denoises the pi0.5 expert.
    Weights are synthetic, so the confidence the module computes means
    nothing: the hook returns a forced trace that refreshes the VLM on one
    iteration in seven (the paper's VLM fraction).  One step = one loop
    iteration; `value` is the control frequency 1000 / mean iteration time."""
    import numpy as np
    import torch

    import synth
    import synth.correction as synth_corr
    import synth.vlm as synth_vlm
    from paper_2607_12659_amd import jpi
    from paper_2607_12659_amd.expert import ActionExpert, to_device

    torch.cuda.set_device(0)
    stream = torch.cuda.current_stream()
    ewl = synth.WORKLOADS["pi05-b1"]
    vwl = synth_vlm.VLM_WORKLOADS["gemma2b-p816"]
    cwl = synth_corr.CORR_WORKLOADS["corr40m-p816"]
    vd, cd = vwl.dims, cwl.dims
    print("bench: Algorithm 1 loop, generating the three models", file=sys.stderr, flush=True)
    ae = ActionExpert(ewl.dims, ewl.dtype, 1, vwl.prefix, max_corr=cd.n_query)
    ae.load_weights(synth.make_weights(ewl))
    vcfg = jpi.jpi_vlm_config(n_layers=vd.n_layers, width=vd.width, n_heads=vd.n_heads, n_kv_heads=vd.n_kv_heads,
                              head_dim=vd.head_dim, mlp_dim=vd.mlp_dim, max_batch=1, max_prefix=vwl.prefix,
                              dtype=jpi.JPI_BF16, rms_eps=1e-6, rope_base=1e4)
    st, vlm = jpi.jpi_vlm_create(vcfg)
    jpi.check(st)
    for name, arr in synth_vlm.make_vlm_weights(vwl).items():
        arr = np.ascontiguousarray(arr)
        jpi.check(jpi.jpi_vlm_set_weight(vlm, name, arr, arr.size, jpi.JPI_BF16 if arr.dtype == np.uint16 else jpi.JPI_F32, 0))
    jpi.check(jpi.jpi_vlm_finalize_weights(vlm))
    ccfg = jpi.jpi_corr_config(width=cd.width, n_heads=cd.n_heads, n_kv_heads=1, head_dim=cd.head_dim,
                               mlp_dim=cd.mlp_dim, action_dim=cd.action_dim, vlm_width=cd.vlm_width,
                               n_query=cd.n_query, max_batch=1, max_actions=ewl.dims.horizon,
                               max_vlm_tokens=vwl.prefix, dtype=jpi.JPI_BF16, rms_eps=1e-6, rope_base=1e4)
    st, corr = jpi.jpi_corr_create(ccfg)
    jpi.check(st)
    for name, arr in synth_corr.make_corr_weights(cwl).items():
        arr = np.ascontiguousarray(arr)
        jpi.check(jpi.jpi_corr_set_weight(corr, name, arr, arr.size, jpi.JPI_BF16 if arr.dtype == np.uint16 else jpi.JPI_F32, 0))
    jpi.check(jpi.jpi_corr_finalize_weights(corr))
    emb = to_device(np.ascontiguousarray(synth_vlm.make_embeddings(vwl), np.float32))
    hidden = torch.empty((1, vwl.prefix, vd.width), dtype=torch.int16, device="cuda")
    item = torch.empty((1, cd.n_query, cd.width), device="cuda")      # the hidden-state buffer B_h
    conf_d = torch.empty((1,), device="cuda")
    noise = to_device(np.ascontiguousarray(synth.make_noise(ewl), np.float32))
    chunk = torch.empty_like(noise)                                    # the expert's latest chunk
    # the action buffer B_a as an absolute timeline: the chunk that starts at
    # action index s occupies rows s .. s + H - 1 (Algorithm 1 reads the
    # committed actions a_t .. a_{t+n-1} from it); sized for every iteration
    H_a = ewl.dims.horizon
    timeline = torch.zeros(((args.steps + max(1, args.warmup) + 4) * 2 * H_a + 64, ewl.dims.action_dim),
                           device="cuda")
    forced = [1.0] * 6 + [-1.0]
    times = {"vlm": [], "corr": [], "act": []}
    calls = {"corr": 0}

    def timed(kind, fn):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        e0.record(stream)
        fn()
        e1.record(stream)
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1)
        times[kind].append(ms)
        return ms

    def vlm_fn():
        jpi.check(jpi.jpi_vlm_prefill(vlm, emb, 1, vwl.prefix, ae.ctx, hidden, stream))
        jpi.check(jpi.jpi_corr_compress(corr, hidden, 1, vwl.prefix, item, stream))  # B_h <- compressed h_t

    def vlm_hook(user, t, ms):
        ms[0] = timed("vlm", vlm_fn)
        return 0

    def corr_hook(user, t, n, from_vlm, start, c, ms):
        n = max(1, min(n, H_a))
        committed = timeline[t:t + n]   # a_t .. a_{t+n-1}, contiguous rows
        # B_h holds the fresh compression after a refresh, else the previous item
        ms[0] = timed("corr", lambda: jpi.check(jpi.jpi_corr_predict(corr, item, committed, 1, n, item, conf_d,
                                                                     stream)))
        c[0] = forced[calls["corr"] % len(forced)]
        calls["corr"] += 1
        return 0

    def act_fn(with_item):
        # f_act(h, B_kv): the predicted item when there is one (not for the first chunk)
        ae.bind_state(None, 0, item if with_item else None, stream=stream)
        ae.denoise(noise, ewl.n_steps, out=chunk, stream=stream)

    def act_hook(user, t, have_corr, start, ms):
        ms[0] = timed("act", lambda: act_fn(have_corr))
        ae.sync(stream)   # a timed-out wait of the single-launch kernel would invalidate the chunk
        timeline[start:start + H_a].copy_(chunk[0])
        return 0

    hooks = jpi.jpi_sched_hooks(jpi.SCHED_VLM_FN(vlm_hook), jpi.SCHED_CORR_FN(corr_hook), jpi.SCHED_ACT_FN(act_hook),
                                None)
    action_ms = 50.0  # a 20 Hz robot
    # warm-up (graph capture, tables), then the measured loop with Delta from the warm timings
    for _ in range(max(1, args.warmup)):
        vlm_hook(None, 0, [0.0])
        corr_hook(None, 0, 10, 1, 0, [0.0], [0.0])
        act_hook(None, 0, 1, 0, [0.0])
    for k in times:
        times[k].clear()
    calls["corr"] = 0
    probe = timed("vlm", vlm_fn) + timed("corr", lambda: None) + timed("act", lambda: act_fn(True))
    for k in times:
        times[k].clear()
    delta = max(1, int(np.ceil(probe / action_ms)))
    cfg = jpi.jpi_sched_config(theta=-0.5, delta=delta, delta_ae=1, chunk_len=ewl.dims.horizon, action_ms=action_ms,
                               iterations=args.steps)
    st, stats, _ = jpi.jpi_sched_run(cfg, hooks, 0)
    jpi.check(st)
    ae.sync()
    finite = bool(torch.isfinite(chunk).all().item())
    mean = {k: (sum(v[1:] if k != "corr" else v) / max(1, len(v[1:] if k != "corr" else v))) for k, v in times.items()}
    sync_ms = mean["vlm"] + mean["act"]  # a synchronous VLA: refresh the VLM before every chunk
    cnt = algorithmic_counts(ewl)
    gbs = cnt["bytes_per_call"] / (mean["act"] * 1e-3) / 1e9
    jpi.jpi_corr_destroy(corr)
    jpi.jpi_vlm_destroy(vlm)
    ae.close()
    result = {
        "metric": "control frequency (Hz) of the confidence-scheduled asynchronous loop (Algorithm 1): Gemma-2B-shape "
                  "VLM prefill, ~40M correction module, pi0.5 expert, all on one GPU",
        "value": round(stats.control_hz, 2), "unit": "Hz", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(stats.reaction_ms, 4), "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "bf16", "data": "synthetic",
        "config": {"workload": "loop-pi05-gemma2b", "vlm_fraction": round(stats.vlm_fraction, 4), "delta": delta,
                   "delta_ae": 1, "action_ms": action_ms, "prefix_tokens": vwl.prefix, "horizon": ewl.dims.horizon},
        "components_ms": {"vlm_refresh": round(mean["vlm"], 4), "correction_predict": round(mean["corr"], 4),
                          "expert_with_item": round(mean["act"], 4)},
        "synchronous_reaction_ms": round(sync_ms, 4),
        "reaction_reduction": round(sync_ms / stats.reaction_ms, 3),
        "roofline": {"bound": "hbm", "kernel": "k_persist (the expert call inside the loop)", "achieved": round(gbs, 1),
                     "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": round(gbs / HBM_PEAK_GBS, 4), "traffic": None},
        "cpu_baseline": None, "outputs_finite": finite,
        "note": "forced confidence trace (synthetic weights); iteration times include host synchronisation per hook",
    }
    print(json.dumps(result), flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="pi05-b1")
    ap.add_argument("--timed-kernel", default="auto",
                    choices=["auto", "persistent", "qkv", "attention", "oproj", "gateup", "down"])
    ap.add_argument("--no-cpu", action="store_true")
    ap.add_argument("--committed-t0", action="store_true",
                    help="committed rows at flow time t = 0 (the variant; the default workloads share t)")
    ap.add_argument("--calibrate-copy", type=int, default=0, metavar="MIB")
    ap.add_argument("--calls-only", type=int, default=0, metavar="N",
                    help="set up the workload, run N denoise calls (after one untimed call), sync and exit "
                         "without a JSON line: a profiler's target")
    args = ap.parse_args()
    if args.calibrate_copy:
        calibrate_copy(args.calibrate_copy)
        return
    if args.gpus != 1:
        print("bench.py measures one GPU: libjpi has no multi-GPU path (the denoise of one chunk runs on "
              "one MI355X; rollouts would shard data-parallel with no exchange). Run with --gpus 1.",
              file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    import synth
    import synth.correction as synth_corr
    import synth.vlm as synth_vlm
    from paper_2607_12659_amd import jpi
    from paper_2607_12659_amd.expert import ActionExpert, to_device

    if args.workload in synth_vlm.VLM_WORKLOADS:
        bench_prefill(args, synth_vlm.VLM_WORKLOADS[args.workload])
        return
    if args.workload in synth_corr.CORR_WORKLOADS:
        bench_corr(args, synth_corr.CORR_WORKLOADS[args.workload])
        return
    if args.workload in LOOP_WORKLOADS:
        bench_loop(args)
        return
    if args.workload in PI0_WORKLOADS:
        # the pi0.5 shape with one prefix slot left for the robot-state token
        bench_pi0(args, synth.WORKLOADS["pi05-b1"].with_(name="pi0-b1", prefix_len=(815,)))
        return
    wl = synth.WORKLOADS[args.workload]
    print("bench: workload %s, generating inputs" % wl.name, file=sys.stderr, flush=True)
    weights = synth.make_weights(wl)
    K, V = synth.make_prefix(wl)
    noise = synth.make_noise(wl)
    committed = synth.make_committed(wl) if wl.n_fixed else None

    torch.cuda.set_device(0)
    stream = torch.cuda.current_stream()
    ae = ActionExpert(wl.dims, wl.dtype, wl.batch, wl.prefix)
    ae.load_weights(weights)
    Kd, Vd = to_device(K), to_device(V)
    ae.bind_prefix(Kd, Vd, wl.valid_lengths(), stream=stream)
    ae.bind_state(None if committed is None else to_device(committed), wl.n_fixed, stream=stream)
    if args.committed_t0:
        ae.set_committed_t0(True)
    noise_d = to_device(noise)
    out = torch.empty_like(noise_d)
    torch.cuda.synchronize()

    if args.calls_only:
        ae.denoise(noise_d, wl.n_steps, out, stream=stream)
        for _ in range(args.calls_only):
            ae.denoise(noise_d, wl.n_steps, out, stream=stream)
        torch.cuda.synchronize()
        ae.sync(stream)
        print("bench: %d calls of %s done" % (args.calls_only + 1, wl.name), file=sys.stderr, flush=True)
        ae.close()
        return

    # first call: modulation tables + graph capture + one replay
    t0 = time.perf_counter()
    ae.denoise(noise_d, wl.n_steps, out, stream=stream)
    torch.cuda.synchronize()
    first_ms = (time.perf_counter() - t0) * 1e3
    print("bench: first call %.1f ms (tables + capture)" % first_ms, file=sys.stderr, flush=True)

    for _ in range(args.warmup):
        ae.denoise(noise_d, wl.n_steps, out, stream=stream)
    torch.cuda.synchronize()

    # timed region
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    per_call = []
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(args.steps)]
    torch.cuda.synchronize()
    ev0.record(stream)
    for i in range(args.steps):
        evs[i][0].record(stream)
        ae.denoise(noise_d, wl.n_steps, out, stream=stream)
        evs[i][1].record(stream)
    ev1.record(stream)
    torch.cuda.synchronize()
    # jpi_sync reports a producer wait of the single-launch kernel that timed
    # out (its output would be invalid): a failed call never counts as timed
    ae.sync(stream)
    timed_out = out.cpu().numpy()
    total_ms = ev0.elapsed_time(ev1)
    per_call = sorted(a.elapsed_time(b) for a, b in evs)
    ms_per_call = total_ms / args.steps
    value = wl.batch * args.steps / (total_ms / 1e3)
    print("bench: %.3f ms per call (median %.3f, p10 %.3f, p90 %.3f)"
          % (ms_per_call, per_call[len(per_call) // 2], per_call[len(per_call) // 10],
             per_call[(9 * len(per_call)) // 10]), file=sys.stderr, flush=True)

    counts = algorithmic_counts(wl)
    # timing pass: start/stop events on the dispatch of every launch of one kernel kind
    kinds = {"persistent": jpi.JPI_KERNEL_PERSISTENT, "qkv": jpi.JPI_KERNEL_QKV,
             "attention": jpi.JPI_KERNEL_ATTENTION, "oproj": jpi.JPI_KERNEL_OPROJ,
             "gateup": jpi.JPI_KERNEL_GATEUP, "down": jpi.JPI_KERNEL_DOWN}
    per_kind = {}
    reps = max(3, min(args.steps, 10))
    for kname, kind in kinds.items():
        jpi.check(jpi.jpi_debug_time_kernel(ae.ctx, kind), ae.ctx)
        tot_ms, tot_n = 0.0, 0
        for i in range(reps + 1):
            ae.denoise(noise_d, wl.n_steps, out, stream=stream)
            torch.cuda.synchronize()
            ae.sync(stream)
            st, ms, n = jpi.jpi_debug_kernel_time(ae.ctx)
            jpi.check(st, ae.ctx)
            if i > 0:  # the first call warms the eager path
                tot_ms += ms
                tot_n += n
        if tot_n == 0:  # this kind does not run on the path the workload takes
            continue
        avg_us = tot_ms / tot_n * 1e3
        entry = {"avg_us": round(avg_us, 3), "launches": tot_n,
                 "share_of_call": round(tot_ms / reps / ms_per_call, 4)}
        if kname in counts["kernel_bytes"]:
            entry["GBs"] = round(counts["kernel_bytes"][kname] / (avg_us * 1e-6) / 1e9, 1)
        per_kind[kname] = entry
    jpi.check(jpi.jpi_debug_time_kernel(ae.ctx, jpi.JPI_KERNEL_NONE), ae.ctx)
    kname = args.timed_kernel
    if kname == "auto":
        kname = "persistent" if "persistent" in per_kind else "gateup"
    k_avg_us = per_kind[kname]["avg_us"]
    tot_n = per_kind[kname]["launches"]
    kbytes = counts["kernel_bytes"][kname]
    achieved = kbytes / (k_avg_us * 1e-6) / 1e9
    print("bench: per-kernel %s" % json.dumps(per_kind), file=sys.stderr, flush=True)

    traffic = MEASURED_TRAFFIC.get((kernel_source_hash(), wl.name)) if kname == "persistent" else None
    traffic_source = ("rocprofv3 --pmc FETCH_SIZE / WRITE_SIZE on this kernel source (sha256 %s...), recorded in "
                      "profiles/traffic_%s_persistent.md" % (kernel_source_hash()[:12], wl.name)
                      if traffic is not None else
                      "none: no counter run on the current kernel source for this workload")
    call_gbs = counts["bytes_per_call"] / (ms_per_call * 1e-3) / 1e9
    call_tflops = counts["flops_per_call"] / (ms_per_call * 1e-3) / 1e12
    mfma_peak = BF16_MFMA_PEAK_TFLOPS if wl.dtype == "bf16" else FP32_MFMA_PEAK_TFLOPS
    result = {
        "metric": METRIC,
        "value": round(value, 3),
        "unit": "chunks/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_call, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": wl.dtype,
        "data": "synthetic",
        "config": {"workload": wl.name, "batch": wl.batch, "prefix_tokens": wl.prefix, "horizon": wl.dims.horizon,
                   "action_dim": wl.dims.action_dim, "euler_steps": wl.n_steps, "layers": wl.dims.n_layers,
                   "width": wl.dims.width, "heads": wl.dims.n_heads, "kv_heads": wl.dims.n_kv_heads,
                   "head_dim": wl.dims.head_dim, "mlp_dim": wl.dims.mlp_dim, "n_fixed": wl.n_fixed,
                   "committed_t0": bool(args.committed_t0), "seed": wl.seed},
        "per_euler_step_us": round(ms_per_call / wl.n_steps * 1e3, 2),
        "first_call_ms": round(first_ms, 2),
        "roofline": {"bound": "hbm", "kernel": ("k_persist (whole denoise call)" if kname == "persistent"
                                                else "GEMM (%s)" % kname), "achieved": round(achieved, 1),
                     "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4),
                     "traffic": traffic,
                     "traffic_source": traffic_source,
                     "bytes_per_launch": kbytes, "avg_launch_us": round(k_avg_us, 3),
                     "launches_timed": tot_n},
        "kernels": per_kind,
        "call_roofline": {"algorithmic_bytes": counts["bytes_per_call"], "achieved_GBs": round(call_gbs, 1),
                          "hbm_frac": round(call_gbs / HBM_PEAK_GBS, 4),
                          "algorithmic_flops": counts["flops_per_call"], "achieved_TFLOPs": round(call_tflops, 2),
                          "mfma_frac": round(call_tflops / mfma_peak, 4)},
    }
    ae.close()
    mp = measured_peaks()
    mp["hbm_frac_of_measured_copy"] = round(result["roofline"]["achieved"] / mp["copy_GBs"], 4) \
        if result["roofline"]["unit"] == "GB/s" else None
    result["measured_peaks"] = mp
    result["parity"] = {"checked": False, "why": "--no-cpu"}
    if not args.no_cpu:
        print("bench: timing the CPU oracle", file=sys.stderr, flush=True)
        result["cpu_baseline"], ref0 = cpu_baseline(wl, weights, K, V, noise, committed, bool(args.committed_t0))
        result["parity"] = check_output(timed_out[0], ref0, wl.dtype)
    print(json.dumps(result), flush=True)
    if not result["parity"].get("ok", True):
        print("bench: the timed output does not match the oracle (%s)" % json.dumps(result["parity"]),
              file=sys.stderr, flush=True)
        sys.exit(3)


if __name__ == "__main__":
    main()
