"""Critical path of the single-launch denoise kernel, link by link.

``--build`` (on any host with hipcc) builds a copy of libjpi with the
persistent kernel's trace mode (-DJPI_PERSIST_TRACE=1: every workgroup stamps
the real-time counter at the end of every phase) as
paper_2607_12659_amd/libjpi_trace.so.  Without it, the script (on the GPU)
runs one workload through that library and prints, for each of the eight phases of a layer, the median
over all (step, layer) pairs of

    link(p) = last workgroup to finish phase p  -  last to finish phase p - 1

(the time from the last producer of the previous phase finishing to the last
workgroup of this phase finishing), split for the workgroup that finished
last into waiting for its producers' flags, loading its operands, and the
rest (compute, stores and their confirmation), plus the sum per layer and
the whole call.  The trace build is for measurement only; the stamps cost one store per
workgroup and phase.

    python -m paper_2607_12659_amd.trace_links --build
    python -m paper_2607_12659_amd.trace_links [--workload pi05-b1] [--calls 3] [--json OUT]
"""
from __future__ import annotations

import argparse
import json
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
TRACE_LIB = os.path.join(HERE, "libjpi_trace.so")
PHASES = ["rows -> QKV", "QKV -> attention", "attention -> combine", "combine -> O-proj", "O-proj -> rows",
          "rows -> GateUp", "GateUp -> Down", "Down -> rows"]


def build_trace_lib() -> str:
    from paper_2607_12659_amd import build as b
    bdir = os.path.join(ROOT, "_build", "trace")
    os.makedirs(bdir, exist_ok=True)
    objs = []
    for src in b.SOURCES:
        obj = os.path.join(bdir, os.path.splitext(src)[0] + ".o")
        b._run([b.HIPCC, *b.FLAGS, "-DJPI_PERSIST_TRACE=1", "-c", os.path.join(b.CSRC, src), "-o", obj])
        objs.append(obj)
    tmp = TRACE_LIB + ".tmp%d" % os.getpid()
    b._run([b.HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", *objs, "-o", tmp])
    os.replace(tmp, TRACE_LIB)
    return TRACE_LIB


def analyse(stamps, ticks_per_us, n_steps, n_layers):
    """Per-link durations (us) from the stamps [workgroups][1 + 3 phases].

    Returns [steps][layers][8][4]: the link (last workgroup to finish this
    phase minus last to finish the previous one) and, for the workgroup that
    finished last, its split into waiting for the producers' flags, loading
    the operands, and the rest (compute, stores, store confirmation)."""
    import numpy as np
    n = n_steps * n_layers * 8
    st = stamps[:, 1:1 + 3 * n].astype(np.float64).reshape(stamps.shape[0], n, 3)
    end = st[:, :, 2]
    crit = end.argmax(axis=0)                                      # workgroup that finished last
    t_end = end.max(axis=0)
    start = float(stamps[:, 0].astype(np.float64).min())
    prev = np.concatenate([[start], t_end[:-1]])
    seen = st[crit, np.arange(n), 0]
    loaded = st[crit, np.arange(n), 1]
    out = np.stack([t_end - prev, np.maximum(seen - prev, 0.0), loaded - np.maximum(seen, prev),
                    t_end - loaded], axis=1) / ticks_per_us
    return out.reshape(n_steps, n_layers, 8, 4)


def run(workload: str, calls: int):
    import numpy as np
    import torch

    import synth
    from paper_2607_12659_amd import jpi
    from paper_2607_12659_amd.expert import ActionExpert, to_device

    wl = synth.WORKLOADS[workload]
    ae = ActionExpert(wl.dims, wl.dtype, wl.batch, wl.prefix)
    ae.load_weights(synth.make_weights(wl))
    K, V = synth.make_prefix(wl)
    ae.bind_prefix(to_device(K), to_device(V), wl.valid_lengths())
    ae.bind_state(None if not wl.n_fixed else to_device(synth.make_committed(wl)), wl.n_fixed)
    noise = to_device(synth.make_noise(wl))
    links = []
    for i in range(calls + 1):
        ae.denoise(noise, wl.n_steps)
        ae.sync()
        torch.cuda.synchronize()
        st, stamps, tpu = jpi.jpi_debug_persist_trace(ae.ctx)
        jpi.check(st, ae.ctx)
        if i > 0:  # the first call builds tables and captures the graph
            links.append(analyse(stamps, tpu, wl.n_steps, wl.dims.n_layers))
    ae.close()
    link = np.stack(links)                                          # [calls][steps][layers][8][4]
    med = np.median(link.reshape(-1, 8, 4), axis=0)
    per_layer = np.median(link[..., 0].sum(axis=3).reshape(-1))
    call_us = float(np.median(link[..., 0].sum(axis=(1, 2, 3))))
    return {"workload": workload, "calls": calls,
            "links": {PHASES[i]: {"link": round(float(med[i, 0]), 2), "wait": round(float(med[i, 1]), 2),
                                  "load": round(float(med[i, 2]), 2), "rest": round(float(med[i, 3]), 2)}
                      for i in range(8)},
            "layer_us_median": round(float(per_layer), 2), "call_us_median": round(call_us, 1)}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--workload", default="pi05-b1")
    ap.add_argument("--calls", type=int, default=3)
    ap.add_argument("--json", default="")
    ap.add_argument("--build", action="store_true", help="build libjpi_trace.so and exit")
    ap.add_argument("--child", action="store_true", help=argparse.SUPPRESS)
    args = ap.parse_args()
    if args.build:
        print(build_trace_lib())
        return
    if not args.child:
        if not os.path.exists(TRACE_LIB):
            sys.exit("%s is not built: run with --build first" % TRACE_LIB)
        env = dict(os.environ, JPI_LIB=TRACE_LIB)
        cmd = [sys.executable, "-m", "paper_2607_12659_amd.trace_links", "--child", "--workload", args.workload,
               "--calls", str(args.calls)] + (["--json", args.json] if args.json else [])
        sys.exit(subprocess.call(cmd, env=env, cwd=ROOT))
    sys.path.insert(0, ROOT)
    res = run(args.workload, args.calls)
    print("| link | median us | critical workgroup: wait for flags | load operands | compute + stores |")
    print("|---|---|---|---|---|")
    for k, v in res["links"].items():
        print("| %s | %.2f | %.2f | %.2f | %.2f |" % (k, v["link"], v["wait"], v["load"], v["rest"]))
    print("| one layer (sum) | %.2f | | | |" % res["layer_us_median"])
    print("| whole call | %.1f | | | |" % res["call_us_median"])
    if args.json:
        with open(args.json, "w") as f:
            json.dump(res, f, indent=1)


if __name__ == "__main__":
    main()
