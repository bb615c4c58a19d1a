"""Write the oracle's outputs for the large workloads to tests/golden/.

Calls only the CPU oracle and the seeded input generator.  Each output file
``<name>.npy`` holds the fp64 actions [rollouts][H][A]; ``<name>.json`` records
how it was made (workload, rollouts, seed, n_steps, dtype, sha256 of the
oracle source and of the generator source at generation time).

    python tests/golden/make_golden.py [name ...]
"""
from __future__ import annotations

import hashlib
import json
import os
import sys
import time

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
sys.path.insert(0, ROOT)

import oracle  # noqa: E402
import synth  # noqa: E402
from synth import correction as synth_corr  # noqa: E402
from synth import pi0 as synth_pi0  # noqa: E402

# name -> (workload key, overrides, rollouts evaluated)
CASES = {
    "pi05-b1": ("pi05-b1", {}, None),
    "pi05-b1-committed10": ("pi05-b1-committed10", {}, None),
    "pi05-b8": ("pi05-b8", {}, None),
    "pi05-b64-p1600": ("pi05-b64-p1600", {}, None),
    # not a benchmark workload: the pi0.5 shape in fp32, checked at 1e-4 so that
    # attention or norm mistakes cannot hide inside the bf16 tolerance
    "pi05-f32-b1": ("pi05-b1", {"dtype": "f32", "name": "pi05-f32-b1"}, None),
    # ragged prefix lengths (masked slots) over two rollouts
    "pi05-b2-ragged": ("pi05-b8", {"batch": 2, "prefix_len": (816, 301), "name": "pi05-b2-ragged"}, None),
    # the correction item of the future correction module (4 tokens) ahead of the
    # action tokens, with the committed rows of the same call
    "pi05-b1-committed10-corr4": ("pi05-b1-committed10", {"name": "pi05-b1-committed10-corr4"}, None),
    # the variant in which the committed rows carry flow time t = 0
    "pi05-b1-committed10-t0": ("pi05-b1-committed10", {"name": "pi05-b1-committed10-t0"}, None),
    # modulation tensors x 8: gates near 0.5 instead of 0.06, so that every
    # sublayer (attention above all) moves the actions far beyond the bf16 bar
    "pi05-b1-amp8": ("pi05-b1", {"name": "pi05-b1-amp8", "mod_gain": 8.0}, None),
}
# cases whose metadata also records the oracle's own output on the same inputs
# with the prefix V negated (how far a broken attention would move the actions)
SENSITIVITY = {"pi05-b1-amp8"}
# cases whose expert call also gets correction tokens: name -> tokens per rollout
CORR_TOKENS = {"pi05-b1-committed10-corr4": 4}
# cases run with the committed rows at t = 0
COMMITTED_T0 = {"pi05-b1-committed10-t0"}
# cases of the pi0-style expert variant (its own oracle, weights and robot state)
PI0 = {"pi0-b1": ("pi05-b1-committed10", {"name": "pi0-b1", "prefix_len": (815,)}, None)}
CASES.update(PI0)


def source_hash(*paths):
    h = hashlib.sha256()
    for p in paths:
        with open(p, "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def workload(name):
    key, over, rollouts = CASES[name]
    return synth.WORKLOADS[key].with_(**over), rollouts


def oracle_files(name):
    """Oracle sources a stored output depends on (their sha256 is recorded)."""
    if name in PI0:
        return [os.path.join(ROOT, "oracle", "actionexpert.py"), os.path.join(ROOT, "oracle", "pi0.py")]
    return [os.path.join(ROOT, "oracle", "actionexpert.py")]


def make(name):
    wl, rollouts = workload(name)
    rl = list(range(wl.batch)) if rollouts is None else rollouts
    t0 = time.time()
    w = synth_pi0.make_pi0_weights(wl) if name in PI0 else synth.make_weights(wl)
    K, V = synth.make_prefix(wl, rl)
    noise = synth.make_noise(wl, rl)
    com = synth.make_committed(wl, rl) if wl.n_fixed else None
    lens = [wl.valid_lengths()[b] for b in rl]
    n_corr = CORR_TOKENS.get(name, 0)
    corr = synth_corr.make_item(wl.seed, wl.batch, n_corr, wl.dims.width, rl) if n_corr else None
    at_t0 = name in COMMITTED_T0
    t1 = time.time()
    if name in PI0:
        out = oracle.pi0.denoise(wl.dims, w, noise, K, V, lens, wl.n_steps, synth_pi0.make_state(wl, rl),
                                 committed=com, n_fixed=wl.n_fixed)
    else:
        ex = oracle.Expert(wl.dims, w)
        out = oracle.denoise(ex, noise, K, V, lens, wl.n_steps, committed=com, n_fixed=wl.n_fixed, corr=corr,
                             committed_t0=at_t0)
    t2 = time.time()
    flip = None
    if name in SENSITIVITY:
        ex = oracle.Expert(wl.dims, w)
        alt = oracle.denoise(ex, noise, K, V ^ np.uint16(0x8000), lens, wl.n_steps, committed=com,
                             n_fixed=wl.n_fixed)
        num = np.sqrt(((alt - out) ** 2).reshape(len(rl), -1).sum(1))
        den = np.sqrt((out ** 2).reshape(len(rl), -1).sum(1))
        flip = float((num / den).min())
    np.save(os.path.join(HERE, name + ".npy"), out, allow_pickle=False)
    meta = {"workload": wl.name, "base_workload": CASES[name][0], "overrides": {k: list(v) if isinstance(v, tuple) else v
                                                                             for k, v in CASES[name][1].items()},
            "rollouts": rl, "seed": wl.seed, "n_steps": wl.n_steps, "n_fixed": wl.n_fixed, "dtype": wl.dtype,
            "prefix": wl.prefix, "prefix_len": lens,
            "oracle_sha256": source_hash(*oracle_files(name)),
            "synth_sha256": source_hash(os.path.join(ROOT, "synth", "synth.c"),
                                        os.path.join(ROOT, "synth", "__init__.py")),
            "oracle_seconds": round(t2 - t1, 2), "setup_seconds": round(t1 - t0, 2),
            "n_corr": n_corr, "committed_t0": at_t0, "mod_gain": wl.mod_gain,
            "made_by": "tests/golden/make_golden.py (oracle + synth only)"}
    if flip is not None:
        meta["prefix_v_negated_rel_l2"] = flip
    if n_corr:
        meta["item_sha256"] = source_hash(os.path.join(ROOT, "synth", "correction.py"))
    if name in PI0:
        meta["variant"] = "action_time"
        meta["variant_synth_sha256"] = source_hash(os.path.join(ROOT, "synth", "pi0.py"))
    with open(os.path.join(HERE, name + ".json"), "w") as f:
        json.dump(meta, f, indent=1)
    print("%s: oracle %.1fs setup %.1fs" % (name, t2 - t1, t1 - t0), flush=True)




# ---------------------------------------------------------------------------
# VLM prefill (the LLM pass that writes the expert's prefix KV) at full depth
# ---------------------------------------------------------------------------
# name -> (VLM workload key, number of sampled token positions)
VLM_CASES = {"gemma2b-p816-l18": ("gemma2b-p816", 32)}


def vlm_oracle_files():
    return [os.path.join(ROOT, "oracle", "vlm.py"), os.path.join(ROOT, "oracle", "actionexpert.py")]


def vlm_synth_files():
    return [os.path.join(ROOT, "synth", "synth.c"), os.path.join(ROOT, "synth", "__init__.py"),
            os.path.join(ROOT, "synth", "vlm.py")]


def make_vlm(name):
    """All layers of the prefill run in the oracle; K and V of every layer and
    the final hidden state are stored at evenly spaced token positions (first
    and last included) as float32 in ``<name>.npz``."""
    import synth.vlm as synth_vlm
    key, n_tok = VLM_CASES[name]
    vwl = synth_vlm.VLM_WORKLOADS[key]
    t0 = time.time()
    vw = synth_vlm.make_vlm_weights(vwl)
    emb = synth_vlm.make_embeddings(vwl)
    t1 = time.time()
    K, V, hid = oracle.vlm_prefill(vwl.dims, vw, emb[0])
    t2 = time.time()
    tok = np.unique(np.round(np.linspace(0, vwl.prefix - 1, n_tok)).astype(np.int64))
    np.savez(os.path.join(HERE, name + ".npz"), tokens=tok, K=K[:, tok].astype(np.float32),
             V=V[:, tok].astype(np.float32), hidden=hid[tok].astype(np.float32))
    meta = {"kind": "vlm_prefill", "workload": vwl.name, "n_layers": vwl.dims.n_layers, "prefix": vwl.prefix,
            "seed": vwl.seed, "tokens": tok.tolist(),
            "vlm_oracle_sha256": source_hash(*vlm_oracle_files()),
            "vlm_synth_sha256": source_hash(*vlm_synth_files()),
            "oracle_seconds": round(t2 - t1, 2), "setup_seconds": round(t1 - t0, 2),
            "made_by": "tests/golden/make_golden.py (oracle + synth only)"}
    with open(os.path.join(HERE, name + ".json"), "w") as f:
        json.dump(meta, f, indent=1)
    print("%s: oracle %.1fs setup %.1fs" % (name, t2 - t1, t1 - t0), flush=True)


if __name__ == "__main__":
    names = sys.argv[1:] or list(CASES) + list(VLM_CASES)
    for n in names:
        make_vlm(n) if n in VLM_CASES else make(n)
