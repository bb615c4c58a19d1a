"""The stored oracle outputs under tests/golden/ were made by the current
oracle and generator (make_golden.py records source hashes), and one of them
is re-derived here from scratch."""
import glob
import json
import os
import sys

import numpy as np
import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.join(HERE, "golden"))
import make_golden  # noqa: E402

ROOT = os.path.dirname(HERE)


def _metas():
    out = []
    for p in sorted(glob.glob(os.path.join(HERE, "golden", "*.json"))):
        with open(p) as f:
            m = json.load(f)
        if "oracle_sha256" in m:
            out.append((os.path.basename(p)[:-5], m))
    return out


def test_every_case_has_a_golden():
    names = {n for n, _ in _metas()}
    assert set(make_golden.CASES) <= names
    for n in make_golden.VLM_CASES:
        assert os.path.exists(os.path.join(HERE, "golden", n + ".npz"))


@pytest.mark.parametrize("name", sorted(make_golden.VLM_CASES))
def test_vlm_golden_made_by_current_sources(name):
    with open(os.path.join(HERE, "golden", name + ".json")) as f:
        meta = json.load(f)
    assert meta["vlm_oracle_sha256"] == make_golden.source_hash(*make_golden.vlm_oracle_files()), \
        "VLM oracle changed since %s was generated: rerun tests/golden/make_golden.py %s" % (name, name)
    assert meta["vlm_synth_sha256"] == make_golden.source_hash(*make_golden.vlm_synth_files())
    g = np.load(os.path.join(HERE, "golden", name + ".npz"), allow_pickle=False)
    L, T = meta["n_layers"], len(meta["tokens"])
    assert g["K"].shape == (L, T, 256) and g["V"].shape == (L, T, 256) and g["hidden"].shape == (T, 2048)
    assert list(g["tokens"]) == meta["tokens"] and meta["tokens"][0] == 0 and meta["tokens"][-1] == meta["prefix"] - 1
    assert all(np.isfinite(g[k]).all() for k in ("K", "V", "hidden"))


@pytest.mark.parametrize("name,meta", _metas())
def test_golden_made_by_current_sources(name, meta):
    assert meta["oracle_sha256"] == make_golden.source_hash(*make_golden.oracle_files(name)), \
        "oracle changed since %s was generated: rerun tests/golden/make_golden.py" % name
    assert meta["synth_sha256"] == make_golden.source_hash(os.path.join(ROOT, "synth", "synth.c"),
                                                           os.path.join(ROOT, "synth", "__init__.py"))
    if meta.get("variant"):
        assert meta["variant_synth_sha256"] == make_golden.source_hash(os.path.join(ROOT, "synth", "pi0.py"))
    if meta.get("n_corr"):
        assert meta["item_sha256"] == make_golden.source_hash(os.path.join(ROOT, "synth", "correction.py"))
    arr = np.load(os.path.join(HERE, "golden", name + ".npy"), allow_pickle=False)
    assert arr.shape == (len(meta["rollouts"]), 50, 32) and np.isfinite(arr).all()


@pytest.mark.slow
def test_regenerate_ragged_golden_bitwise(tmp_path, monkeypatch):
    name = "pi05-b2-ragged"
    ref = np.load(os.path.join(HERE, "golden", name + ".npy"), allow_pickle=False)
    monkeypatch.setattr(make_golden, "HERE", str(tmp_path))
    make_golden.make(name)
    assert np.array_equal(np.load(os.path.join(tmp_path, name + ".npy")), ref)
