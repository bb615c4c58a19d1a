"""The oracle's pins have teeth: each of twelve plausible mistakes, planted
one at a time into a copy of the oracle, makes tests/test_oracle_pins.py fail.

Each case copies the oracle, the input generator, the pin tests and their
fixtures into a temporary tree, replaces one exact piece of
oracle/actionexpert.py (the replacement must apply), and runs the pins there
in a subprocess; the run must fail.  The unmodified copy must pass.
"""
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

# (name, exact text in oracle/actionexpert.py, replacement)
MUTATIONS = [
    ("rope sign", "x1 * s + x2 * c", "x1 * s - x2 * c"),
    ("modulation without 1 +", "* (1.0 + scale) + shift", "* scale + shift"),
    ("modulation split reversed",
     "return tuple(m[i * ex.W:(i + 1) * ex.W] for i in range(m.shape[0] // ex.W))",
     "return tuple(m[i * ex.W:(i + 1) * ex.W] for i in range(m.shape[0] // ex.W))[::-1]"),
    ("rope position ignores the prefix", "pos = pl + np.arange(S)", "pos = np.arange(S)"),
    ("logits not scaled", "s = (q @ K.T) / math.sqrt(Dh)", "s = (q @ K.T)"),
    ("mlp gate dropped", 'h = h + gate * (z @ w[p + "down.w"].T)', 'h = h + (z @ w[p + "down.w"].T)'),
    ("euler step sign", "dt = -1.0 / n_steps", "dt = 1.0 / n_steps"),
    ("step grid shifted", "return [1.0 - k / n_steps for k in range(n_steps)]",
     "return [1.0 - (k + 1) / n_steps for k in range(n_steps)]"),
    ("time mlp swish dropped", 'c = swish(w["time_mlp.0.w"] @ e + w["time_mlp.0.b"])',
     'c = w["time_mlp.0.w"] @ e + w["time_mlp.0.b"]'),
    ("sin / cos order", "return np.concatenate([np.cos(arg), np.sin(arg)])",
     "return np.concatenate([np.sin(arg), np.cos(arg)])"),
    ("suffix keys dropped", "K = np.concatenate([Kp[:prefix_len], ks], axis=0)",
     "K = np.concatenate([Kp[:prefix_len], ks * 0], axis=0)"),
    ("head-major reshape", "o[b] = np.transpose(ob, (1, 0, 2)).reshape(S, nH * Dh)",
     "o[b] = ob.reshape(S, nH * Dh)"),
]


def _tree(tmp, mutation=None):
    """A minimal copy of the repository with the oracle optionally mutated."""
    for d in ("oracle", "synth"):
        shutil.copytree(os.path.join(ROOT, d), os.path.join(tmp, d),
                        ignore=shutil.ignore_patterns("__pycache__", "*.tmp*"))
    os.makedirs(os.path.join(tmp, "tests"))
    for f in ("conftest.py", "test_oracle_pins.py"):
        shutil.copy(os.path.join(ROOT, "tests", f), os.path.join(tmp, "tests", f))
    shutil.copytree(os.path.join(ROOT, "tests", "golden"), os.path.join(tmp, "tests", "golden"),
                    ignore=shutil.ignore_patterns("*.npy", "*.npz", "__pycache__"))
    if mutation is not None:
        path = os.path.join(tmp, "oracle", "actionexpert.py")
        with open(path) as f:
            src = f.read()
        _, old, new = mutation
        assert src.count(old) == 1, "mutation site not found exactly once: %r" % old
        with open(path, "w") as f:
            f.write(src.replace(old, new))


def _pins_pass(tmp):
    env = dict(os.environ, PYTHONDONTWRITEBYTECODE="1")
    env.pop("PYTHONPATH", None)
    r = subprocess.run([sys.executable, "-m", "pytest", "tests/test_oracle_pins.py", "-x", "-q", "-p", "no:cacheprovider"],
                       cwd=tmp, env=env, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True, timeout=600)
    return r.returncode == 0, r.stdout[-2000:]


def test_unmutated_copy_passes_the_pins(tmp_path):
    _tree(str(tmp_path))
    ok, out = _pins_pass(str(tmp_path))
    assert ok, out


@pytest.mark.parametrize("mutation", MUTATIONS, ids=[m[0] for m in MUTATIONS])
def test_planted_mistake_fails_a_pin(tmp_path, mutation):
    _tree(str(tmp_path), mutation)
    ok, out = _pins_pass(str(tmp_path))
    assert not ok, "the pins did not catch: %s" % mutation[0]
