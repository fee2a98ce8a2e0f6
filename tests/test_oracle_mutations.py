"""The oracle's pins catch plausible mistakes.

Each case copies the oracle and its pin tests into a temporary directory, plants one
mistake in the copy (on the CPU; nothing here touches a GPU or the product path) and
runs the pins: they must fail.  The mistakes are the ones a reader of the paper could
plausibly make: the flatten order of vec(H_t), softmax instead of independent sigmoid
gates, a dropped normalisation, epsilon outside the square root, a RoPE sign, the
attention scale, gate and up swapped, the block positions off by one, the wrong key
weights, a dropped residual, an acceptance off-by-one, the argmax tie rule, the RMS
formula, the bf16 tie rule, and drafts taken from the anchor slot.
"""
import concurrent.futures as cf
import os
import shutil
import subprocess
import sys
import tempfile

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

MUTATIONS = [
    ("reducer.py", "x = H.reshape(n, m * d)", "x = H.transpose(0, 2, 1).reshape(n, m * d)"),
    ("reducer.py", "alpha = sigmoid(z) + gate_offset",
     "alpha = np.exp(z) / np.exp(z).sum(1, keepdims=True) + gate_offset"),
    ("reducer.py", "z = gate_scale * r * (x @ W.T) + b", "z = gate_scale * (x @ W.T) + b"),
    ("reducer.py", "r = 1.0 / np.sqrt(ms + eps)", "r = 1.0 / (np.sqrt(ms) + eps)"),
    ("drafter.py", "x2 * c + x1 * s], axis=1)", "x2 * c - x1 * s], axis=1)"),
    ("drafter.py", "s = (q @ k.T) / np.sqrt(hd)", "s = (q @ k.T) / hd"),
    ("drafter.py", "act = store(silu(gu[:, :W.F]) * gu[:, W.F:], dt)",
     "act = store(silu(gu[:, W.F:]) * gu[:, :W.F], dt)"),
    ("drafter.py", "pos = pos_shift + T + np.arange(B)", "pos = pos_shift + T - 1 + np.arange(B)"),
    ("drafter.py", "wk = W.w_qkv[l][d:2 * d]", "wk = W.w_qkv[l][0:d]"),
    ("drafter.py", "h = round_f32(h + o @ W.w_o[l].T)", "h = round_f32(o @ W.w_o[l].T)"),
    ("accept.py", "anchor[s] = target[s, n]", "anchor[s] = target[s, min(n + 1, K)]"),
    ("lm_head.py", "am = np.argmax(z32, axis=1)",
     "am = (z32.shape[1] - 1 - np.argmax(z32[:, ::-1], axis=1))"),
    ("numerics.py", "ms = np.mean(x * x, axis=-1, keepdims=True)",
     "ms = np.mean(np.abs(x), axis=-1, keepdims=True) ** 2"),
    ("numerics.py", "lsb = (u >> np.uint64(_DROP)) & np.uint64(1)", "lsb = np.uint64(1)"),
    ("step.py", "draft = am.reshape(len(seqs), B)[:, 1:]",
     "draft = am.reshape(len(seqs), B)[:, :-1]"),
]


def _run_mutant(i):
    fname, old, new = MUTATIONS[i]
    tmp = tempfile.mkdtemp(prefix="hdf_mut_")
    try:
        shutil.copytree(os.path.join(ROOT, "oracle"), os.path.join(tmp, "oracle"))
        shutil.copytree(os.path.join(ROOT, "synth"), os.path.join(tmp, "synth"))
        os.makedirs(os.path.join(tmp, "tests"))
        for f in ("conftest.py", "_tol.py", "test_oracle_pins.py"):
            shutil.copy(os.path.join(ROOT, "tests", f), os.path.join(tmp, "tests", f))
        shutil.copytree(os.path.join(ROOT, "tests", "golden"), os.path.join(tmp, "tests", "golden"))
        open(os.path.join(tmp, "tests", "__init__.py"), "w").close()
        path = os.path.join(tmp, "oracle", fname)
        src = open(path).read()
        assert old in src, (fname, old)
        open(path, "w").write(src.replace(old, new, 1))
        r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider",
                            os.path.join("tests", "test_oracle_pins.py")],
                           cwd=tmp, capture_output=True, text=True, timeout=300)
        return r.returncode
    finally:
        shutil.rmtree(tmp, ignore_errors=True)


def test_every_planted_mistake_fails_a_pin():
    with cf.ThreadPoolExecutor(4) as ex:
        codes = list(ex.map(_run_mutant, range(len(MUTATIONS))))
    missed = [MUTATIONS[i][2] for i, c in enumerate(codes) if c == 0]
    assert not missed, f"pins missed: {missed}"
