"""Mutation check of the oracle's pins.

Each entry below plants one plausible mistake in a copy of the oracle (a
transposed walk order, a dropped sign vector, a wrong tie order, GQA map or
forced block, a non-causal softmax row, ...). The oracle pins
(tests/test_oracle_*.py) then run against that copy in a child process, and at
least one of them must fail: a mistake no pin catches would mean the pins do
not fix that part of the oracle. The unmutated copy must pass, and every
planted mistake must still find its target text in the oracle source.
"""
import concurrent.futures
import glob
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
ORACLE = os.path.join(ROOT, "oracle", "sketchwalk_oracle.py")
HERE = os.path.basename(__file__)

# (name, text in the oracle, replacement)
MUTATIONS = [
    ("walk order transposed",
     "R = W.copy() if R_prev is None else R_prev @ W",
     "R = W.copy() if R_prev is None else W @ R_prev"),
    ("SRHT scale dropped",
     "return math.sqrt(d / r) * (Xbar @ DWS)",
     "return (Xbar @ DWS)"),
    ("partial block divided by B",
     "out[i] = seg.sum(axis=0) / seg.shape[0]",
     "out[i] = seg.sum(axis=0) / B"),
    ("tie order reversed",
     "order = sorted(cand, key=lambda j: (-float(values[j]), j))",
     "order = sorted(cand, key=lambda j: (-float(values[j]), -j))"),
    ("causal mask dropped in attention",
     "logits = np.where(toks[None, :] <= rows[:, None], logits, -np.inf)",
     "pass"),
    ("power one too high",
     "    for _ in range(int(s) - 1):\n        W = W * X",
     "    for _ in range(int(s)):\n        W = W * X"),
    ("decode column update dropped",
     "st.A[:b_q + 1, b_cur] = (Qs @ Ks[b_cur]) / math.sqrt(r)",
     "pass"),
    ("budget in floating point",
     "t = (avail * pct + 99) // 100",
     "t = math.ceil(avail * pct / 100.0 * 1.0000001)"),
    ("SRHT signs dropped",
     "DWS = (signs[:, None] * W)[:, cols]",
     "DWS = W[:, cols]"),
    ("block scores transposed",
     "A = (Qs @ Ks.T) / math.sqrt(r)",
     "A = (Ks @ Qs.T) / math.sqrt(r)"),
    ("causal block mask dropped",
     "        A = np.tril(A)\n    return A",
     "        pass\n    return A"),
    ("decode open block never restarts",
     "    if p % B == 0:\n        st.qtok",
     "    if p % B == 1:\n        st.qtok"),
    ("decode query representative from keys",
     "st.qbar[b_q] = block_means(st.qtok, B)[0]",
     "st.qbar[b_q] = block_means(st.ktok, B)[0]"),
    ("decode prompt tokens of the open block dropped",
     "first = (b - 1) * B                      # first token of the last block",
     "first = n - 1"),
    ("prompt score matrix placed transposed",
     'A[:b, :b] = sk["A"]',
     'A[:b, :b] = sk["A"].T'),
    ("decode row without 1/sqrt(r)",
     "st.A[b_q, :b_cur + 1] = (Ks @ q_t) / math.sqrt(r)",
     "st.A[b_q, :b_cur + 1] = (Ks @ q_t)"),
    ("GQA map u % h_kv",
     "    g = u // G\n    sc = (1.0 / math.sqrt(d)) if scale is None else scale\n    rows",
     "    g = u % K.shape[0]\n    sc = (1.0 / math.sqrt(d)) if scale is None else scale\n    rows"),
    ("forced last block is i - 1",
     "        F.add(i)",
     "        F.add(max(0, i - 1))"),
    ("clipped power uses |A|",
     "return walk_weights(np.maximum(A, 0.0), c, s)",
     "return walk_weights(np.abs(A), c, s)"),
    ("clipped power keeps the negative part",
     "return walk_weights(np.maximum(A, 0.0), c, s)",
     "return walk_weights(np.minimum(A, 0.0), c, s)"),
    ("softmax row not causal",
     "        z = logit_scale * A[i, :i + 1]\n        e = np.exp(z - np.max(z))\n"
     "        W[i, :i + 1] = e / e.sum()",
     "        z = logit_scale * A[i, :]\n        e = np.exp(z - np.max(z))\n"
     "        W[i, :i + 1] = (e / e.sum())[:i + 1]"),
    ("softmax logit scale dropped",
     "        z = logit_scale * A[i, :i + 1]",
     "        z = A[i, :i + 1]"),
    ("softmax normaliser dropped",
     "        W[i, :i + 1] = e / e.sum()",
     "        W[i, :i + 1] = e"),
    ("matrix power transposed factor",
     "        W = W @ X\n",
     "        W = W @ X.T\n"),
    ("matrix power one too high",
     "    for _ in range(int(s) - 1):\n        W = W @ X",
     "    for _ in range(int(s)):\n        W = W @ X"),
    ("matrix power taken element-wise",
     "        W = W @ X\n",
     "        W = W * X\n"),
    ("clipped power dispatched to the plain power",
     "    if variant == WALK_RELU:\n        return walk_weights_relu(A, c, s)",
     "    if variant == WALK_RELU:\n        return walk_weights(A, c, s)"),
    ("decode ignores the walk variant",
     "    W = walk_weights_variant(variant, st.A[:b_cur + 1, :b_cur + 1], st.c, s)",
     "    W = walk_weights(st.A[:b_cur + 1, :b_cur + 1], st.c, s)"),
]

CONFTEST = """import os, sys
HERE = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, HERE)
"""


def _tree(base: str, source: str) -> str:
    """A copy of the oracle package (with `source` as its module) and of the
    oracle pins under `base`."""
    pkg = os.path.join(base, "oracle")
    tst = os.path.join(base, "tests")
    os.makedirs(pkg)
    os.makedirs(tst)
    shutil.copy(os.path.join(ROOT, "oracle", "__init__.py"), pkg)
    with open(os.path.join(pkg, "sketchwalk_oracle.py"), "w") as f:
        f.write(source)
    for p in glob.glob(os.path.join(ROOT, "tests", "test_oracle_*.py")):
        if os.path.basename(p) != HERE:
            shutil.copy(p, tst)
    shutil.copytree(os.path.join(ROOT, "tests", "golden"), os.path.join(tst, "golden"))
    with open(os.path.join(tst, "conftest.py"), "w") as f:
        f.write(CONFTEST)
    return base


def _run_pins(base: str) -> int:
    env = dict(os.environ, PYTHONDONTWRITEBYTECODE="1", OMP_NUM_THREADS="2")
    env.pop("PYTHONPATH", None)
    res = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider",
                          "tests"], cwd=base, env=env, capture_output=True, text=True,
                         timeout=600)
    return res.returncode


def test_every_mutation_targets_the_current_oracle():
    src = open(ORACLE).read()
    missing = [name for name, a, _ in MUTATIONS if a not in src]
    assert not missing, missing


def test_every_planted_mistake_is_caught_by_a_pin(tmp_path):
    src = open(ORACLE).read()
    jobs = [("unmutated", src)] + [(name, src.replace(a, b, 1)) for name, a, b in MUTATIONS]
    bases = [_tree(str(tmp_path / f"m{i}"), s) for i, (_, s) in enumerate(jobs)]
    with concurrent.futures.ThreadPoolExecutor(max_workers=4) as ex:
        codes = list(ex.map(_run_pins, bases))
    assert codes[0] == 0, "the unmutated copy of the oracle fails its pins"
    # exit status 1: tests ran and some failed (not a collection or usage error)
    missed = [name for (name, _), rc in zip(jobs[1:], codes[1:]) if rc != 1]
    assert not missed, f"planted mistakes no pin catches (or that break collection): {missed}"
