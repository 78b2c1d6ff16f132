"""The oracle's pins catch plausible mistakes: each case plants one mistake
in a copy of the oracle (on the CPU, in a temporary directory) and runs the
pin tests against that copy; at least one pin must fail.  The library's own
comparisons are left out of these runs (a mutated oracle disagrees with the
library trivially), so only the pins against the paper's definitions and the
mathematics count."""

import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

# (name, oracle file, original text, planted mistake, pin file)
MUTATIONS = [
    ("zero point sign", "quant.py", "z = np.clip(np.rint(-lo / s16), 0, qmax)",
     "z = np.clip(np.rint(lo / s16), 0, qmax)", "test_oracle.py"),
    ("grid without 0", "quant.py", "lo = np.minimum(Wg.min(axis=2), 0.0)", "lo = Wg.min(axis=2)", "test_oracle.py"),
    ("floor for rint", "quant.py", "q = np.clip(np.rint(Wg / s16[:, :, None])",
     "q = np.clip(np.floor(Wg / s16[:, :, None])", "test_oracle.py"),
    ("unrounded scale", "quant.py", "s16 = fp16_rne(s).astype(np.float64)", "s16 = s.copy()", "test_oracle.py"),
    ("bit order within a code", "quant.py", "bitstr = ((c[:, :, None] >> np.arange(bits)) & 1)",
     "bitstr = ((c[:, :, None] >> np.arange(bits)[::-1]) & 1)", "test_oracle.py"),
    ("straddling code loses its high word", "quant.py", "w1 = np.minimum(w0 + 1, nw - 1)", "w1 = w0",
     "test_oracle.py"),
    ("dequant without the zero point", "quant.py", "return s * (codes - z)", "return s * codes", "test_oracle.py"),
    ("sign of the correction", "linear.py", "Y = Y + T @ B.T", "Y = Y - T @ B.T", "test_oracle.py"),
    ("factor rows off by one", "linear.py", "A = np.asarray(A, dtype=np.float64)[:r]",
     "A = np.asarray(A, dtype=np.float64)[1:r + 1]", "test_oracle.py"),
    ("SiLU sign", "linear.py", "return v / (1.0 + np.exp(-v))", "return v / (1.0 + np.exp(v))", "test_oracle.py"),
    ("factor scaling", "comp.py", "root = np.sqrt(sigma[:r_max])", "root = sigma[:r_max]", "test_oracle.py"),
    ("residual sign", "comp.py",
     "return np.asarray(W, dtype=np.float64) - np.asarray(W_hat, dtype=np.float64)",
     "return np.asarray(W_hat, dtype=np.float64) - np.asarray(W, dtype=np.float64)", "test_oracle.py"),
    ("wrong expert rank", "moe.py", "r = int(ranks[e]) if slot_ranks is None",
     "r = int(ranks[(e + 1) % len(ranks)]) if slot_ranks is None", "test_oracle.py"),
    ("slot rank ignored", "moe.py", "else int(slot_ranks[t][j])", "else int(ranks[e])", "test_oracle.py"),
    ("knee excludes its index", "ranks.py", "    s_sum = 0.0\n    for v in sigma[:r]:",
     "    r = r - 1 if r > 1 else r\n    s_sum = 0.0\n    for v in sigma[:r]:", "test_ranks.py"),
    ("curvature of the raw spectrum", "ranks.py", "        k = hat[j - 2] - 2.0 * hat[j - 1] + hat[j]",
     "        k = sigma[j - 2] - 2.0 * sigma[j - 1] + sigma[j]", "test_ranks.py"),
    ("level ties round up", "ranks.py", "        if abs(x - lv) < abs(x - best):",
     "        if abs(x - lv) <= abs(x - best):", "test_ranks.py"),
    ("residual ranks shared first", "ranks.py",
     "    stage1 = _proportional(r_cont, [float(c) for c in sal], total)",
     "    stage1 = _proportional(r_cont, [float(lens[i] - sal[i]) for i in range(n)], total)", "test_ranks.py"),
    ("layer score against the maximum", "ranks.py", "    dmin = min(float(D[l]) for l in top)",
     "    dmin = max(float(D[l]) for l in top)", "test_ranks.py"),
    ("recoverability inverted", "ranks.py", "    return r, (s_mean / r_mean if r_mean > 0.0 else math.inf)",
     "    return r, (r_mean / s_mean if r_mean > 0.0 else math.inf)", "test_ranks.py"),
    ("sensitivities not normalised", "ranks.py",
     "    S = [(float(d) / dsum if dsum > 0.0 else 1.0 / n) for d in sens]", "    S = [float(d) for d in sens]",
     "test_ranks.py"),
    ("knee ties take the last", "ranks.py", "        if k > best:", "        if k >= best:", "test_ranks.py"),
]


def _copy_tree(dst):
    for d in ("oracle", "tests"):
        shutil.copytree(os.path.join(ROOT, d), os.path.join(dst, d),
                        ignore=shutil.ignore_patterns("__pycache__", "test_oracle_mutations.py"))
    # the Python side of the package (input generators, binding); no library
    pkg = os.path.join(dst, "paper_2605_05819_amd")
    os.makedirs(pkg)
    for f in os.listdir(os.path.join(ROOT, "paper_2605_05819_amd")):
        if f.endswith(".py"):
            shutil.copy(os.path.join(ROOT, "paper_2605_05819_amd", f), pkg)
    shutil.copy(os.path.join(ROOT, "pytest.ini"), dst)


@pytest.mark.parametrize("name,fname,old,new,pins", MUTATIONS, ids=[m[0] for m in MUTATIONS])
def test_planted_mistake_fails_a_pin(tmp_path, name, fname, old, new, pins):
    _copy_tree(str(tmp_path))
    path = os.path.join(str(tmp_path), "oracle", fname)
    src = open(path).read()
    assert src.count(old) == 1, "the oracle no longer holds the text this mutation replaces"
    open(path, "w").write(src.replace(old, new))
    args = [sys.executable, "-m", "pytest", "-q", "-x", "-p", "no:cacheprovider", "-m", "not gpu",
            os.path.join("tests", pins)]
    if pins == "test_ranks.py":
        args += ["-k", "not library and not validation"]
    env = dict(os.environ, PYTHONDONTWRITEBYTECODE="1")
    r = subprocess.run(args, cwd=str(tmp_path), capture_output=True, text=True, env=env, timeout=600)
    assert r.returncode == 1, "planted mistake '%s' passed every pin:\n%s" % (name, r.stdout[-2000:])
