"""Each plausible slip in the oracle (a dropped term, a flipped sign, a wrong index
or tie rule, a transposed operand) must make at least one oracle pin fail.

Mutants are planted in a copy of the oracle on the CPU; the pins run against that
copy in a subprocess."""
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

MUTANTS = [
    ("frontier gate sign", "sigmoid((c_hat - th + w) / ta) * sigmoid((th - c_hat) / ta)",
     "sigmoid((c_hat - th - w) / ta) * sigmoid((th - c_hat) / ta)"),
    ("progress factor dropped", "return F * P, F, P, v_bar, c_hat", "return F, F, P, v_bar, c_hat"),
    ("progress sign", "sigmoid((_p64(v_ref) - np.asarray(v_bar, dtype=np.float64)) / _p64(tau))",
     "sigmoid((np.asarray(v_bar, dtype=np.float64) - _p64(v_ref)) / _p64(tau))"),
    ("velocity not clipped", "v_bar = np.minimum(np.maximum(v, -w / 2.0), w / 2.0)", "v_bar = v"),
    ("forecast ignores velocity", "np.minimum(np.maximum(c1 + v_bar, 0.0), 1.0), c1)",
     "np.minimum(np.maximum(c1, 0.0), 1.0), c1)"),
    ("d <= 1 read as d < 1", "np.where(dist <= 1, k_base + delta_role", "np.where(dist < 1, k_base + delta_role"),
    ("distance without abs", "d[lo:hi] = np.abs(b[lo:hi] - int(active_block[s]))",
     "d[lo:hi] = (b[lo:hi] - int(active_block[s]))"),
    ("FPS ties to higher token", "order = np.lexsort((np.asarray(token), -np.asarray(score, dtype=np.float64)))",
     "order = np.lexsort((-np.asarray(token), -np.asarray(score, dtype=np.float64)))"),
    ("ranking ascending", "order = np.lexsort((np.asarray(token), -np.asarray(score, dtype=np.float64)))",
     "order = np.lexsort((np.asarray(token), np.asarray(score, dtype=np.float64)))"),
    ("outer groups rounded up", "n_q = int(np.floor(_p64(q) * m))", "n_q = int(np.ceil(_p64(q) * m))"),
    ("no clamp", "k = np.minimum(np.maximum(k, p.k_min), p.k_max)", "k = k"),
    ("tokens without history ranked", "Jp = J[hist[J] >= 1]", "Jp = J"),
    ("TopK ties to higher expert", "order = np.lexsort((e_idx, -row))", "order = np.lexsort((-e_idx, -row))"),
    ("alpha not renormalised", "den = num.sum() if norm_topk else np.exp(row - rmax).sum()",
     "den = np.exp(row - rmax).sum()"),
    ("SiLU on the up projection", "a = g * sigmoid(g) * u", "a = g * sigmoid(u) * u"),
    ("down projection transposed", "return a @ wd.T", "return a @ wd"),
    ("pairs sorted by token first", "order = np.lexsort((pair_token, pair_expert))",
     "order = np.lexsort((pair_expert, pair_token))"),
    ("FLOPs per pair 4hd", "return 6 * int(d) * int(f) * int(pairs)", "return 4 * int(d) * int(f) * int(pairs)"),
    ("router bias dropped", "r = r + np.asarray(bias, dtype=np.float64)[None, :]", "r = r"),
    ("bf16 rounding truncates", "r = np.ldexp(np.rint(np.ldexp(m, 8)), e - 8)",
     "r = np.ldexp(np.trunc(np.ldexp(m, 8)), e - 8)"),
    ("Top-p needs strictly more than p", "if cum >= pp:", "if cum > pp:"),
    ("Top-p ranks ascending", "order = np.lexsort((e_idx, -(r[i] + 0.0)))",
     "order = np.lexsort((e_idx, (r[i] + 0.0)))"),
    ("threshold inclusive", "n = (prob > _p64(tau)).sum(axis=1)", "n = (prob >= _p64(tau)).sum(axis=1)"),
    ("threshold counts unclamped", "return np.clip(n, k_min, k_max).astype(np.int64)",
     "return n.astype(np.int64)"),
    ("commit strictly above theta", "C = J[ct[J] >= th]", "C = J[ct[J] > th]"),
    ("history not shifted", "c2[was_masked] = c1[was_masked]", "c2[was_masked] = c2[was_masked]"),
    ("block advances with tokens left", "if left_in_active == 0 and a[s] < last_block:",
     "if a[s] < last_block:"),
    ("frontier and progress keys swapped", "SIGNAL_FRONTIER: F, SIGNAL_PROGRESS: P",
     "SIGNAL_FRONTIER: P, SIGNAL_PROGRESS: F"),
    ("frontier key ranks by the score", "SIGNAL_FRONTIER: F, SIGNAL_PROGRESS: P",
     "SIGNAL_FRONTIER: S, SIGNAL_PROGRESS: P"),
    ("progress key ranks by the score", "SIGNAL_FRONTIER: F, SIGNAL_PROGRESS: P",
     "SIGNAL_FRONTIER: F, SIGNAL_PROGRESS: S"),
    ("progress guard ties to higher position", "best = J[np.lexsort((J, -ct[J].astype(np.float64)))[0]]",
     "best = J[np.lexsort((-J, -ct[J].astype(np.float64)))[0]]"),
]


@pytest.fixture(scope="module")
def source():
    with open(os.path.join(ROOT, "oracle", "reflex.py")) as fh:
        return fh.read()


@pytest.mark.parametrize("name,old,new", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_pins_catch_mutant(name, old, new, source, tmp_path):
    assert source.count(old) == 1, name
    for sub in ("oracle", "synth", "tests"):
        shutil.copytree(os.path.join(ROOT, sub), tmp_path / sub,
                        ignore=shutil.ignore_patterns("__pycache__", "test_oracle_mutants.py"))
    (tmp_path / "oracle" / "reflex.py").write_text(source.replace(old, new))
    r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider",
                        "tests/test_oracle_budget.py", "tests/test_oracle_layer.py",
                        "tests/test_oracle_rules.py", "tests/test_oracle_state.py"],
                       cwd=tmp_path, capture_output=True, text=True, timeout=300)
    assert r.returncode != 0, f"mutant '{name}' survived the oracle pins"
