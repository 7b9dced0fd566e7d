"""The oracle's pins catch planted mistakes (no GPU).

Each case copies the oracle's C source, plants one plausible mistake (a
transposed operand, a flipped sign, a wrong index, a dropped term, the wrong
tie-break or group order), builds it with gcc into a temporary library, and
runs the pin tests against that build in a subprocess.  Every planted mistake
must make at least one pin fail.
"""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "moe_oracle.c")

MUTATIONS = [
    ("router reads a transposed weight",
     "elem(w_router, e * H + h, dtype)", "elem(w_router, (h * E + e) % (E * H), dtype)"),
    ("router subtracts the bias", "if (bias) s += (double)bias[e];", "if (bias) s -= (double)bias[e];"),
    ("ties go to the higher index",
     "if (best < 0 || s[e] > s[best]) best = e;", "if (best < 0 || s[e] >= s[best]) best = e;"),
    ("gate exponent has the wrong sign", "exp(sj - top)", "exp(top - sj)"),
    ("offloaded experts packed first", "if ((pass == 0) != is_res) continue;", "if ((pass == 1) != is_res) continue;"),
    ("inverse permutation wrong", "inv_perm[perm[p]] = (int32_t)p;", "inv_perm[p] = perm[p];"),
    ("gate and up projections swapped", "a[f] = silu(g) * u;", "a[f] = silu(u) * g;"),
    ("up projection dropped", "a[f] = silu(g) * u;", "a[f] = silu(g);"),
    ("up projection reads the gate rows",
     "u += xv * elem(w13, (F + f) * H + h, dtype);", "u += xv * elem(w13, f * H + h, dtype);"),
    ("down projection transposed",
     "elem(w2, h * F + f, dtype)", "elem(w2, (f * H + h) % (H * F), dtype)"),
    ("silu sign", "return z / (1.0 + exp(-z));", "return z / (1.0 + exp(z));"),
    ("bf16 widened with the wrong shift", "<< 16;", "<< 15;"),
]


@pytest.mark.parametrize("name,old,new", MUTATIONS, ids=[m[0] for m in MUTATIONS])
def test_pins_catch_planted_mistake(tmp_path, name, old, new):
    src = open(SRC).read()
    assert src.count(old) == 1, f"mutation anchor not unique: {old!r}"
    mutated = tmp_path / "moe_oracle.c"
    mutated.write_text(src.replace(old, new))
    lib = tmp_path / "libmoe_oracle_mut.so"
    subprocess.run(["gcc", "-O2", "-std=c11", "-fopenmp", "-fPIC", "-shared", "-o", str(lib), str(mutated), "-lm"],
                   check=True)
    env = dict(os.environ, MOE_ORACLE_LIB=str(lib), OMP_NUM_THREADS="2")
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-x", "-p", "no:cacheprovider",
                        os.path.join(ROOT, "tests", "test_oracle_pins.py")],
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=600)
    assert r.returncode != 0, f"planted mistake '{name}' passed every pin:\n{r.stdout[-2000:]}"
    assert "failed" in r.stdout


# The stage-boundary and coherence functions are Python; a mistake is planted in a copy
# of the oracle package that shadows the real one for the pin tests' subprocess.
PY_SRC = os.path.join(ROOT, "oracle", "__init__.py")
PY_PINS = [os.path.join(ROOT, "tests", "test_cue_fsm.py"), os.path.join(ROOT, "tests", "test_temporal_coherence.py")]

PY_MUTATIONS = [
    ("cue ties go to the higher id", "take = hit & (L > best_len)", "take = hit & (L >= best_len)"),
    ("first cue wins instead of the longest", "take = hit & (L > best_len)", "take = hit & (best < 0)"),
    ("negative ids match a cue token", "hit &= shifted == c[j]", "hit &= (shifted == c[j]) | (shifted == -1)"),
    ("cue compared in reverse order", "back = L - 1 - j", "back = j"),
    ("stage cut one step early", "cuts = [int(i) + 1 for i in ev if int(i) + 1 < steps]",
     "cuts = [int(i) for i in ev if 0 < int(i) < steps]"),
    ("TC_seq averaged over P stages", "return total / (P - 1)", "return total / P"),
    ("TC_seq without the cosine's norms", "sim += dot / (nu * nv)", "sim += dot"),
    ("TC_seq compares with the last stage", "u, v = R[p][l], R[p + 1][l]", "u, v = R[p][l], R[-1][l]"),
]


@pytest.mark.parametrize("name,old,new", PY_MUTATIONS, ids=[m[0] for m in PY_MUTATIONS])
def test_pins_catch_planted_python_mistake(tmp_path, name, old, new):
    src = open(PY_SRC).read()
    assert src.count(old) == 1, f"mutation anchor not unique: {old!r}"
    pkg = tmp_path / "oracle"
    pkg.mkdir()
    (pkg / "__init__.py").write_text(src.replace(old, new))
    env = dict(os.environ, MOE_ORACLE_LIB=os.path.join(ROOT, "oracle", "libmoe_oracle.so"),
               PYTHONPATH=os.pathsep.join([str(tmp_path), ROOT]))
    # run from the copy's directory: it comes first on sys.path, ahead of the repository
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-x", "-p", "no:cacheprovider", "--rootdir", ROOT,
                        "-k", "oracle", *PY_PINS],
                       cwd=str(tmp_path), env=env, capture_output=True, text=True, timeout=600)
    assert r.returncode != 0, f"planted mistake '{name}' passed every pin:\n{r.stdout[-2000:]}"
    assert "failed" in r.stdout
