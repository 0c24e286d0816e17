"""The oracle's pins catch plausible mistakes.

Each case copies oracle/sfa_oracle.c, plants one mistake by a textual substitution
(a wrong mask, a dropped scale, a wrong sign or index, a transposed role), builds the
copy with gcc and runs the pin suite (tests/test_oracle_pins.py) against it in a
subprocess: at least one pin must fail.  An unmodified copy must pass, so the mechanism
itself is checked too.  CPU only; the planted mistakes never leave the temporary
directory.
"""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "sfa_oracle.c")

# (name, text in the oracle, replacement)
MUTANTS = [
    ("intra layer sees other streams", "return sk == s && pk <= pq;", "return pk <= pq;"),
    ("cross-stream query misses its own key", "int causal = tk < t || (tk == t && sk <= s);",
     "int causal = tk < t || (tk == t && sk < s);"),
    ("softmax scale dropped", "x[j] = P->scale * dot;", "x[j] = dot;"),
    ("lse in log2", "*lse = m + log(l);", "*lse = m + log2(l);"),
    ("dS sign of Delta", "double ds = x[j] * (dp - delta);", "double ds = x[j] * (dp + delta);"),
    ("dK scale dropped", "P->scale * ds * load_elem(P->q,", "ds * load_elem(P->q,"),
    ("dV takes dS for P", "x[j] * load_elem(P->dout, P->dtype, q_index(P, b, p, hq, d));",
     "(x[j] * (dp - delta)) * load_elem(P->dout, P->dtype, q_index(P, b, p, hq, d));"),
    ("grouped-query heads interleaved", "const int64_t hk = hq / (P->Hq / P->Hkv);",
     "const int64_t hk = hq % P->Hkv;"),
    ("local window one too wide", "return causal && pq - pk < window;",
     "return causal && pq - pk <= window;"),
    ("expansion stream-major", "int64_t p = t * n + s;", "int64_t p = s * L + t;"),
    ("expansion gradient into the wrong table", "double *dst = dtables + (s * V + id) * Dm;",
     "double *dst = dtables + ((n - 1 - s) * V + id) * Dm;"),
    ("cyclic replication in blocks", "(const char *)src + (s % n) * table",
     "(const char *)src + (s / (m / n)) * table"),
    ("final-stream gather of the first stream", "(b * n * L + i * n + n - 1) * row, row);",
     "(b * n * L + i * n) * row, row);"),
]


def _run_pins(tmp_path, text, tag):
    src = tmp_path / f"{tag}.c"
    src.write_text(text)
    env = dict(os.environ, HD_ORACLE_SRC=str(src), HD_ORACLE_LIB=str(tmp_path / f"lib{tag}.so"))
    r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider",
                        os.path.join(ROOT, "tests", "test_oracle_pins.py")],
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=900)
    return r


def test_unmodified_copy_passes(tmp_path):
    r = _run_pins(tmp_path, open(SRC).read(), "control")
    assert r.returncode == 0, r.stdout[-2000:]


@pytest.mark.parametrize("name,old,new", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_planted_mistake_fails_a_pin(tmp_path, name, old, new):
    text = open(SRC).read()
    assert old in text, f"mutation site not found: {old}"
    r = _run_pins(tmp_path, text.replace(old, new), "mutant")
    # exit code 1: tests ran and at least one failed (not a build or collection error)
    assert r.returncode == 1, f"{name}: pins did not fail (rc={r.returncode})\n{r.stdout[-2000:]}"
