"""Planted mistakes in the oracle must each make a pin fail.

Each case patches one plausible error into a copy of oracle/sense_oracle.c
(a dropped term, a wrong index or window offset, a flipped tie rule, < for
<=, a wrong log base, a misplaced parenthesis, a lost length), builds it into
a temporary library and runs the oracle's pin tests against that library in a
subprocess: at least one pin must fail.  The unpatched source built the same
way must pass them all, so a failure is the planted mistake's doing."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "sense_oracle.c")
PINS = ["tests/test_oracle_retrieval.py", "tests/test_oracle_verify.py",
        "tests/test_oracle_select.py"]

# (name, text in the source, replacement, which occurrence (0 = first))
MUTATIONS = [
    ("cosine drops the key norm", "dot / (qnorm * knorm)", "dot / qnorm", 0),
    ("dot product drops the last element",
     "for (int32_t t = 0; t < d; ++t) {\n                double kv",
     "for (int32_t t = 0; t < d - 1; ++t) {\n                double kv", 0),
    ("retrieval ties go to the higher row",
     "return (a->i < b->i) ? -1 : (a->i > b->i);",
     "return (a->i > b->i) ? -1 : (a->i < b->i);", 0),
    ("NaN scores sort first", "if (an != bn) return an ? 1 : -1;",
     "if (an != bn) return an ? -1 : 1;", 0),
    ("gather ignores span lengths", "len = span_len ? span_len[id] : max_span;",
     "len = max_span;", 0),
    ("window includes the position itself",
     "for (int32_t u = 1; u <= window; ++u) r += bbar[j + u];",
     "for (int32_t u = 0; u < window; ++u) r += bbar[j + u];", 0),
    ("entropy normalised by log2", "const double log_v = log((double)vocab);",
     "const double log_v = log2((double)vocab);", 0),
    ("top-k ties go to the higher vocabulary index",
     "return (a->v < b->v) ? -1 : (a->v > b->v);",
     "return (a->v > b->v) ? -1 : (a->v < b->v);", 0),
    ("window tolerance strict", "int con = (r <= tau);", "int con = (r < tau);", 0),
    ("gate grouped as em | ent & topk | con", "(em[p] || (ent[p] && (tk[p] || con)))",
     "(em[p] || (ent[p] && tk[p]) || con)", 0),
    ("softmax drops the first term", "for (int32_t v = 0; v < vocab; ++v) z += exp(",
     "for (int32_t v = 1; v < vocab; ++v) z += exp(", 0),
    ("argmax takes the last maximum", "if (e[v].x > m) { m = e[v].x; y = v; }",
     "if (e[v].x >= m) { m = e[v].x; y = v; }", 0),
    ("entropy gate not strict", "ent[p] = (g > gamma);", "ent[p] = (g >= gamma);", 0),
    ("best candidate is the last maximiser",
     "if (out_accept_len[g * gsz + i] > out_accept_len[g * gsz + b]) b = i;",
     "if (out_accept_len[g * gsz + i] >= out_accept_len[g * gsz + b]) b = i;", 0),
    ("rows past the draft length judged", "if (j >= lens[c]) continue;",
     "if (0) continue;", 0),
    ("empty drafts match the anchor", "int match = len > 0 && row[0] == anchor;",
     "int match = row[0] == anchor;", 0),
    ("delta added to static hits too",
     "double s = dyn ? scores_d[r] + delta : scores_s[r];",
     "double s = (dyn ? scores_d[r] : scores_s[r]) + delta;", 0),
    ("override only at the first draft", "int32_t ends[2] = {0, top_n - 1};",
     "int32_t ends[2] = {0, 0};", 0),
    ("composite ties go to the later position",
     "return (a->i < b->i) ? -1 : (a->i > b->i);",
     "return (a->i > b->i) ? -1 : (a->i < b->i);", 1),
]


def build(src_text: str, out: str) -> None:
    c = out + ".c"
    with open(c, "w") as f:
        f.write(src_text)
    subprocess.check_call(["gcc", "-O1", "-std=c11", "-fPIC", "-shared", "-fopenmp", c, "-o",
                           out, "-lm"])


def run_pins(lib: str) -> subprocess.CompletedProcess:
    env = dict(os.environ, SENSE_ORACLE_LIB=lib, OMP_NUM_THREADS="2")
    return subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider",
                           "-m", "not gpu", *PINS], cwd=ROOT, env=env, capture_output=True,
                          text=True, timeout=600)


def patched(name, old, new, which):
    text = open(SRC).read()
    at = -1
    for _ in range(which + 1):
        at = text.index(old, at + 1)
    return text[:at] + new + text[at + len(old):]


def test_unpatched_oracle_passes_its_pins(tmp_path):
    lib = str(tmp_path / "liboracle_ref.so")
    build(open(SRC).read(), lib)
    r = run_pins(lib)
    assert r.returncode == 0, r.stdout[-2000:]


@pytest.mark.parametrize("name,old,new,which", MUTATIONS, ids=[m[0] for m in MUTATIONS])
def test_planted_mistake_fails_a_pin(tmp_path, name, old, new, which):
    lib = str(tmp_path / "liboracle_mut.so")
    build(patched(name, old, new, which), lib)
    r = run_pins(lib)
    assert r.returncode != 0, f"no pin caught: {name}\n{r.stdout[-1500:]}"
