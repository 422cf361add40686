"""The pins are strong enough: each plausible mistake planted in a copy of the
C oracle (compiled on the CPU into a temporary library) makes at least one pin
of tests/test_oracle_pins.py or tests/test_oracle_profiling_pins.py fail.

The pin suite runs in a child pytest process with FKV_ORACLE_LIB pointing at
the mutated build; -x stops it at the first failing pin."""
import os
import subprocess
import sys

import pytest

import oracle

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)

# (name, original text, mutated text): the first occurrence is replaced.
MUTATIONS = [
    ("score dot uses a*a", "dot += a * b;", "dot += a * a;"),
    ("score nb from the first segment", "nb += b * b;", "nb += a * a;"),
    ("score partner is the same frame", "long y = x + F; /* same position, next frame */", "long y = x;"),
    ("score zero-norm guard missing", "double cosv = (na * nb == 0.0) ? 0.0 : dot / sqrt(na * nb);",
     "double cosv = dot / sqrt(na * nb);"),
    ("score without the square root", "double cosv = (na * nb == 0.0) ? 0.0 : dot / sqrt(na * nb);",
     "double cosv = (na * nb == 0.0) ? 0.0 : dot / (na * nb);"),
    ("select keeps the most similar", "        if (a->s < b->s) return -1;\n        if (a->s > b->s) return 1;",
     "        if (a->s < b->s) return 1;\n        if (a->s > b->s) return -1;"),
    ("select keeps NaN first", "if (na != nb) return na - nb;", "if (na != nb) return nb - na;"),
    ("select ties by the higher index", "return (a->g > b->g) - (a->g < b->g);", "return (a->g < b->g) - (a->g > b->g);"),
    ("select recent window one short", "int forced = first < sink || last >= (long)H - recent;",
     "int forced = first < sink || last > (long)H - recent;"),
    ("static recent window one short", "if (t < sink || t >= H - recent)", "if (t < sink || t > H - recent)"),
    ("gather ignores the slot map", "(size_t)frame_slot[frames[i]] * frame_bytes", "(size_t)frames[i] * frame_bytes"),
    ("compaction reverses token order", "(const char *)hist + hist_row(x, F, d, frame_slot) * esize",
     "(const char *)hist + hist_row(x1 - 1 - (x - x0), F, d, frame_slot) * esize"),
    ("attention without the scale", "z[j] = scale * acc;", "z[j] = acc;"),
    ("attention not normalised", "for (int c = 0; c < d; ++c) o[c] /= den;", ""),
    ("attention reads V from K", "const void *vb = j < kv_len ? Vc : Vcur;", "const void *vb = j < kv_len ? Kc : Kcur;"),
    ("pooled score uses head 0 only", "for (int h = 0; h < n_heads; ++h) {", "for (int h = 0; h < 1; ++h) {"),
    ("mass not normalised by the row sum", "acc[j / F] += exp(z[j] - m) / den;", "acc[j / F] += exp(z[j] - m);"),
    ("mass binned one key late", "acc[j / F] += exp(z[j] - m) / den;",
     "acc[(j + 1) / F < n_bins ? (j + 1) / F : n_bins - 1] += exp(z[j] - m) / den;"),
    ("append ignores the slot", "(char *)hist + (size_t)dst_slot[f] * frame_bytes", "(char *)hist + (size_t)f * frame_bytes"),
]


@pytest.mark.parametrize("name,old,new", MUTATIONS, ids=[m[0] for m in MUTATIONS])
def test_pins_catch_planted_mistake(tmp_path, name, old, new):
    src = open(oracle._SRC).read()
    assert old in src, f"mutation anchor not found: {old!r}"
    (tmp_path / "fkv_oracle.c").write_text(src.replace(old, new, 1))
    for h in ("fkv_oracle.h",):
        (tmp_path / h).write_text(open(os.path.join(os.path.dirname(oracle._SRC), h)).read())
    so = tmp_path / "liboracle_mut.so"
    subprocess.run(["gcc", "-O1", "-std=c11", "-fopenmp", "-fPIC", "-shared", "-ffp-contract=off",
                    str(tmp_path / "fkv_oracle.c"), "-o", str(so), "-lm"], check=True, capture_output=True)
    env = dict(os.environ, FKV_ORACLE_LIB=str(so), OMP_NUM_THREADS="4")
    r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider",
                        os.path.join(HERE, "test_oracle_pins.py"), os.path.join(HERE, "test_oracle_profiling_pins.py")],
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=300)
    assert r.returncode != 0, f"no pin caught the mutation '{name}':\n{r.stdout[-2000:]}"
    assert "failed" in r.stdout or "error" in r.stdout.lower(), r.stdout[-2000:]
