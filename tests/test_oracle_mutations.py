"""The pins catch plausible mistakes in the oracle (CPU only).

Each case plants one mistake in a copy of oracle/poseidon_oracle.c (a dropped
term, a flipped sign, a transposed operand, a dropped shard or message, the
wrong tie rule), builds it, and runs the oracle's pin tests against that
build in a fresh process: at least one pin must fail.  The unmodified source,
built the same way, must pass them all."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "poseidon_oracle.c")
PINS = ["tests/test_oracle_sfb.py", "tests/test_oracle_ps.py", "tests/test_oracle_hybcomm.py",
        "tests/test_oracle_kv.py"]

# (name, [(text in the source, replacement)], replace every occurrence)
MUTATIONS = [
    ("SF drops the last factor pair",
     [("for (int64_t k = 0; k < K; ++k)", "for (int64_t k = 0; k < K - 1; ++k)")], True),
    ("SGD step with the wrong sign",
     [("w[n] = (float)((double)w[n] - (double)lr * acc[n]);", "w[n] = (float)((double)w[n] + (double)lr * acc[n]);"),
      ("out[i] = (float)((double)W[m * N + n] - (double)lr * acc);",
       "out[i] = (float)((double)W[m * N + n] + (double)lr * acc);")], False),
    ("U read transposed", [("(double)U[k * M + m]", "(double)U[m * K + k]")], True),
    ("PS sum drops a shard",
     [("for (int32_t p = 0; p < P; ++p)\n        s += (double)tmp[p];",
       "for (int32_t p = 0; p < P - 1; ++p)\n        s += (double)tmp[p];")], False),
    ("momentum adds the negated gradient",
     [("(float)((double)mu * (double)(*b) + s)", "(float)((double)mu * (double)(*b) - s)")], False),
    ("PS pulls not counted",
     [("if (add_msg(per_node, s, w, ps_units)) return -1;  /* pull */", "")], False),
    ("SFB factors not scaled to 1/P2 units",
     [("if (__builtin_mul_overflow(bmn, P2, &sf_units)) return -1;", "sf_units = bmn;")], False),
    ("Alg. 1 tie goes to PS", [("rc = (tsfb <= tps) ? 1 : 0;", "rc = (tsfb < tps) ? 1 : 0;")], False),
]


def _build(src_text, out_dir):
    src = os.path.join(out_dir, "oracle.c")
    lib = os.path.join(out_dir, "liboracle.so")
    with open(src, "w") as f:
        f.write(src_text)
    subprocess.run(["gcc", "-std=c11", "-O2", "-fopenmp", "-fPIC", "-shared", "-ffp-contract=off",
                    "-fno-fast-math", src, "-o", lib], check=True, capture_output=True)
    return lib


def _run_pins(lib):
    env = dict(os.environ, POSEIDON_ORACLE_LIB=lib)
    return subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider", *PINS],
                          cwd=ROOT, env=env, capture_output=True, text=True, timeout=600)


def test_unmodified_oracle_passes_the_pins(tmp_path):
    r = _run_pins(_build(open(SRC).read(), str(tmp_path)))
    assert r.returncode == 0, r.stdout[-2000:]


@pytest.mark.parametrize("name,edits,every", MUTATIONS, ids=[m[0] for m in MUTATIONS])
def test_pins_catch_a_planted_mistake(name, edits, every, tmp_path):
    text = open(SRC).read()
    for old, new in edits:
        assert old in text, f"{name}: the source no longer contains {old!r}"
        text = text.replace(old, new) if every else text.replace(old, new, 1)
    r = _run_pins(_build(text, str(tmp_path)))
    assert r.returncode == 1, f"{name}: no pin failed\n{r.stdout[-2000:]}"
