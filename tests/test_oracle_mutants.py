"""The pins must catch plausible mistakes in the oracle.

Each case plants one mistake in a copy of the oracle's C source (on the CPU),
builds it, and runs the pin suite against it with PIVOT_ORACLE_LIB; the suite
has to fail.  The unmodified source must pass the same run.
"""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "pivot_oracle.c")

MUTANTS = {
    "relu dropped (Eq. 1)": ("double relu = dot > 0.0 ? dot : 0.0;", "double relu = dot;"),
    "gate sign flipped (Eq. 1)": ("total += ((double)w_row[j] * sq) * relu;",
                                  "total -= ((double)w_row[j] * sq) * relu;"),
    "key scale ignored (App. A)": ("return ks * total;", "return total;"),
    "key scale divides (App. A)": ("return ks * total;", "return total / ks;"),
    "query operand transposed": ("elem(fmt, q_row, (int64_t)j * d + i)", "elem(fmt, q_row, (int64_t)i * H + j)"),
    "query scale ignored": ("total += ((double)w_row[j] * sq) * relu;", "total += ((double)w_row[j]) * relu;"),
    "causal prefix excludes t": ("    int64_t n = t + 1;\n    int32_t* pos", "    int64_t n = t;\n    int32_t* pos"),
    "tie-break by higher position": ("return (a->s < b->s) ? -1 : (a->s > b->s) ? 1 : 0;",
                                     "return (a->s > b->s) ? -1 : (a->s < b->s) ? 1 : 0;"),
    "proxy ignores member scales (Eq. 4)": ("float deq = sq * x;", "float deq = x;"),
    "proxy sums instead of averaging (Eq. 4)": ("mean[e] = sum / count;", "mean[e] = sum;"),
    "proxy gate sums instead of averaging (Eq. 4)": ("pw[j] = sum / count;", "pw[j] = sum;"),
    "fp8 ties round up": ("((lo & 1) ? hi : lo)", "hi"),
    "bf16 ties round up": ("(rest == 0x8000u && (keep & 1u))", "(rest == 0x8000u)"),
    "proxy scan past t0 (Eq. 5)": ("int64_t n = t0 + 1;                                          /* Eq. (5) */",
                                   "int64_t n = t0 + gs;"),
    "guardrail inverted (Alg. 1)": ("if (mode == OR_DENSE || t0 < dense_below)", "if (mode == OR_DENSE || t0 >= dense_below)"),
    "guardrail off (Alg. 1)": ("if (mode == OR_DENSE || t0 < dense_below)", "if (mode == OR_DENSE)"),
    "reuse not shared (Eq. 6)": ("for (int t = 1; t < gs; ++t) memcpy(og + (size_t)t * m, og, sizeof(int32_t) * (size_t)m);", ""),
    "candidate budget k instead of c (Eq. 7)": ("int nc = topk(f, pos, n, c, cand);", "int nc = topk(f, pos, n, m, cand);"),
    "refine re-scores with the proxy (Eq. 8)": ("score_positions(&K, qg + (size_t)t * rowb, sg ? (double)sg[t] : 1.0,\n                                wg + (size_t)t * H, cand, nc, fc);",
                                                "score_positions(&K, pq, fmt == OR_FP8 ? (double)psc : 1.0, pw, cand, nc, fc);"),
    "proxy scale from amax/240": ("amax / 448.0f", "amax / 240.0f"),
}


def _run_pins(lib_path):
    env = dict(os.environ, PIVOT_ORACLE_LIB=lib_path)
    return subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider",
                           os.path.join(ROOT, "tests", "test_oracle_pins.py")],
                          cwd=ROOT, env=env, capture_output=True, text=True, timeout=600)


def _build(tmp_path, name, text):
    import oracle
    src = tmp_path / f"{name}.c"
    src.write_text(text)
    return oracle.compile_source(str(src), str(tmp_path / f"lib{name}.so"))


def test_unmodified_oracle_passes(tmp_path):
    lib = _build(tmp_path, "clean", open(SRC).read())
    r = _run_pins(lib)
    assert r.returncode == 0, r.stdout[-2000:]


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_planted_mistake_is_caught(tmp_path, name):
    old, new = MUTANTS[name]
    text = open(SRC).read()
    assert text.count(old) == 1, f"mutation anchor not unique/present: {name}"
    lib = _build(tmp_path, "mutant", text.replace(old, new))
    r = _run_pins(lib)
    assert r.returncode != 0, f"pins did not catch: {name}"
