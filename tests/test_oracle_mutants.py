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
    "proxy scan past t0 (Eq. 5)": ("int64_t lim = (W > 0 && window_kind == 0) ? t0 - W : t0;",
                                   "int64_t lim = (W > 0 && window_kind == 0) ? t0 - W : t0 + gs - 1;"),
    "guardrail inverted (Alg. 1)": ("if (mode == OR_DENSE || t0 < dense_below)", "if (mode == OR_DENSE || t0 >= dense_below)"),
    "guardrail off (Alg. 1)": ("if (mode == OR_DENSE || t0 < dense_below)", "if (mode == OR_DENSE)"),
    "reuse not shared (Eq. 6)": ("for (int t = 1; t < gs; ++t) memcpy(og + (size_t)t * m, og, sizeof(int32_t) * (size_t)m);", ""),
    "candidate budget k instead of c (Eq. 7)": ("int proxy_slots = (W > 0 && window_kind == 0) ? c - wg : c;",
                                                "int proxy_slots = (W > 0 && window_kind == 0) ? c - wg : m;"),
    "refine re-scores with the proxy (Eq. 8)": ("score_positions(&K, qg + (size_t)t * rowb, sg ? (double)sg[t] : 1.0,\n                                wg_ + (size_t)t * H, use, nu, fc);",
                                                "score_positions(&K, pq, fmt == OR_FP8 ? (double)psc : 1.0, pw, use, nu, fc);"),
    "window union starts one late (App. B)": ("int64_t p = t0 - W + 1 + u;", "int64_t p = t0 - W + 2 + u;"),
    "prefill proxy part overlaps the window (App. B)": ("int64_t lim = (W > 0 && window_kind == 0) ? t0 - W : t0;",
                                                        "int64_t lim = t0;"),
    "window slots past the member kept (causality)": ("if (p < 0 || p > tt) continue;", "if (p < 0) continue;"),
    "decode window not per query (App. B)": ("if (W > 0 && window_kind == 1 && i >= c && p < tt - W + 1) continue;", ""),
    "decode pool duplicates kept (App. B)": ("if (cand[i] == (int32_t)p) { ok = 0; break; }", "if (cand[i] == (int32_t)p) { break; }"),
    "window reserves W slots, not W + g - 1 (App. B)": ("const int wg = W > 0 ? W + g - 1 : 0;", "const int wg = W;"),
    "first and last member swapped": ("int t = (agg == OR_AGG_LAST) ? gs - 1 : 0;", "int t = (agg == OR_AGG_FIRST) ? gs - 1 : 0;"),
    "proxy scale from amax/240": ("amax / 448.0f", "amax / 240.0f"),
    "IndexCache followers reuse layer 0 (Sec. 5.1)": ("            src = l;", "            src = 0;"),
    "IndexCache followers index themselves (Sec. 5.1)": ("        if (anchor[l]) {", "        if (1) {"),
    "IndexCache only the first layer indexes (Sec. 5.1)": ("        if (anchor[l]) {", "        if (l == 0) {"),
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
