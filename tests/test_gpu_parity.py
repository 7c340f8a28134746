"""End-to-end GPU parity of pivot_dense_index / pivot_group_index with the
oracle (Algorithm 1), on inputs small enough for the oracle, spanning several
score segments and top-k tiles, with ragged groups, chunked calls, the
guardrail on and off, and batched decode groups."""
import numpy as np
import pytest

import oracle
import paper_2607_24593_amd as pv
from gpu_util import dev, host, say
from parity import check_pivot
from workload.gen import make_decode, make_prefill

pytestmark = pytest.mark.gpu

MODES = {"dense": oracle.DENSE, "reuse": oracle.REUSE, "refine": oracle.REFINE}
PV_MODE = {"reuse": pv.PIVOT_REUSE, "refine": pv.PIVOT_REFINE}


def run_gpu(x, mode, p0, n_q, topk, g=1, c=0, dense_below=-1):
    q = x.q[p0:p0 + n_q]
    qs = None if x.q_scale is None else x.q_scale[p0:p0 + n_q]
    w = x.w[p0:p0 + n_q]
    n_k = p0 + n_q
    say(mode, x.dtype, "p0", p0, "n_q", n_q, "topk", topk, "g", g, "c", c, "db", dense_below)
    args = (dev(q), dev(qs), dev(w), dev(x.k[:n_k]), dev(None if x.k_scale is None else x.k_scale[:n_k]), p0, n_k, topk)
    cand = None
    if mode == "dense":
        idx = pv.pivot_dense_index(*args)
    else:
        ng = (n_q + g - 1) // g
        cand_t = None
        if mode == "refine":
            import torch
            cand_t = torch.full((1, ng, c), -7, dtype=torch.int32, device="cuda")
        idx = pv.pivot_group_index(*args, mode=PV_MODE[mode], g=g, c=c, dense_below=dense_below, out_cand=cand_t)
        cand = None if cand_t is None else host(cand_t)[0]
    return host(idx), cand, (q, qs, w, n_k)


def check(x, mode, p0, n_q, topk, g=1, c=0, dense_below=-1, groups=None, label=""):
    idx, cand, (q, qs, w, n_k) = run_gpu(x, mode, p0, n_q, topk, g, c, dense_below)
    if groups is not None:
        keep = np.zeros(n_q, bool)
        for j in groups:
            keep[j * g:(j + 1) * g] = True
    return check_pivot(x.dtype, q, qs, w, p0, x.k[:n_k], None if x.k_scale is None else x.k_scale[:n_k], n_k,
                       mode=MODES[mode], g=g, c=c, topk=topk, dense_below=dense_below, gpu_idx=idx,
                       gpu_cand=cand, groups=groups, label=label)


@pytest.fixture(scope="module")
def small_bf16():
    return make_prefill(1100, "bf16", seed=31, threads=4)


@pytest.fixture(scope="module")
def long_fp8():
    return make_prefill(9000, "fp8", seed=32, threads=8)


@pytest.mark.parametrize("mode", ["dense", "reuse", "refine"])
def test_bf16_every_query(small_bf16, mode):
    """Every query of a 1100-position bf16 prefill (ragged last group, g=4)."""
    check(small_bf16, mode, 0, 1099, 64, g=4, c=256, label=f"bf16 {mode}")


def _sample_groups(n_q, g, p0, c, rng, extra=()):
    ng = (n_q + g - 1) // g
    pick = {0, 1, ng - 1, ng - 2} | set(int(v) for v in rng.integers(0, ng, 12))
    for t in (c - g, c, c + g) + tuple(extra):      # around the guardrail and segment edges
        j = (t - p0) // g
        if 0 <= j < ng:
            pick.add(j)
    return sorted(pick)


@pytest.mark.parametrize("mode", ["dense", "reuse", "refine"])
@pytest.mark.parametrize("g", [2, 4, 8])
def test_fp8_sampled_groups(long_fp8, mode, g):
    """fp8, 8999 queries (segments of 4096 keys, ragged tail), sampled groups."""
    rng = np.random.default_rng(g)
    n_q = 8999
    groups = _sample_groups(n_q, g if mode != "dense" else 1, 0, 1024, rng, extra=(4095, 4096, 8191, 8192))
    check(long_fp8, mode, 0, n_q, 256, g=g if mode != "dense" else 1, c=1024, groups=groups,
          label=f"fp8 {mode} g{g}")


@pytest.mark.parametrize("mode", ["reuse", "refine"])
def test_fp8_chunk_with_offset(long_fp8, mode):
    """A later chunk of a prefill: queries 5120 .. 8999 against keys 0 .. 8999."""
    rng = np.random.default_rng(5)
    p0, n_q, g = 5120, 3880, 4
    groups = _sample_groups(n_q, g, p0, 1024, rng)
    check(long_fp8, mode, p0, n_q, 256, g=g, c=1024, groups=groups, label=f"chunk {mode}")


@pytest.mark.parametrize("dense_below", [0, 3000])
def test_guardrail_threshold(long_fp8, dense_below):
    """Guardrail disabled (every group on the proxy path, also t0 < c, where the
    candidate set is the whole prefix) and set above c."""
    rng = np.random.default_rng(9)
    n_q, g = 4000, 4
    groups = _sample_groups(n_q, g, 0, 1024, rng, extra=(0, 4, 8, 300, 2996, 3000))
    check(long_fp8, "refine", 0, n_q, 128, g=g, c=1024, dense_below=dense_below, groups=groups,
          label=f"db {dense_below}")
    check(long_fp8, "reuse", 0, n_q, 128, g=g, c=1024, dense_below=dense_below, groups=groups,
          label=f"db {dense_below}")


def test_group_of_one_equals_dense(long_fp8):
    """App. A identity on the GPU: g = 1 Reuse and Refine give the dense sets
    exactly.  A group of one is its own proxy; every tile shape adds a score's
    heads in the same order, so the proxy scan and Refine's re-score produce
    the dense path's score bits, and the top-k of the top-c is the top-k."""
    x = long_fp8
    for p0, n_q in ((3000, 64), (1024, 2000)):
        d, _, _ = run_gpu(x, "dense", p0, n_q, 100)
        r, _, _ = run_gpu(x, "reuse", p0, n_q, 100, g=1, c=200, dense_below=0)
        assert np.array_equal(np.sort(r, 1), np.sort(d, 1)), ("reuse", p0)
        r, _, _ = run_gpu(x, "refine", p0, n_q, 100, g=1, c=200, dense_below=0)
        assert np.array_equal(np.sort(r, 1), np.sort(d, 1)), ("refine", p0)


@pytest.mark.parametrize("L", [5000, 20000])
def test_group_of_one_equals_dense_decode(L):
    """The same identity at decode shapes (one query per sequence, keys-mode
    scan with one row per wave, the split select for 20000-key contexts)."""
    B = 5
    x = make_decode(B, L, 1, "fp8", seed=48, threads=6)
    q, qs, w, k, ks = dev(x.q), dev(x.q_scale), dev(x.w), dev(x.k), dev(x.k_scale)
    pos, nk = [L - 1] * B, [L] * B
    say("decode g=1 identity", L)
    d = host(pv.pivot_dense_index(q, qs, w, k, ks, pos, nk, 256))
    for mode in ("reuse", "refine"):
        r = host(pv.pivot_group_index(q, qs, w, k, ks, pos, nk, 256, mode=PV_MODE[mode], g=1, c=1024,
                                      dense_below=0))
        assert np.array_equal(np.sort(r, -1), np.sort(d, -1)), mode


@pytest.mark.parametrize("B,L", [(6, 5000), (5, 20000)])
@pytest.mark.parametrize("g", [2, 4])
@pytest.mark.parametrize("mode", ["dense", "reuse", "refine"])
def test_decode_batch(mode, g, B, L):
    """Decode: B sequences, each one MTP group of g queries at the end of its
    context (20000-key contexts take the split select and split re-score)."""
    x = make_decode(B, L, g, "fp8", seed=40 + g, threads=6)
    import torch
    say("decode", mode, "B", B, "L", L, "g", g)
    q, qs, w = dev(x.q), dev(x.q_scale), dev(x.w)
    k, ks = dev(x.k), dev(x.k_scale)
    topk, c = 256, 1024
    if mode == "dense":
        idx = pv.pivot_dense_index(q, qs, w, k, ks, [L - g] * B, [L] * B, topk)
        cand = None
    else:
        cand_t = torch.full((B, 1, c), -7, dtype=torch.int32, device="cuda") if mode == "refine" else None
        idx = pv.pivot_group_index(q, qs, w, k, ks, [L - g] * B, [L] * B, topk, mode=PV_MODE[mode], g=g, c=c,
                                   out_cand=cand_t)
        cand = None if cand_t is None else host(cand_t)
    idx = host(idx)
    for b in range(B):
        check_pivot("fp8", x.q[b], x.q_scale[b], x.w[b], L - g, x.k[b], x.k_scale[b], L, mode=MODES[mode], g=g,
                    c=c, topk=topk, dense_below=-1, gpu_idx=idx[b], gpu_cand=None if cand is None else cand[b],
                    label=f"decode b{b}")


def test_repeatable(long_fp8):
    """Same inputs, same indices (fixed tie-breaks, no order dependence)."""
    a, ca, _ = run_gpu(long_fp8, "refine", 4000, 2000, 256, g=4, c=1024)
    b, cb, _ = run_gpu(long_fp8, "refine", 4000, 2000, 256, g=4, c=1024)
    assert np.array_equal(np.sort(a, 1), np.sort(b, 1))
    assert np.array_equal(np.sort(ca, 1), np.sort(cb, 1))


def _tied(L, fmt, seed, pool):
    """A prefill whose keys repeat `pool` distinct key vectors (position s holds
    vector s % pool), so every score row has `pool` distinct values and the
    top-k boundary falls inside a run of exact ties."""
    x = make_prefill(L, fmt, seed=seed, threads=8)
    src = np.arange(L) % pool
    x.k = np.ascontiguousarray(x.k[src])
    if x.k_scale is not None:
        x.k_scale = np.ascontiguousarray(x.k_scale[src])
    return x


def _separated(f, rtol=4e-2):
    v = np.unique(f)
    return len(v) < 2 or (np.diff(v) > rtol * np.abs(v[1:])).all()


@pytest.mark.parametrize("fmt,L,c,topk,pool", [("fp8", 3000, 1024, 256, 6), ("bf16", 3000, 1024, 256, 5),
                                               ("fp8", 9000, 4096, 2048, 6)])
@pytest.mark.parametrize("mode", ["dense", "reuse", "refine"])
def test_tied_keys_exact(fmt, L, c, topk, pool, mode):
    """Exact ties at the boundary go to the lower position: the GPU sets equal the
    oracle's, entry for entry, in every row whose distinct scores are far apart
    compared with the score error (candidate sets likewise)."""
    x = _tied(L, fmt, 41 + L + pool, pool)
    g = 4
    n_q = L
    groups = sorted({0, 255, 256, 300, (n_q - 1) // g} | set(range(c // g, n_q // g, 97)))
    idx, cand, (q, qs, w, n_k) = run_gpu(x, mode, 0, n_q, topk, g=g, c=c)
    rows = [r for j in groups for r in range(j * g, min(n_q, (j + 1) * g))]
    res = oracle.index(fmt, q, qs, w, 0, x.k, x.k_scale, n_k, mode=MODES[mode], g=1 if mode == "dense" else g,
                       c=c, topk=topk, groups=rows if mode == "dense" else groups,
                       want_cand=(mode == "refine"), want_proxy=(mode != "dense"))
    pool_pos = np.arange(pool, dtype=np.int32)
    checked = 0
    for r in rows:
        f = oracle.scores_at(fmt, q[r], 1.0 if qs is None else qs[r], w[r], x.k, x.k_scale, pool_pos)
        if not _separated(f):
            continue
        j = r // g
        if mode != "dense" and j * g >= c:
            fp = oracle.scores_at(fmt, res["pq"][j], res["psc"][j], res["pw"][j], x.k, x.k_scale, pool_pos)
            if not _separated(fp):
                continue
            if mode == "refine":
                assert sorted(cand[j].tolist()) == sorted(res["cand"][j].tolist()), ("cand", j)
        assert sorted(idx[r].tolist()) == sorted(res["idx"][r].tolist()), (mode, r)
        checked += 1
    say("tied rows checked", checked, "of", len(rows))
    assert checked >= len(rows) // 2


@pytest.fixture(scope="module")
def long20k_fp8():
    return make_prefill(20000, "fp8", seed=33, threads=8)


@pytest.mark.parametrize("mode", ["dense", "reuse", "refine"])
def test_many_long_rows(long20k_fp8, mode):
    """More than 256 rows of 16384+ scores in one select launch: the one-pass
    select with candidates in the workspace scratch (dense: 2048 rows; proxies:
    512 rows of g=4)."""
    x = long20k_fp8
    p0, n_q = 20000 - 2048, 2048
    g = 1 if mode == "dense" else 4
    rng = np.random.default_rng(5)
    groups = sorted({0, n_q // g - 1} | set(int(v) for v in rng.integers(0, n_q // g, 10)))
    check(x, mode, p0, n_q, 2048, g=g, c=4096, groups=groups, label=f"20k {mode}")


@pytest.mark.parametrize("c", [6000, 8192])
def test_large_candidate_budget(long20k_fp8, c):
    """Refine with c above 5120 (up to the 8192-slot limit): each member's
    select holds 32 (score, position) pairs per thread."""
    x = long20k_fp8
    p0, n_q, g = 20000 - 2048, 2048, 4
    rng = np.random.default_rng(c)
    groups = sorted({0, n_q // g - 1} | set(int(v) for v in rng.integers(0, n_q // g, 8)))
    check(x, "refine", p0, n_q, 2048, g=g, c=c, groups=groups, label=f"20k refine c{c}")


@pytest.mark.parametrize("mode", ["dense", "reuse", "refine"])
def test_outlier_keys_span_the_score_range(mode):
    """Two keys with scales 2^40: a row that sees one scores it about 2^40
    times the others, of either sign, so its scores span ~40 binades and the
    value buckets of a select crowd nearly every other score into one bucket.
    The exact fallbacks then decide: in every dense and proxy row, and in the
    member rows whose candidates hold an outlier.  Checked against the oracle."""
    x = make_prefill(6000, "fp8", seed=57, threads=8)
    x.k_scale = x.k_scale.copy()
    x.k_scale[[123, 2345]] = np.float32(2.0 ** 40)
    p0, n_q, c, topk = 1500, 4500, 1024, 256
    g = 1 if mode == "dense" else 4
    groups = sorted({0, 1, n_q // g - 1} | set(int(v) for v in np.random.default_rng(9).integers(0, n_q // g, 8)))
    check(x, mode, p0, n_q, topk, g=g, c=0 if mode == "dense" else c, groups=groups, label=f"outlier keys {mode}")


@pytest.mark.parametrize("mode,g,topk,c", [
    ("refine", 16, 64, 512),   # proxies of two member batches; four 4-row re-score blocks per group
    ("reuse", 16, 64, 512),
    ("refine", 4, 1, 16),      # top-1 of 16 candidates
    ("refine", 5, 7, 8),       # c barely above k, groups of five (a 4-row and a 1-row block)
])
def test_group_and_selection_extremes(long_fp8, mode, g, topk, c):
    """Large groups (16 members), top-1, and c one above k, on sampled groups
    of a later fp8 chunk."""
    p0, n_q = 4000, 3000
    groups = _sample_groups(n_q, g, p0, c, np.random.default_rng(g * 100 + topk))
    check(long_fp8, mode, p0, n_q, topk, g=g, c=c, groups=groups, label=f"{mode} g{g} k{topk} c{c}")
