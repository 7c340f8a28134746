"""Refine's two execution paths (Sec. 4.4 Eqs. 8-9): the fused launch, in
which each group's member scores stay in LDS and its members select there,
and the split one (re-score into the workspace, then a select launch).  Both
re-score with the same tile and summation order and select by (score desc,
position asc), so their top-k sets must be equal row for row; the fused path
is also checked against the oracle directly.  Cases cover g = 1..4, ragged
last groups, candidate rows shorter than c (guardrail off), topk equal to
the candidate count, exact ties, and paged keys."""
import numpy as np
import pytest
import torch

import oracle
import paper_2607_24593_amd as pv
from gpu_util import dev, host, say
from parity import check_pivot
from workload.gen import make_prefill

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def x9k():
    return make_prefill(9000, "fp8", seed=61, threads=8)


def _run(x, p0, n_q, topk, g, c, path, dense_below=-1):
    n_k = p0 + n_q
    ng = (n_q + g - 1) // g
    say("refine path", path, "p0", p0, "n_q", n_q, "topk", topk, "g", g, "c", c, "db", dense_below)
    cand = torch.full((1, ng, c), -7, dtype=torch.int32, device="cuda")
    idx = pv.pivot_group_index_opts(dev(x.q[p0:n_k]), dev(x.q_scale[p0:n_k]), dev(x.w[p0:n_k]), dev(x.k[:n_k]),
                                    dev(x.k_scale[:n_k]), p0, n_k, topk, mode=pv.PIVOT_REFINE, g=g, c=c,
                                    dense_below=dense_below, out_cand=cand, refine_path=path)
    return host(idx), host(cand)[0]


def _same_sets(a, b, label):
    assert a.shape == b.shape
    sa, sb = np.sort(a, 1), np.sort(b, 1)
    bad = np.nonzero((sa != sb).any(1))[0]
    assert len(bad) == 0, (label, "rows differ", bad[:10])


@pytest.mark.parametrize("g,p0,n_q,c,topk,db", [
    (4, 5000, 4000, 1024, 256, -1),    # 1000 groups of four
    (3, 5000, 3998, 1024, 512, -1),    # R = 4 tile with three members, ragged last group (two members)
    (2, 6000, 2999, 4096, 2048, -1),   # R = 2 tile, full 4096-slot rows, ragged last group
    (1, 7000, 1500, 2048, 100, -1),    # one member per group
    (4, 0, 9000, 4096, 2048, 0),       # guardrail off: early groups have fewer than c candidates
    (4, 2000, 3000, 512, 512, -1),     # topk == c: every candidate selected
])
def test_fused_equals_split(x9k, g, p0, n_q, c, topk, db):
    a, ca = _run(x9k, p0, n_q, topk, g, c, pv.PIVOT_REFINE_FUSED, db)
    b, cb = _run(x9k, p0, n_q, topk, g, c, pv.PIVOT_REFINE_SPLIT, db)
    _same_sets(ca, cb, "candidates")  # the proxy select's output order is not fixed
    _same_sets(a, b, f"g{g} c{c} k{topk}")


def test_fused_matches_oracle(x9k):
    """Two-stage parity of the fused path: candidate sets against the proxy's,
    member sets against Eq. 9 on the GPU's own candidates."""
    x = x9k
    p0, n_q, g, c, topk = 4000, 5000, 4, 2048, 512
    idx, cand = _run(x, p0, n_q, topk, g, c, pv.PIVOT_REFINE_FUSED)
    rng = np.random.default_rng(7)
    groups = sorted({0, n_q // g - 1} | set(int(v) for v in rng.integers(0, n_q // g, 12)))
    n_k = p0 + n_q
    check_pivot("fp8", x.q[p0:n_k], x.q_scale[p0:n_k], x.w[p0:n_k], p0, x.k[:n_k], x.k_scale[:n_k], n_k,
                mode=oracle.REFINE, g=g, c=c, topk=topk, dense_below=-1, gpu_idx=idx, gpu_cand=cand,
                groups=groups, label="fused refine")


def test_fused_ties_equal_split():
    """Keys drawn from 6 distinct vectors: every member row's boundary falls in
    a long run of equal scores, settled by position on both paths."""
    x = make_prefill(6000, "fp8", seed=62, threads=8)
    src = np.arange(6000) % 6
    x.k = np.ascontiguousarray(x.k[src])
    x.k_scale = np.ascontiguousarray(x.k_scale[src])
    a, ca = _run(x, 2000, 4000, 2048, 4, 4096, pv.PIVOT_REFINE_FUSED, dense_below=0)
    b, cb = _run(x, 2000, 4000, 2048, 4, 4096, pv.PIVOT_REFINE_SPLIT, dense_below=0)
    _same_sets(ca, cb, "candidates")
    _same_sets(a, b, "ties")


def test_fused_paged_equals_split():
    """Paged keys (shuffled pages of 64): the fused path gathers through the
    pool rows and breaks ties by sequence position, like the split one."""
    from test_gpu_layout import _page_pool
    x = make_prefill(7000, "fp8", seed=63, threads=8)
    pool, pool_s, table = _page_pool([x.k], [x.k_scale], 64, np.random.default_rng(3))
    p0, n_q = 3000, 4000
    lay = pv.make_layout(cu_q=[0, n_q], block_table=dev(table), page_size=64, pool_keys=len(pool))
    outs = {}
    for path in (pv.PIVOT_REFINE_FUSED, pv.PIVOT_REFINE_SPLIT):
        say("paged refine path", path)
        outs[path] = host(pv.pivot_group_index_layout(
            dev(x.q[p0:p0 + n_q]), dev(x.q_scale[p0:p0 + n_q]), dev(x.w[p0:p0 + n_q]), dev(pool), dev(pool_s),
            [p0], [p0 + n_q], 1024, lay, mode=pv.PIVOT_REFINE, g=4, c=2048, refine_path=path))
    _same_sets(outs[pv.PIVOT_REFINE_FUSED], outs[pv.PIVOT_REFINE_SPLIT], "paged")


@pytest.mark.parametrize("case", ["bf16", "window"])
def test_fused_request_outside_its_scope_takes_the_split_path(case):
    """PIVOT_REFINE_FUSED applies to fp8 groups without a window; a bf16 call
    or a windowed one asking for it runs the split path and returns its sets."""
    fmt = "bf16" if case == "bf16" else "fp8"
    x = make_prefill(3000, fmt, seed=64, threads=8)
    p0, n_q, g, c, topk = 1000, 2000, 4, 1024, 256
    n_k = p0 + n_q
    W = 4 if case == "window" else 0
    outs = {}
    for path in (pv.PIVOT_REFINE_FUSED, pv.PIVOT_REFINE_SPLIT):
        say("out-of-scope fused request", case, "path", path)
        outs[path] = host(pv.pivot_group_index_opts(
            dev(x.q[p0:n_k]), dev(None if x.q_scale is None else x.q_scale[p0:n_k]), dev(x.w[p0:n_k]),
            dev(x.k[:n_k]), dev(None if x.k_scale is None else x.k_scale[:n_k]), p0, n_k, topk,
            mode=pv.PIVOT_REFINE, g=g, c=c, window=W, refine_path=path))
    _same_sets(outs[pv.PIVOT_REFINE_FUSED], outs[pv.PIVOT_REFINE_SPLIT], case)
