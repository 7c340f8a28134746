"""GPU parity of PIVOT's options beyond Algorithm 1, through
pivot_group_index_opts: App. B's local window (the shared prefill union and the
per-query decode pool) and the first / last member as the proxy (the query
aggregation ablation of Sec. 5.4), against the oracle on the same inputs."""
import numpy as np
import pytest
import torch

import oracle
import paper_2607_24593_amd as pv
from gpu_util import dev, host, say
from parity import check_pivot
from workload.gen import make_decode, make_prefill

pytestmark = pytest.mark.gpu

MODES = {"reuse": oracle.REUSE, "refine": oracle.REFINE}
PV_MODE = {"reuse": pv.PIVOT_REUSE, "refine": pv.PIVOT_REFINE}
KIND = {"shared": pv.PIVOT_WINDOW_SHARED, "per_query": pv.PIVOT_WINDOW_PER_QUERY}


def run_opts(x, mode, p0, n_q, topk, g, c, dense_below=-1, window=0, kind="shared", agg=pv.PIVOT_AGG_MEAN,
             want_cand=True):
    q = x.q[p0:p0 + n_q]
    qs = None if x.q_scale is None else x.q_scale[p0:p0 + n_q]
    w = x.w[p0:p0 + n_q]
    n_k = p0 + n_q
    say("opts", mode, x.dtype, "p0", p0, "n_q", n_q, "topk", topk, "g", g, "c", c, "db", dense_below, "W", window,
        kind, "agg", agg)
    width = oracle.cand_width(c, g, window, KIND[kind])
    ng = (n_q + g - 1) // g
    cand_t = None
    if mode == "refine" and want_cand:
        cand_t = torch.full((1, ng, width), -7, dtype=torch.int32, device="cuda")
    idx = pv.pivot_group_index_opts(dev(q), dev(qs), dev(w), dev(x.k[:n_k]),
                                    dev(None if x.k_scale is None else x.k_scale[:n_k]), p0, n_k, topk,
                                    mode=PV_MODE[mode], g=g, c=c, dense_below=dense_below, window=window,
                                    window_kind=KIND[kind], aggregate=agg, out_cand=cand_t)
    return host(idx), (None if cand_t is None else host(cand_t)[0]), (q, qs, w, n_k)


def check(x, mode, p0, n_q, topk, g, c, dense_below=-1, window=0, kind="shared", agg=pv.PIVOT_AGG_MEAN,
          groups=None, label=""):
    idx, cand, (q, qs, w, n_k) = run_opts(x, mode, p0, n_q, topk, g, c, dense_below, window, kind, agg)
    return check_pivot(x.dtype, q, qs, w, p0, x.k[:n_k], None if x.k_scale is None else x.k_scale[:n_k], n_k,
                       mode=MODES[mode], g=g, c=c, topk=topk, dense_below=dense_below, gpu_idx=idx,
                       gpu_cand=cand, groups=groups, label=label, window=window, window_kind=KIND[kind], agg=agg)


def _groups(n_q, g, p0, c, W, seed, extra=()):
    rng = np.random.default_rng(seed)
    ng = (n_q + g - 1) // g
    pick = {0, 1, 2, ng - 1, ng - 2} | set(int(v) for v in rng.integers(0, ng, 10))
    for t in (W - g, W, W + g, c - g, c, c + g, c + W) + tuple(extra):  # where the window or the guardrail ends
        j = (t - p0) // g
        if 0 <= j < ng:
            pick.add(j)
    return sorted(pick)


@pytest.fixture(scope="module")
def small_bf16():
    return make_prefill(1100, "bf16", seed=51, threads=4)


@pytest.fixture(scope="module")
def long_fp8():
    return make_prefill(6000, "fp8", seed=52, threads=8)


@pytest.mark.parametrize("dense_below", [-1, 0])
def test_shared_window_bf16_every_query(small_bf16, dense_below):
    """Prefill window W=16 with g=4 on every query of a 1100-position bf16 prefill
    (ragged last group); without the guardrail the first groups' proxy range
    [0, t0 - W] is empty or short."""
    check(small_bf16, "refine", 0, 1099, 64, g=4, c=256, dense_below=dense_below, window=16,
          label=f"bf16 W16 db{dense_below}")


@pytest.mark.parametrize("g,W,c,topk", [(4, 64, 1024, 256), (8, 128, 2048, 512), (2, 5, 1024, 256)])
def test_shared_window_fp8(long_fp8, g, W, c, topk):
    """Prefill window on 5999 fp8 queries (key segments of 4096, ragged tail), sampled groups."""
    n_q = 5999
    groups = _groups(n_q, g, 0, c, W, seed=g + W, extra=(4095, 4096))
    check(long_fp8, "refine", 0, n_q, topk, g=g, c=c, dense_below=0, window=W, groups=groups,
          label=f"fp8 shared g{g} W{W}")


def test_shared_window_takes_all_slots(small_bf16):
    """c = W + g - 1: the union fills every slot and the proxy scan is skipped."""
    check(small_bf16, "refine", 0, 1099, 32, g=4, c=64, dense_below=0, window=61, label="bf16 W61 c64")


def test_shared_window_chunk_with_offset(long_fp8):
    """A later chunk of a prefill with the window: queries 3000 .. 5999."""
    p0, n_q, g, c = 3000, 3000, 4, 1024
    groups = _groups(n_q, g, p0, c, 64, seed=7)
    check(long_fp8, "refine", p0, n_q, 256, g=g, c=c, window=64, groups=groups, label="chunk W64")


def test_window_without_cand_output(long_fp8):
    """The candidate rows in the workspace give the indices of the run with out_cand."""
    a, _, _ = run_opts(long_fp8, "refine", 2000, 1000, 128, 4, 512, window=32, want_cand=False)
    b, _, _ = run_opts(long_fp8, "refine", 2000, 1000, 128, 4, 512, window=32, want_cand=True)
    assert np.array_equal(np.sort(a, 1), np.sort(b, 1))


@pytest.mark.parametrize("agg", [pv.PIVOT_AGG_FIRST, pv.PIVOT_AGG_LAST])
@pytest.mark.parametrize("mode", ["reuse", "refine"])
def test_first_last_aggregation(long_fp8, small_bf16, mode, agg):
    """The first or the last member stands for its group (fp8 sampled groups, bf16 every query)."""
    n_q, g, c = 5999, 4, 1024
    groups = _groups(n_q, g, 0, c, 0, seed=agg)
    check(long_fp8, mode, 0, n_q, 256, g=g, c=c, agg=agg, groups=groups, label=f"fp8 {mode} agg{agg}")
    check(small_bf16, mode, 0, 1099, 64, g=3, c=256, dense_below=0, agg=agg, label=f"bf16 {mode} agg{agg}")


def test_aggregation_with_window(long_fp8):
    """The last member as proxy together with the prefill window."""
    n_q, g, c = 5999, 4, 1024
    groups = _groups(n_q, g, 0, c, 64, seed=11)
    check(long_fp8, "refine", 0, n_q, 256, g=g, c=c, window=64, agg=pv.PIVOT_AGG_LAST, groups=groups,
          label="fp8 W64 last")


@pytest.mark.parametrize("B,L,g,W", [(5, 5000, 2, 4), (5, 5000, 3, 3), (4, 20000, 4, 64), (3, 3000, 2, 2)])
def test_per_query_window_decode(B, L, g, W):
    """Decode: each of the g MTP queries adds its own W-window to the proxy's
    top-c pool (20000-key contexts take the split select and split re-score)."""
    x = make_decode(B, L, g, "fp8", seed=60 + g + W, threads=6)
    say("decode window", "B", B, "L", L, "g", g, "W", W)
    topk, c = 256, 1024
    width = c + W + g - 1
    cand_t = torch.full((B, 1, width), -7, dtype=torch.int32, device="cuda")
    idx = pv.pivot_group_index_opts(dev(x.q), dev(x.q_scale), dev(x.w), dev(x.k), dev(x.k_scale), [L - g] * B,
                                    [L] * B, topk, mode=pv.PIVOT_REFINE, g=g, c=c, window=W,
                                    window_kind=pv.PIVOT_WINDOW_PER_QUERY, out_cand=cand_t)
    idx, cand = host(idx), host(cand_t)
    for b in range(B):
        check_pivot("fp8", x.q[b], x.q_scale[b], x.w[b], L - g, x.k[b], x.k_scale[b], L, mode=oracle.REFINE, g=g,
                    c=c, topk=topk, dense_below=-1, gpu_idx=idx[b], gpu_cand=cand[b], label=f"decode W{W} b{b}",
                    window=W, window_kind=oracle.WINDOW_PER_QUERY)


def test_per_query_window_short_context():
    """A decode context shorter than c: the pool holds every position up to t0,
    so the window union keeps only the last member's own position, and members
    keep all they may use."""
    B, L, g, W = 3, 700, 2, 8
    x = make_decode(B, L, g, "bf16", seed=77, threads=4)
    topk, c = 512, 1024
    cand_t = torch.full((B, 1, c + W + g - 1), -7, dtype=torch.int32, device="cuda")
    say("decode window short", "L", L)
    idx = pv.pivot_group_index_opts(dev(x.q), None, dev(x.w), dev(x.k), None, [L - g] * B, [L] * B, topk,
                                    mode=pv.PIVOT_REFINE, g=g, c=c, dense_below=0, window=W,
                                    window_kind=pv.PIVOT_WINDOW_PER_QUERY, out_cand=cand_t)
    idx, cand = host(idx), host(cand_t)
    for b in range(B):
        # the pool holds every position <= t0; only the last member's own position is new
        assert (cand[b, 0, c:-1] == -1).all() and cand[b, 0, -1] == L - 1
        check_pivot("bf16", x.q[b], None, x.w[b], L - g, x.k[b], None, L, mode=oracle.REFINE, g=g, c=c, topk=topk,
                    dense_below=0, gpu_idx=idx[b], gpu_cand=cand[b], label=f"short b{b}", window=W,
                    window_kind=oracle.WINDOW_PER_QUERY)
