"""GPU parity at the full sizes of the five named workloads, called exactly as
bench.py calls the library (one call per prefill chunk against the full causal
prefix; one batched call per decode step), checked against the oracle on
sampled groups: the guardrail boundary, chunk edges, the last group and random
positions.  The 2K bf16 prefill is checked on every query."""
import numpy as np
import pytest
import torch

import oracle
import paper_2607_24593_amd as pv
from gpu_util import dev, host, say
import parity
from parity import check_pivot
from workload.gen import WORKLOADS, make

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True)
def tolerance_budget(request):
    """Reports, per test, how many checked rows differ from the oracle's set
    and how much of the tolerance their boundary swaps used, and requires the
    swaps to fit the path's error model (parity.SWAP_BOUND), not just rtol."""
    parity.BUDGET = parity.Budget()
    yield
    say("tolerance budget", request.node.name, parity.BUDGET.summary())
    assert parity.BUDGET.worst <= 1.0, ("boundary swaps beyond the error model", parity.BUDGET.summary())

MODES = {"dense": oracle.DENSE, "reuse": oracle.REUSE, "refine": oracle.REFINE}


class Resident:
    """A workload's inputs in HBM plus host copies for the oracle."""

    def __init__(self, name):
        self.wl = WORKLOADS[name]
        say("generate", name)
        self.x = make(self.wl, threads=16)
        self.q, self.qs, self.w = dev(self.x.q), dev(self.x.q_scale), dev(self.x.w)
        self.k, self.ks = dev(self.x.k), dev(self.x.k_scale)

    def run_chunk(self, mode, g, p0, n, window=0, dense_below=-1):
        wl = self.wl
        sl = slice(p0, p0 + n)
        args = (self.q[sl], None if self.qs is None else self.qs[sl], self.w[sl], self.k[:p0 + n],
                None if self.ks is None else self.ks[:p0 + n], p0, p0 + n, wl.topk)
        say(wl.name, mode, "g", g, "chunk", p0, n, "W", window, "db", dense_below)
        cand = None
        if mode == "dense":
            idx = pv.pivot_dense_index(*args)
        else:
            ng = (n + g - 1) // g
            ct = torch.full((1, ng, wl.c), -7, dtype=torch.int32, device="cuda") if mode == "refine" else None
            pm = pv.PIVOT_REUSE if mode == "reuse" else pv.PIVOT_REFINE
            if window:  # App. B's prefill window
                idx = pv.pivot_group_index_opts(*args, mode=pm, g=g, c=wl.c, dense_below=dense_below,
                                                window=window, window_kind=pv.PIVOT_WINDOW_SHARED, out_cand=ct)
            else:
                idx = pv.pivot_group_index(*args, mode=pm, g=g, c=wl.c, dense_below=dense_below, out_cand=ct)
            cand = None if ct is None else host(ct)[0]
        return host(idx), cand

    def check_chunk(self, mode, g, p0, n, groups, label, window=0, dense_below=-1):
        idx, cand = self.run_chunk(mode, g, p0, n, window, dense_below)
        x, wl = self.x, self.wl
        sl = slice(p0, p0 + n)
        return check_pivot(x.dtype, x.q[sl], None if x.q_scale is None else x.q_scale[sl], x.w[sl], p0,
                           x.k[:p0 + n], None if x.k_scale is None else x.k_scale[:p0 + n], p0 + n,
                           mode=MODES[mode], g=g if mode != "dense" else 1, c=wl.c, topk=wl.topk,
                           dense_below=dense_below, gpu_idx=idx, gpu_cand=cand, groups=groups, label=label,
                           window=window, window_kind=oracle.WINDOW_SHARED)


def sample_groups(p0, n, g, c, rng, count=8):
    ng = (n + g - 1) // g
    pick = {0, ng - 1} | set(int(v) for v in rng.integers(0, ng, count))
    for t in (c - g, c, c + g):                 # around Algorithm 1's guardrail
        j = (t - p0) // g
        if 0 <= j < ng:
            pick.add(j)
    return sorted(pick)


@pytest.fixture(scope="module")
def cfg0():
    return Resident("prefill-2k-bf16")


@pytest.mark.parametrize("mode", ["dense", "reuse", "refine"])
def test_prefill_2k_bf16_every_query(cfg0, mode):
    wl = cfg0.wl
    swaps = cfg0.check_chunk(mode, wl.g[0], 0, wl.L, None, f"2k bf16 {mode}")
    say("boundary swaps", swaps)


@pytest.fixture(scope="module")
def cfg1():
    return Resident("prefill-32k-fp8")


@pytest.mark.parametrize("mode", ["dense", "reuse", "refine"])
def test_prefill_32k_fp8(cfg1, mode):
    wl = cfg1.wl
    g = wl.g[0] if mode != "dense" else 1
    groups = sample_groups(0, wl.L, g, wl.c, np.random.default_rng(1), 10)
    cfg1.check_chunk(mode, g, 0, wl.L, groups, f"32k {mode}")


@pytest.fixture(scope="module")
def cfg2():
    return Resident("prefill-128k-fp8")


@pytest.mark.parametrize("g", [2, 4, 8])
@pytest.mark.parametrize("mode", ["reuse", "refine"])
def test_prefill_128k_fp8_chunks(cfg2, mode, g):
    """Chunks of 8192 queries: the first (guardrail boundary), a middle one and the last."""
    wl = cfg2.wl
    rng = np.random.default_rng(g)
    for p0 in (0, 65536, wl.L - wl.chunk):
        groups = sample_groups(p0, wl.chunk, g, wl.c, rng, 4)
        cfg2.check_chunk(mode, g, p0, wl.chunk, groups, f"128k {mode} g{g} p0 {p0}")


@pytest.mark.parametrize("dense_below", [-1, 0])
def test_prefill_128k_fp8_window(cfg2, dense_below):
    """App. B's window at the paper's W = 4 (g = 4, c = 4096): the first chunk
    (with and without the guardrail) and the last chunk."""
    wl = cfg2.wl
    g, W = 4, 4
    rng = np.random.default_rng(21)
    for p0 in ((0,) if dense_below == 0 else (0, wl.L - wl.chunk)):
        groups = sample_groups(p0, wl.chunk, g, wl.c, rng, 4)
        if p0 == 0:
            groups = sorted(set(groups) | {1, 2})      # proxy ranges [0, t0 - W] empty or short
        cfg2.check_chunk("refine", g, p0, wl.chunk, groups, f"128k W{W} db{dense_below} p0 {p0}", window=W,
                         dense_below=dense_below)


def test_prefill_128k_fp8_dense(cfg2):
    wl = cfg2.wl
    rng = np.random.default_rng(7)
    for p0 in (0, wl.L - wl.chunk):
        rows = sample_groups(p0, wl.chunk, 1, wl.c, rng, 6)
        cfg2.check_chunk("dense", 1, p0, wl.chunk, rows, f"128k dense p0 {p0}")


@pytest.mark.parametrize("mode", ["dense", "reuse", "refine"])
def test_decode_32x128k(mode):
    wl = WORKLOADS["decode-32x128k-fp8"]
    x = make(wl, threads=16)
    B, L, g = wl.batch, wl.L, wl.g[0]
    say("decode", mode, B, L, g)
    q, qs, w, k, ks = dev(x.q), dev(x.q_scale), dev(x.w), dev(x.k), dev(x.k_scale)
    cand = None
    if mode == "dense":
        idx = pv.pivot_dense_index(q, qs, w, k, ks, [L - g] * B, [L] * B, wl.topk)
    else:
        ct = torch.full((B, 1, wl.c), -7, dtype=torch.int32, device="cuda") if mode == "refine" else None
        idx = pv.pivot_group_index(q, qs, w, k, ks, [L - g] * B, [L] * B, wl.topk,
                                   mode=pv.PIVOT_REUSE if mode == "reuse" else pv.PIVOT_REFINE, g=g, c=wl.c,
                                   out_cand=ct)
        cand = None if ct is None else host(ct)
    idx = host(idx)
    for b in (0, 5, 13, 21, 30, 31):
        check_pivot("fp8", x.q[b], x.q_scale[b], x.w[b], L - g, x.k[b], x.k_scale[b], L, mode=MODES[mode], g=g,
                    c=wl.c, topk=wl.topk, dense_below=-1, gpu_idx=idx[b],
                    gpu_cand=None if cand is None else cand[b], label=f"decode {mode} b{b}")


def test_decode_32x128k_window():
    """Decode with App. B's per-query window (W = 4 >= g = 2): c + W + g - 1 slots per group."""
    wl = WORKLOADS["decode-32x128k-fp8"]
    x = make(wl, threads=16)
    B, L, g, W = wl.batch, wl.L, wl.g[0], 4
    say("decode window", B, L, g, W)
    q, qs, w, k, ks = dev(x.q), dev(x.q_scale), dev(x.w), dev(x.k), dev(x.k_scale)
    ct = torch.full((B, 1, wl.c + W + g - 1), -7, dtype=torch.int32, device="cuda")
    idx = pv.pivot_group_index_opts(q, qs, w, k, ks, [L - g] * B, [L] * B, wl.topk, mode=pv.PIVOT_REFINE, g=g,
                                    c=wl.c, window=W, window_kind=pv.PIVOT_WINDOW_PER_QUERY, out_cand=ct)
    idx, cand = host(idx), host(ct)
    for b in (0, 7, 19, 31):
        check_pivot("fp8", x.q[b], x.q_scale[b], x.w[b], L - g, x.k[b], x.k_scale[b], L, mode=oracle.REFINE, g=g,
                    c=wl.c, topk=wl.topk, dense_below=-1, gpu_idx=idx[b], gpu_cand=cand[b],
                    label=f"decode W{W} b{b}", window=W, window_kind=oracle.WINDOW_PER_QUERY)


@pytest.fixture(scope="module")
def cfg4():
    return Resident("prefill-256k-fp8-pareto")


@pytest.mark.parametrize("mode", ["dense", "refine"])
def test_prefill_256k_fp8_pareto(cfg4, mode):
    """Chunks of 16384 queries against up to 262144 keys (the largest rows)."""
    wl = cfg4.wl
    g = wl.g[0] if mode != "dense" else 1
    rng = np.random.default_rng(11)
    for p0 in (0, wl.L - wl.chunk):
        groups = sample_groups(p0, wl.chunk, g, wl.c, rng, 5 if mode == "refine" else 3)
        cfg4.check_chunk(mode, g, p0, wl.chunk, groups, f"256k {mode} p0 {p0}")
