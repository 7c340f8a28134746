"""GPU parity of the batch layouts: several requests of different lengths and
positions packed into one call (groups restart at every request) and keys
held in a paged pool through a block table.  Every request is checked against
the oracle run on that request alone; the paged results must equal the
contiguous ones exactly (the same arithmetic on the same keys)."""
import numpy as np
import pytest
import torch

import oracle
import paper_2607_24593_amd as pv
from gpu_util import dev, host, say
from parity import check_pivot
from workload.gen import make_decode, make_prefill

pytestmark = pytest.mark.gpu

MODES = {"dense": oracle.DENSE, "reuse": oracle.REUSE, "refine": oracle.REFINE}
PV_MODE = {"reuse": pv.PIVOT_REUSE, "refine": pv.PIVOT_REFINE}

# (keys, first query position, queries) of three prefill requests
SPECS = [(1100, 0, 1100), (5000, 3000, 517), (2500, 0, 64)]


def _page_pool(ks, kss, page, rng):
    """Scatter each request's keys into pages of a shuffled pool; returns the pool,
    its scales and the block table [B, max_pages] (unused entries point at page 0)."""
    counts = [(len(k) + page - 1) // page for k in ks]
    n_pages = sum(counts) + 3                         # a few pages nobody uses
    order = rng.permutation(n_pages)
    d = ks[0].shape[1]
    pool = np.zeros((n_pages * page, d), dtype=ks[0].dtype)
    pool_s = None if kss[0] is None else np.zeros(n_pages * page, dtype=np.float32)
    table = np.zeros((len(ks), max(counts) + 1), dtype=np.int32)
    nxt = 0
    for b, k in enumerate(ks):
        for j in range(counts[b]):
            pg = int(order[nxt])
            nxt += 1
            table[b, j] = pg
            part = k[j * page:(j + 1) * page]
            pool[pg * page:pg * page + len(part)] = part
            if pool_s is not None:
                pool_s[pg * page:pg * page + len(part)] = kss[b][j * page:(j + 1) * page]
    return pool, pool_s, table


def run_batch(xs, specs, mode, topk, g=1, c=0, paged=False, page=64, dense_below=-1, window=0,
              window_kind=pv.PIVOT_WINDOW_SHARED, seed=0):
    fmt = xs[0].dtype
    q = np.concatenate([x.q[p0:p0 + n] for x, (_, p0, n) in zip(xs, specs)])
    qs = None if fmt == "bf16" else np.concatenate([x.q_scale[p0:p0 + n] for x, (_, p0, n) in zip(xs, specs)])
    w = np.concatenate([x.w[p0:p0 + n] for x, (_, p0, n) in zip(xs, specs)])
    cu = np.concatenate([[0], np.cumsum([n for _, _, n in specs])]).tolist()
    pos = [p0 for _, p0, _ in specs]
    nk = [L for L, _, _ in specs]
    ks = [x.k[:L] for x, (L, _, _) in zip(xs, specs)]
    kss = [None if fmt == "bf16" else x.k_scale[:L] for x, (L, _, _) in zip(xs, specs)]
    if paged:
        pool, pool_s, table = _page_pool(ks, kss, page, np.random.default_rng(seed))
        k_t, ks_t = dev(pool), dev(pool_s)
        bt = dev(table)
        layout = pv.make_layout(cu_q=cu, block_table=bt, page_size=page, pool_keys=pool.shape[0])
    else:
        S = max(nk)
        kp = np.zeros((len(specs), S, ks[0].shape[1]), dtype=ks[0].dtype)
        ksp = None if fmt == "bf16" else np.zeros((len(specs), S), dtype=np.float32)
        for b in range(len(specs)):
            kp[b, :nk[b]] = ks[b]
            if ksp is not None:
                ksp[b, :nk[b]] = kss[b]
        k_t, ks_t = dev(kp), dev(ksp)
        layout = pv.make_layout(cu_q=cu)
    say("layout", mode, fmt, "paged" if paged else "contiguous", "specs", specs, "g", g, "c", c, "W", window)
    cand = None
    if mode == "dense":
        idx = pv.pivot_dense_index_layout(dev(q), dev(qs), dev(w), k_t, ks_t, pos, nk, topk, layout)
    else:
        n_groups = sum((n + g - 1) // g for _, _, n in specs)
        width = oracle.cand_width(c, g, window, window_kind)
        ct = torch.full((n_groups, width), -7, dtype=torch.int32, device="cuda") if mode == "refine" else None
        idx = pv.pivot_group_index_layout(dev(q), dev(qs), dev(w), k_t, ks_t, pos, nk, topk, layout,
                                          mode=PV_MODE[mode], g=g, c=c, dense_below=dense_below, window=window,
                                          window_kind=window_kind, out_cand=ct)
        cand = None if ct is None else host(ct)
    return host(idx), cand, cu


def check_batch(xs, specs, mode, topk, idx, cand, cu, g=1, c=0, dense_below=-1, window=0,
                window_kind=pv.PIVOT_WINDOW_SHARED, groups=None):
    fmt = xs[0].dtype
    g0 = 0
    for r, (x, (L, p0, n)) in enumerate(zip(xs, specs)):
        rows = slice(cu[r], cu[r + 1])
        gg = 1 if mode == "dense" else g
        ng = (n + gg - 1) // gg
        check_pivot(fmt, x.q[p0:p0 + n], None if fmt == "bf16" else x.q_scale[p0:p0 + n], x.w[p0:p0 + n], p0,
                    x.k[:L], None if fmt == "bf16" else x.k_scale[:L], L, mode=MODES[mode], g=gg, c=c, topk=topk,
                    dense_below=dense_below, gpu_idx=idx[rows],
                    gpu_cand=None if cand is None else cand[g0:g0 + ng], groups=None if groups is None else groups[r],
                    label=f"request {r}", window=window, window_kind=window_kind)
        g0 += ng


@pytest.fixture(scope="module")
def reqs_fp8():
    return [make_prefill(L, "fp8", seed=80 + i, threads=4) for i, (L, _, _) in enumerate(SPECS)]


@pytest.fixture(scope="module")
def reqs_bf16():
    return [make_prefill(L, "bf16", seed=90 + i, threads=4) for i, (L, _, _) in enumerate(SPECS)]


def _groups(specs, g, c, rng):
    out = []
    for L, p0, n in specs:
        ng = (n + g - 1) // g
        pick = {0, ng - 1} | set(int(v) for v in rng.integers(0, ng, 6))
        j = (c - p0) // g
        if 0 <= j < ng:
            pick |= {j, max(0, j - 1)}
        out.append(sorted(pick))
    return out


@pytest.mark.parametrize("paged", [False, True])
@pytest.mark.parametrize("mode", ["dense", "reuse", "refine"])
def test_varlen_batch_fp8(reqs_fp8, mode, paged):
    """Three fp8 requests (a whole 1100-token prefill, a chunk at 3000 of a
    5000-key prefix, 64 queries of a 2500-key one) in one call, g=4, c=256."""
    g, c, topk = (1, 0, 128) if mode == "dense" else (4, 256, 128)
    idx, cand, cu = run_batch(reqs_fp8, SPECS, mode, topk, g, c, paged=paged, seed=1)
    groups = _groups(SPECS, g, c, np.random.default_rng(3))
    check_batch(reqs_fp8, SPECS, mode, topk, idx, cand, cu, g, c, groups=groups)


@pytest.mark.parametrize("mode", ["dense", "reuse", "refine"])
def test_paged_equals_contiguous(reqs_bf16, mode):
    """bf16, every query: the paged pool (pages of 16 keys, shuffled) gives the
    contiguous layout's indices exactly, and both pass the oracle."""
    g, c, topk = (1, 0, 64) if mode == "dense" else (3, 128, 64)
    a, ca, cu = run_batch(reqs_bf16, SPECS, mode, topk, g, c, paged=False, dense_below=0)
    b, cb, _ = run_batch(reqs_bf16, SPECS, mode, topk, g, c, paged=True, page=16, dense_below=0, seed=5)
    assert np.array_equal(np.sort(a, 1), np.sort(b, 1))
    if ca is not None:
        assert np.array_equal(np.sort(ca, 1), np.sort(cb, 1))
    check_batch(reqs_bf16, SPECS, mode, topk, b, cb, cu, g, c, dense_below=0)


def test_varlen_window_paged(reqs_fp8):
    """App. B's prefill window on the packed, paged batch."""
    g, c, topk, W = 4, 256, 128, 8
    idx, cand, cu = run_batch(reqs_fp8, SPECS, "refine", topk, g, c, paged=True, page=32, dense_below=0, window=W,
                              seed=7)
    groups = _groups(SPECS, g, c, np.random.default_rng(4))
    check_batch(reqs_fp8, SPECS, "refine", topk, idx, cand, cu, g, c, dense_below=0, window=W, groups=groups)


def test_empty_and_single_query_runs(reqs_fp8):
    """Runs of 0 and 1 queries between others."""
    specs = [(SPECS[0][0], 500, 0), (SPECS[1][0], 4999, 1), (SPECS[2][0], 2400, 100)]
    for mode in ("dense", "reuse", "refine"):
        g, c = (1, 0) if mode == "dense" else (4, 256)
        idx, cand, cu = run_batch(reqs_fp8, specs, mode, 64, g, c, paged=True, seed=9)
        check_batch(reqs_fp8, specs, mode, 64, idx, cand, cu, g, c)


@pytest.mark.parametrize("mode", ["dense", "reuse", "refine"])
def test_paged_decode_batch(mode):
    """Decode over paged caches of different lengths (8 sequences, 17000 to
    40000 keys, pages of 64): equals the padded contiguous batch exactly."""
    B, g, topk, c = 8, 2, 256, 1024
    lens = [17000 + 3000 * b for b in range(B)]
    S = max(lens)
    x = make_decode(B, S, g, "fp8", seed=95, threads=8)
    # each sequence's MTP queries sit at its own last two positions
    kp = x.k.copy()
    ksp = x.k_scale.copy()
    pos = [L - g for L in lens]
    q, qs, w = dev(x.q), dev(x.q_scale), dev(x.w)
    say("paged decode", mode, lens)
    if mode == "dense":
        ref = pv.pivot_dense_index(q, qs, w, dev(kp), dev(ksp), pos, lens, topk)
    else:
        ref = pv.pivot_group_index(q, qs, w, dev(kp), dev(ksp), pos, lens, topk, mode=PV_MODE[mode], g=g, c=c)
    ref = host(ref).reshape(B * g, topk)
    ks = [kp[b, :lens[b]] for b in range(B)]
    kss = [ksp[b, :lens[b]] for b in range(B)]
    pool, pool_s, table = _page_pool(ks, kss, 64, np.random.default_rng(11))
    layout = pv.make_layout(cu_q=[g * b for b in range(B + 1)], block_table=dev(table), page_size=64,
                            pool_keys=pool.shape[0])
    qf, qsf, wf = q.reshape(B * g, 64, 128), qs.reshape(B * g), w.reshape(B * g, 64)
    ct = torch.full((B, c), -7, dtype=torch.int32, device="cuda") if mode == "refine" else None
    if mode == "dense":
        got = pv.pivot_dense_index_layout(qf, qsf, wf, dev(pool), dev(pool_s), pos, lens, topk, layout)
    else:
        got = pv.pivot_group_index_layout(qf, qsf, wf, dev(pool), dev(pool_s), pos, lens, topk, layout,
                                          mode=PV_MODE[mode], g=g, c=c, out_cand=ct)
    got = host(got)
    cand = None if ct is None else host(ct)
    assert np.array_equal(np.sort(got, 1), np.sort(ref, 1))
    for b in (0, B - 1):
        check_pivot("fp8", x.q[b], x.q_scale[b], x.w[b], pos[b], kp[b, :lens[b]], ksp[b, :lens[b]], lens[b],
                    mode=MODES[mode], g=1 if mode == "dense" else g, c=c, topk=topk, dense_below=-1,
                    gpu_idx=got[b * g:(b + 1) * g], gpu_cand=None if cand is None else cand[b:b + 1],
                    label=f"paged decode b{b}")


@pytest.mark.parametrize("mode", ["dense", "reuse", "refine"])
def test_more_sequences_than_one_launch(mode):
    """80 decode sequences (a launch's sequence table holds 64): the host splits
    every stage; packed runs of 1 to 3 queries with their own lengths."""
    B, L, topk, c = 80, 3000, 128, 512
    x = make_decode(B, L, 3, "bf16", seed=97, threads=8)
    rng = np.random.default_rng(13)
    runs = [int(v) for v in rng.integers(1, 4, B)]           # 1..3 queries per sequence
    lens = [int(v) for v in rng.integers(2000, L + 1, B)]
    pos = [lens[b] - runs[b] for b in range(B)]
    q = np.concatenate([x.q[b, :runs[b]] for b in range(B)])
    w = np.concatenate([x.w[b, :runs[b]] for b in range(B)])
    cu = [0] + np.cumsum(runs).tolist()
    kp = x.k.copy()
    layout = pv.make_layout(cu_q=cu)
    g = 2
    say("80 sequences", mode)
    cand = None
    if mode == "dense":
        idx = pv.pivot_dense_index_layout(dev(q), None, dev(w), dev(kp), None, pos, lens, topk, layout)
    else:
        ng = sum((r + g - 1) // g for r in runs)
        ct = torch.full((ng, c), -7, dtype=torch.int32, device="cuda") if mode == "refine" else None
        idx = pv.pivot_group_index_layout(dev(q), None, dev(w), dev(kp), None, pos, lens, topk, layout,
                                          mode=PV_MODE[mode], g=g, c=c, dense_below=0, out_cand=ct)
        cand = None if ct is None else host(ct)
    idx = host(idx)
    g0 = 0
    for b in range(B):
        ng_b = 1 if mode == "dense" else (runs[b] + g - 1) // g
        if b in (0, 1, 63, 64, 65, B - 1) or b % 11 == 0:
            check_pivot("bf16", x.q[b, :runs[b]], None, x.w[b, :runs[b]], pos[b], kp[b, :lens[b]], None, lens[b],
                        mode=MODES[mode], g=1 if mode == "dense" else g, c=c, topk=topk, dense_below=0,
                        gpu_idx=idx[cu[b]:cu[b + 1]],
                        gpu_cand=None if cand is None else cand[g0:g0 + ng_b], label=f"seq {b}")
        g0 += (runs[b] + g - 1) // g if mode != "dense" else 0
