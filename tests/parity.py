"""Parity rule between a GPU index set and the oracle's.

For one output row with oracle set O (top-m of the oracle scores f over a
domain D) and GPU set G, both padded with -1:
  * same number of -1 entries, no duplicates, G within D;
  * with tau = the oracle score of O's m-th element (its minimum) and
    tol = rtol * |tau|: every s in G \\ O has f(s) >= tau - tol and every s in
    O \\ G has f(s) <= tau + tol.
rtol is 2e-3 for bf16 inputs and 2e-2 for fp8 inputs (scores compared with the
fp64 oracle).  Scores are only computed for rows whose sets differ.

Besides the tolerance, the swaps must fit the error model of the path
(SWAP_BOUND, relative to |tau|): with fp8 inputs the GPU ranks bf16-rounded
scores (unit roundoff 2^-8), so two scores change order only when their exact
values lie within 2 * 2^-8 of each other, plus at most 2e-3 for the fp8
linear term's last residual and the fp32 sums; bf16 inputs rank fp32 sums.
"""
from __future__ import annotations

import numpy as np

RTOL = {"bf16": 2e-3, "fp8": 2e-2}
SWAP_BOUND = {"bf16": 1e-4, "fp8": 2 * 2.0 ** -8 + 2e-3}


class ParityError(AssertionError):
    pass


class Budget:
    """How much of the tolerance the checked rows used: rows checked, rows
    whose set differs from the oracle's, boundary swaps (GPU entries outside
    the oracle set), the most swaps in one row, and the largest |f - tau| /
    |tau| over swapped entries (compare with rtol)."""

    def __init__(self):
        self.rows = self.rows_diff = self.swaps = self.max_row_swaps = 0
        self.max_rel = 0.0
        self.worst = 0.0  # largest max_rel / SWAP_BOUND of the rows' format

    def add(self, swaps, rel, bound=None):
        self.rows += 1
        if swaps:
            self.rows_diff += 1
            self.swaps += swaps
            self.max_row_swaps = max(self.max_row_swaps, swaps)
            self.max_rel = max(self.max_rel, rel)
            if bound:
                self.worst = max(self.worst, rel / bound)

    def summary(self):
        return (f"{self.rows} rows, {self.rows_diff} not identical to the oracle's set, {self.swaps} boundary "
                f"swaps (at most {self.max_row_swaps} in a row), largest |f - tau|/|tau| of a swapped entry "
                f"{self.max_rel:.2e}")


BUDGET = Budget()  # accumulated by check_row; tests reset and report it


def check_row(gpu, ora, f_of, rtol, in_domain, label="", swap_bound=None):
    """gpu, ora: int arrays (-1 padded); f_of(idx array) -> oracle fp64 scores;
    in_domain(idx array) -> bool array; swap_bound: the path's SWAP_BOUND,
    recorded in BUDGET.  Returns the number of boundary swaps."""
    gpu = np.asarray(gpu)
    ora = np.asarray(ora)
    G = gpu[gpu >= 0]
    O = ora[ora >= 0]
    if (gpu < -1).any():
        raise ParityError(f"{label}: invalid entries {gpu[gpu < -1][:5]}")
    if len(np.unique(G)) != len(G):
        raise ParityError(f"{label}: duplicate indices")
    if (gpu == -1).sum() != (ora == -1).sum():
        raise ParityError(f"{label}: {(gpu == -1).sum()} pads vs oracle {(ora == -1).sum()}")
    if len(G) and not in_domain(G).all():
        raise ParityError(f"{label}: indices outside the domain: {G[~in_domain(G)][:5]}")
    sg, so = set(G.tolist()), set(O.tolist())
    if sg == so:
        BUDGET.add(0, 0.0)
        return 0
    extra = np.array(sorted(sg - so), dtype=np.int64)
    missing = np.array(sorted(so - sg), dtype=np.int64)
    tau = float(f_of(O).min())
    tol = rtol * abs(tau)
    fe = f_of(extra)
    fm = f_of(missing)
    if (fe < tau - tol).any() or (fm > tau + tol).any():
        raise ParityError(f"{label}: tau={tau:.6g} tol={tol:.3g}; extra f={np.sort(fe)[:4]}, "
                          f"missing f={np.sort(fm)[-4:]}")
    dev = max(float(np.max(tau - fe, initial=0.0)), float(np.max(fm - tau, initial=0.0)))
    BUDGET.add(len(extra), dev / abs(tau) if tau != 0 else 0.0, swap_bound)
    return len(extra)


def check_pivot(fmt, q, qs, w, p0, k, ks, n_k, *, mode, g, c, topk, dense_below, gpu_idx,
                gpu_cand=None, groups=None, label="", window=0, window_kind=0, agg=0):
    """Check one sequence's GPU result against the oracle (Algorithm 1).

    q / qs / w: the call's n_q query rows (numpy); k / ks: the sequence's keys.
    mode: oracle.DENSE / REUSE / REFINE.  Refine needs gpu_cand ([n_groups,
    width]) for the two-stage check: (1) the candidate set against the
    oracle's proxy top-c, (2) each member's set against the oracle's Refine
    run on the GPU's own candidates.  With App. B's window (window > 0) the
    proxy's slots are checked as in (1) over the proxy's own range, the window
    union exactly (it follows from t0, W, g and, per query, the GPU's pool),
    and member t against the oracle's Refine over the slots it may use.
    agg: the proxy aggregation.  Returns the number of boundary swaps accepted."""
    import oracle

    rtol = RTOL[fmt]
    sb = SWAP_BOUND[fmt]
    n_q = q.shape[0]
    if mode == oracle.DENSE:
        g, db = 1, n_k + 1
    else:
        db = c if dense_below < 0 else dense_below
    res = oracle.index(fmt, q, qs, w, p0, k, ks, n_k, mode=mode, g=g, c=c, topk=topk,
                       dense_below=(0 if mode == oracle.DENSE else db), groups=groups,
                       want_cand=(mode == oracle.REFINE), want_proxy=(mode != oracle.DENSE),
                       window=window, window_kind=window_kind, agg=agg)
    n_groups = (n_q + g - 1) // g
    sel = range(n_groups) if groups is None else groups
    swaps = 0

    def member_scores(r):
        return lambda idx: oracle.scores_at(fmt, q[r], 1.0 if qs is None else qs[r], w[r], k, ks, idx)

    for j in sel:
        t0 = p0 + j * g
        gs = min(g, n_q - j * g)
        rows = list(range(j * g, j * g + gs))
        if mode == oracle.DENSE or t0 < db:
            for r in rows:
                t = p0 + r
                swaps += check_row(gpu_idx[r], res["idx"][r], member_scores(r), rtol,
                                   lambda idx, t=t: (idx >= 0) & (idx <= t), f"{label} dense row {r}", swap_bound=sb)
            if mode == oracle.REFINE and gpu_cand is not None:
                if not (gpu_cand[j] == -1).all():
                    raise ParityError(f"{label}: guardrail group {j} has candidates")
            continue
        pq, psc, pw = res["pq"][j], res["psc"][j], res["pw"][j]

        def fbar(idx, pq=pq, psc=psc, pw=pw):
            return oracle.scores_at(fmt, pq, psc, pw, k, ks, idx)

        def dom0(idx, t0=t0):
            return (idx >= 0) & (idx <= t0)

        if mode == oracle.REUSE:
            for r in rows:
                swaps += check_row(gpu_idx[r], res["idx"][r], fbar, rtol, dom0, f"{label} reuse row {r}",
                                   swap_bound=sb)
            continue
        if window > 0:
            swaps += _check_window_group(fmt, q, qs, w, k, ks, rows, t0, gs, c, g, topk, window, window_kind,
                                         gpu_idx, gpu_cand[j], res["cand"][j], fbar, rtol, member_scores,
                                         f"{label} group {j}")
            continue
        swaps += check_row(gpu_cand[j], res["cand"][j], fbar, rtol, dom0, f"{label} candidates of group {j}",
                           swap_bound=sb)
        C = gpu_cand[j][gpu_cand[j] >= 0]
        ref2 = oracle.refine_on(fmt, q[rows], None if qs is None else qs[rows], w[rows], k, ks, C, topk)
        for u, r in enumerate(rows):
            swaps += check_row(gpu_idx[r], ref2[u], member_scores(r), rtol,
                               lambda idx, C=C: np.isin(idx, C), f"{label} refine row {r}", swap_bound=sb)
    return swaps


def _check_window_group(fmt, q, qs, w, k, ks, rows, t0, gs, c, g, topk, W, kind, gpu_idx, gcand, ocand, fbar,
                        rtol, member_scores, label):
    """One Refine group with App. B's window (see check_pivot)."""
    import oracle

    sb = SWAP_BOUND[fmt]
    wg = W + g - 1
    per_query = kind == oracle.WINDOW_PER_QUERY
    npx = c if per_query else c - wg                      # the proxy's slots
    hi = t0 if per_query else t0 - W                      # the proxy scans [0, hi]
    gcand = np.asarray(gcand)
    swaps = 0
    if npx > 0:
        swaps += check_row(gcand[:npx], ocand[:npx], fbar, rtol, lambda idx: (idx >= 0) & (idx <= hi),
                           f"{label} proxy slots", swap_bound=sb)
    pool = set(gcand[:npx][gcand[:npx] >= 0].tolist())
    want = []
    for u in range(wg):
        p = t0 - W + 1 + u
        ok = 0 <= p <= t0 + gs - 1 and not (per_query and p in pool)
        want.append(p if ok else -1)
    if gcand[npx:npx + wg].tolist() != want:
        raise ParityError(f"{label}: window slots {gcand[npx:npx + wg].tolist()} != {want}")
    for t, r in enumerate(rows):
        tt = t0 + t
        use = [int(p) for i, p in enumerate(gcand)
               if 0 <= p <= tt and not (per_query and i >= npx and p < tt - W + 1)]
        C = np.array(use, dtype=np.int32)
        ref = oracle.refine_on(fmt, q[[r]], None if qs is None else qs[[r]], w[[r]], k, ks, C, topk)[0]
        swaps += check_row(gpu_idx[r], ref, member_scores(r), rtol, lambda idx, C=C: np.isin(idx, C),
                           f"{label} window refine row {r}", swap_bound=sb)
    return swaps
