"""The GPU parity rule itself, on the CPU: the oracle's own Refine results
with App. B's window pass check_pivot, and planted mistakes in a candidate row
or a member's set are caught."""
import numpy as np
import pytest

import oracle
from parity import ParityError, check_pivot
from workload.gen import make_prefill

H, D = 8, 16


@pytest.fixture(scope="module")
def x():
    return make_prefill(160, "fp8", seed=91, H=H, d=D, threads=2)


def _run(x, W, kind, p0=0, g=4, c=24, m=8, db=0):
    n_q = x.q.shape[0] - p0
    q, qs, w = x.q[p0:], x.q_scale[p0:], x.w[p0:]
    n_k = x.q.shape[0]
    res = oracle.index("fp8", q, qs, w, p0, x.k, x.k_scale, n_k, mode=oracle.REFINE, g=g, c=c, topk=m,
                       dense_below=db, want_cand=True, window=W, window_kind=kind)
    return res, (q, qs, w, n_k, g, c, m, db)


def _check(x, res, shape, W, kind, idx=None, cand=None):
    q, qs, w, n_k, g, c, m, db = shape
    return check_pivot("fp8", q, qs, w, 0, x.k, x.k_scale, n_k, mode=oracle.REFINE, g=g, c=c, topk=m,
                       dense_below=db, gpu_idx=res["idx"] if idx is None else idx,
                       gpu_cand=res["cand"] if cand is None else cand, window=W, window_kind=kind)


@pytest.mark.parametrize("W,kind", [(6, oracle.WINDOW_SHARED), (5, oracle.WINDOW_PER_QUERY)])
def test_oracle_passes_its_own_rule(x, W, kind):
    res, shape = _run(x, W, kind)
    assert _check(x, res, shape, W, kind) == 0


def test_wrong_union_slot_is_caught(x):
    W, kind = 5, oracle.WINDOW_PER_QUERY
    res, shape = _run(x, W, kind)
    cand = res["cand"].copy()
    j = 20
    union = cand[j, 24:]
    u = int(np.flatnonzero(union >= 0)[0])
    cand[j, 24 + u] = -1                      # a window position dropped
    with pytest.raises(ParityError, match="window slots"):
        _check(x, res, shape, W, kind, cand=cand)


def test_member_outside_its_window_is_caught(x):
    """Member 0 of a per-query group may not use the last member's position."""
    W, kind = 5, oracle.WINDOW_PER_QUERY
    res, shape = _run(x, W, kind, m=24)
    j, g = 20, 4
    t0 = j * g
    idx = res["idx"].copy()
    row = idx[j * g]
    assert (row == t0 + g - 1).sum() == 0
    row[np.flatnonzero(row >= 0)[0]] = t0 + g - 1
    with pytest.raises(ParityError):
        _check(x, res, shape, W, kind, idx=idx)


def test_shared_proxy_slot_past_its_range_is_caught(x):
    """The shared window's proxy slots hold positions <= t0 - W only."""
    W, kind = 6, oracle.WINDOW_SHARED
    res, shape = _run(x, W, kind)
    cand = res["cand"].copy()
    j, g, c = 30, 4, 24
    t0 = j * g
    proxy = cand[j, :c - (W + g - 1)]
    proxy[np.argmin(proxy)] = t0 - W + 1       # a union position in a proxy slot
    with pytest.raises(ParityError):
        _check(x, res, shape, W, kind, cand=cand)


def test_budget_records_swaps_against_the_error_model():
    """A boundary swap inside rtol is accepted; the budget records its distance
    from tau relative to the path's error model, so one beyond the model (but
    inside rtol) is visible and a full-size test can reject it."""
    import parity
    f = {0: 10.0, 1: 9.0, 2: 8.0, 3: 7.97, 4: 7.9}  # oracle top-3 = {0, 1, 2}, tau = 8.0
    f_of = lambda idx: np.array([f[int(i)] for i in idx], dtype=np.float64)  # noqa: E731
    dom = lambda idx: np.ones(len(idx), bool)  # noqa: E731
    ora = np.array([0, 1, 2])
    bound = parity.SWAP_BOUND["fp8"]
    parity.BUDGET = parity.Budget()
    assert parity.check_row(np.array([0, 1, 2]), ora, f_of, 2e-2, dom, swap_bound=bound) == 0
    assert parity.check_row(np.array([0, 1, 3]), ora, f_of, 2e-2, dom, swap_bound=bound) == 1   # 0.375% below tau
    assert parity.BUDGET.rows == 2 and parity.BUDGET.rows_diff == 1
    assert abs(parity.BUDGET.max_rel - 0.03 / 8.0) < 1e-12 and parity.BUDGET.worst <= 1.0
    assert parity.check_row(np.array([0, 1, 4]), ora, f_of, 2e-2, dom, swap_bound=bound) == 1   # 1.25%: inside rtol
    assert parity.BUDGET.worst > 1.0
    with pytest.raises(ParityError):
        parity.check_row(np.array([0, 1, 4]), ora, f_of, 1e-2, dom)                             # outside rtol
