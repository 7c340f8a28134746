"""Pins for the CPU oracle: checks against values fixed by the paper's
definitions and by mathematics, not against the oracle itself.

  * hand-derived worked examples (tests/golden/*.json, each citing its equation)
  * library routines for the number formats (torch's E4M3FN and bf16 casts)
  * closed forms (one head, one dimension: the top-k are the largest scalar keys)
  * identities stated by the paper or implied by Algorithm 1 (g = 1 is dense;
    c >= L with the guardrail is dense; Reuse shares one set per group;
    causality; identical members; Refine with a full candidate set)
  * invariances (positive scaling of gates / query scales, head permutation)
  * exact integer arithmetic for fp8 inner products
  * brute force on tiny inputs (Python sorting)
"""
import json
import math
import os

import numpy as np
import pytest
import torch

import oracle
from workload.gen import encode_bf16, make_prefill

GOLD = os.path.join(os.path.dirname(__file__), "golden")


def gold(name):
    with open(os.path.join(GOLD, name)) as f:
        return json.load(f)


def bf16_bits(x):
    return encode_bf16(np.asarray(x, dtype=np.float32))


@pytest.fixture(scope="module", autouse=True)
def _built(oracle_lib):
    return oracle_lib


# ------------------------------------------------------------------ codecs
def test_e4m3_decode_matches_torch_for_all_codes():
    codes = torch.arange(256, dtype=torch.int32).to(torch.uint8)
    ref = codes.view(torch.float8_e4m3fn).to(torch.float64).numpy()
    ours = np.array([oracle.e4m3_decode(c) for c in range(256)])
    nan = np.isnan(ref)
    assert list(np.nonzero(nan)[0]) == [0x7F, 0xFF]
    assert np.array_equal(np.isnan(ours), nan)
    assert np.array_equal(ours[~nan], ref[~nan])
    assert ours[0x7E] == 448.0 and ours[0x01] == 2.0 ** -9


def test_e4m3_encode_matches_torch_rne():
    vals = np.array([oracle.e4m3_decode(c) for c in range(0x7F)])       # non-negative finite
    mids = (vals[:-1] + vals[1:]) / 2                                     # exact ties
    rng = np.random.default_rng(7)
    rand = rng.uniform(-448, 448, 20000)
    small = rng.uniform(-0.05, 0.05, 20000)
    xs = np.concatenate([vals, -vals, mids, -mids, rand, small]).astype(np.float32)
    ref = torch.from_numpy(xs).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    ours = np.array([oracle.e4m3_encode(float(x)) for x in xs], dtype=np.uint8)
    # +-0: torch keeps the sign of zero, as the oracle does
    assert np.array_equal(ours, ref)


def test_e4m3_encode_saturates():
    assert oracle.e4m3_encode(449.0) == 0x7E
    assert oracle.e4m3_encode(1e30) == 0x7E
    assert oracle.e4m3_encode(-500.0) == 0xFE


def test_bf16_codec_matches_torch():
    rng = np.random.default_rng(3)
    xs = np.concatenate([rng.standard_normal(20000) * 10.0 ** rng.integers(-8, 8, 20000),
                         [0.0, -0.0, 1.0, 1.00390625, 1.01171875]]).astype(np.float32)
    ref = bf16_bits(xs)
    ours = np.array([oracle.bf16_encode(float(x)) for x in xs], dtype=np.uint16)
    assert np.array_equal(ours, ref)
    back = np.array([oracle.bf16_decode(int(b)) for b in ref])
    assert np.array_equal(back, torch.from_numpy(ref.view(np.int16)).view(torch.bfloat16).double().numpy())


# ------------------------------------------------------------------ golden
def test_golden_scores_bf16():
    G = gold("scores_bf16_h2_d3.json")
    k = bf16_bits(G["keys"])
    for case in G["queries"]:
        q = bf16_bits(case["q"])
        w = np.array(case["w"], dtype=np.float32)
        t = case["t"]
        f = oracle.scores("bf16", q, 1.0, w, k, None, t)
        assert list(f) == case["scores"], case["derivation"]
        for m, expect in case["topk"].items():
            qq = q[None]
            ww = w[None]
            out = oracle.index("bf16", qq, None, ww, t, k, None, len(G["keys"]),
                               mode=oracle.DENSE, topk=int(m))["idx"][0]
            assert list(out) == expect, (t, m)


def test_golden_scores_fp8_scaled():
    G = gold("scores_fp8_scaled.json")
    kc = np.array(G["key_codes"], dtype=np.uint8)
    for code, v in zip(kc.ravel(), np.array(G["key_values"]).ravel()):
        assert oracle.e4m3_decode(int(code)) == v
    ks = np.array(G["key_scale"], dtype=np.float32)
    for case in G["queries"]:
        qc = np.array(case["q_codes"], dtype=np.uint8)
        w = np.array(case["w"], dtype=np.float32)
        f = oracle.scores("fp8", qc, case["q_scale"], w, kc, ks, case["t"])
        assert list(f) == case["scores"], case["derivation"]
        for m, expect in case["topk"].items():
            out = oracle.index("fp8", qc[None], np.array([case["q_scale"]], np.float32), w[None],
                               case["t"], kc, ks, len(kc), mode=oracle.DENSE, topk=int(m))["idx"][0]
            assert list(out) == expect


def test_golden_proxy_fp8():
    G = gold("proxy_fp8_h1_d4.json")
    q = np.array([m["q_codes"] for m in G["members"]], dtype=np.uint8)
    for code, v in zip(q.ravel(), np.array([m["q_values"] for m in G["members"]]).ravel()):
        assert oracle.e4m3_decode(int(code)) == v
    qs = np.array([m["q_scale"] for m in G["members"]], dtype=np.float32)
    w = np.array([m["w"] for m in G["members"]], dtype=np.float32)
    pq, psc, pw = oracle.proxy("fp8", q, qs, w)
    assert pq.tolist() == G["proxy_codes"], G["derivation"]
    assert psc == G["proxy_scale"]
    assert pw.tolist() == G["proxy_w"]


def test_golden_proxy_bf16():
    G = gold("proxy_bf16_h1_d2.json")
    q = bf16_bits([m["q_values"] for m in G["members"]])
    w = np.array([m["w"] for m in G["members"]], dtype=np.float32)
    pq, psc, pw = oracle.proxy("bf16", q, None, w)
    assert pq.tolist() == bf16_bits(G["proxy_values"]).tolist(), G["derivation"]
    assert psc == 1.0 and pw.tolist() == G["proxy_w"]


def test_golden_group_reuse_refine():
    G = gold("group_reuse_refine_h1_d2.json")
    k = bf16_bits(G["keys"])
    q = bf16_bits([m["q"] for m in G["queries"]])
    w = np.array([m["w"] for m in G["queries"]], dtype=np.float32)
    p0, g, c, m = G["p0"], G["g"], G["c"], G["k"]
    n_k = len(G["keys"])
    r = oracle.index("bf16", q, None, w, p0, k, None, n_k, mode=oracle.REUSE, g=g, c=c, topk=m,
                     want_proxy=True)
    assert [sorted(x) for x in r["idx"].tolist()] == [sorted(x) for x in G["reuse"]]
    f = oracle.scores("bf16", r["pq"][0], 1.0, r["pw"][0], k, None, p0)
    assert list(f) == G["proxy_scores"], G["derivation"]
    r = oracle.index("bf16", q, None, w, p0, k, None, n_k, mode=oracle.REFINE, g=g, c=c, topk=m,
                     want_cand=True)
    assert sorted(r["cand"][0].tolist()) == sorted(G["refine_cand"])
    assert [sorted(x) for x in r["idx"].tolist()] == [sorted(x) for x in G["refine"]]
    r = oracle.index("bf16", q, None, w, p0, k, None, n_k, mode=oracle.DENSE, topk=m)
    assert [sorted(x) for x in r["idx"].tolist()] == [sorted(x) for x in G["dense"]]


# ------------------------------------------------------------------ closed form / brute force
@pytest.mark.parametrize("fmt", ["bf16", "fp8"])
def test_closed_form_one_head_one_dim(fmt):
    """H = d = 1, w > 0, q > 0: I(s) = w q ks k_s for k_s > 0 and 0 otherwise, so the
    top-k over [0, t] is the k largest scalar keys (ties: lower position)."""
    rng = np.random.default_rng(11)
    L, m = 200, 17
    kv = rng.choice([-2.0, -1.0, -0.5, 0.0, 0.25, 0.5, 1.0, 1.5, 2.0, 3.0], size=L)
    if fmt == "fp8":
        kc = np.array([oracle.e4m3_encode(x) for x in kv], np.uint8)[:, None]
        ks = rng.choice([0.5, 1.0, 2.0], size=L).astype(np.float32)
        qc = np.array([[[oracle.e4m3_encode(1.5)]]], np.uint8)
        qs = np.array([0.25], np.float32)
        key_val = np.array([oracle.e4m3_decode(int(c)) for c in kc[:, 0]]) * ks
    else:
        kc = bf16_bits(kv[:, None])
        ks, qs = None, None
        qc = bf16_bits([[[1.5]]])
        key_val = kv
    w = np.array([[0.75]], np.float32)
    for t in [0, 5, 16, 17, 120, L - 1]:
        out = oracle.index(fmt, qc, qs, w, t, kc, ks, L, mode=oracle.DENSE, topk=m)["idx"][0]
        vals = [max(0.0, key_val[s]) for s in range(t + 1)]
        order = sorted(range(t + 1), key=lambda s: (-vals[s], s))[:m]
        expect = order + [-1] * (m - len(order))
        assert out.tolist() == expect, t


def test_topk_bruteforce_with_ties():
    rng = np.random.default_rng(5)
    for trial in range(200):
        n = int(rng.integers(0, 60))
        f = rng.integers(-3, 4, size=n).astype(np.float64)
        f[rng.random(n) < 0.1] = -0.0
        pos = rng.permutation(1000)[:n].astype(np.int32)
        m = int(rng.integers(1, 70))
        out = oracle.topk(f, pos, m)
        order = sorted(range(n), key=lambda i: (-f[i], pos[i]))[:m]
        expect = [int(pos[i]) for i in order] + [-1] * max(0, m - n)
        assert out.tolist() == expect


def test_fp8_inner_products_are_exact():
    """Values of E4M3FN codes times 2^9 are integers, so with one head, unit gate
    and unit scales the score equals the integer dot product / 2^18 exactly."""
    rng = np.random.default_rng(2)
    d, L = 128, 64
    finite = [c for c in range(256) if c not in (0x7F, 0xFF)]
    ints = {c: int(round(oracle.e4m3_decode(c) * 512)) for c in finite}
    assert all(abs(oracle.e4m3_decode(c) * 512 - ints[c]) == 0 for c in finite)
    kc = rng.choice(finite, size=(L, d)).astype(np.uint8)
    qc = rng.choice(finite, size=(1, d)).astype(np.uint8)
    f = oracle.scores("fp8", qc, 1.0, np.ones(1, np.float32), kc, np.ones(L, np.float32), L - 1)
    for s in range(L):
        dot = sum(ints[int(a)] * ints[int(b)] for a, b in zip(qc[0], kc[s]))
        assert f[s] == max(0, dot) / 2.0 ** 18


# ------------------------------------------------------------------ identities of Algorithm 1
def small(fmt, L=96, seed=21, H=4, d=8, rho=0.95):
    return make_prefill(L, fmt, seed=seed, rho=rho, H=H, d=d, threads=1)


def run(x, mode, **kw):
    L = x.q.shape[0]
    p0 = kw.pop("p0", 0)
    n_q = kw.pop("n_q", L - p0)
    return oracle.index(x.dtype, x.q[p0:p0 + n_q], None if x.q_scale is None else x.q_scale[p0:p0 + n_q],
                        x.w[p0:p0 + n_q], p0, x.k, x.k_scale, L, mode=mode, **kw)


def as_sets(idx):
    return [frozenset(int(v) for v in row) for row in idx]


@pytest.mark.parametrize("fmt", ["bf16", "fp8"])
def test_group_of_one_is_dense(fmt):
    """App. A: a group size of one recovers the per-query indexer exactly."""
    x = small(fmt)
    dense = run(x, oracle.DENSE, topk=10)["idx"]
    for mode in (oracle.REUSE, oracle.REFINE):
        for db in (0, 16):
            r = run(x, mode, g=1, c=20, topk=10, dense_below=db)["idx"]
            assert np.array_equal(np.sort(r, 1), np.sort(dense, 1)), (mode, db)


@pytest.mark.parametrize("fmt", ["bf16", "fp8"])
def test_budget_covering_the_sequence_is_dense(fmt):
    """c >= L: every group starts before c, so Algorithm 1's guardrail sends
    all of them to the dense path."""
    x = small(fmt, L=64)
    dense = run(x, oracle.DENSE, topk=8)["idx"]
    for mode in (oracle.REUSE, oracle.REFINE):
        r = run(x, mode, g=4, c=64, topk=8)["idx"]
        assert np.array_equal(r, dense)


@pytest.mark.parametrize("fmt", ["bf16", "fp8"])
@pytest.mark.parametrize("g", [2, 3, 4])
def test_reuse_shares_one_set_and_is_causal(fmt, g):
    x = small(fmt, L=90)
    c, m = 24, 8
    r = run(x, oracle.REUSE, g=g, c=c, topk=m)["idx"]
    L = x.q.shape[0]
    for start in range(0, L, g):
        rows = r[start:min(start + g, L)]
        if start >= c:                                  # proxy group
            assert all(np.array_equal(rows[0], row) for row in rows)
            assert rows.max() <= start                  # Eq. 5 cutoff at t0
        for i, row in enumerate(rows):
            valid = row[row >= 0]
            assert valid.max() <= start + i and len(set(valid)) == len(valid)


@pytest.mark.parametrize("fmt", ["bf16", "fp8"])
@pytest.mark.parametrize("g", [2, 4])
def test_refine_with_full_candidates_is_truncated_dense(fmt, g):
    """Guardrail off and c > t0: C is the whole prefix [0, t0], so each member's
    set is the top-k of its own scores over [0, t0] (brute-force sort)."""
    x = small(fmt, L=40)
    m = 6
    r = run(x, oracle.REFINE, g=g, c=64, topk=m, dense_below=0)["idx"]
    for t in range(40):
        t0 = (t // g) * g
        f = oracle.scores(x.dtype, x.q[t], 1.0 if x.q_scale is None else x.q_scale[t], x.w[t],
                          x.k, x.k_scale, t0)
        order = sorted(range(t0 + 1), key=lambda s: (-f[s], s))[:m]
        assert sorted(r[t][r[t] >= 0].tolist()) == sorted(order), t


@pytest.mark.parametrize("fmt", ["bf16", "fp8"])
def test_identical_members_proxy_is_the_member(fmt):
    """Equal members (g a power of two): the mean equals the member, so Reuse,
    Refine and the dense set truncated at t0 coincide."""
    x = small(fmt, L=48)
    g = 4
    for a in (x.q, x.w) + ((x.q_scale,) if x.q_scale is not None else ()):
        for t in range(48):
            a[t] = a[(t // g) * g]
    m = 6
    reuse = run(x, oracle.REUSE, g=g, c=64, topk=m, dense_below=0, want_proxy=True)
    refine = run(x, oracle.REFINE, g=g, c=64, topk=m, dense_below=0)["idx"]
    for t in range(48):
        t0 = (t // g) * g
        if x.dtype == "bf16":
            assert np.array_equal(reuse["pq"][t // g], x.q[t0])
        f = oracle.scores(x.dtype, x.q[t0], 1.0 if x.q_scale is None else x.q_scale[t0], x.w[t0],
                          x.k, x.k_scale, t0)
        order = sorted(range(t0 + 1), key=lambda s: (-f[s], s))[:m]
        order += [-1] * (m - len(order))
        assert sorted(reuse["idx"][t].tolist()) == sorted(order)
        assert sorted(refine[t].tolist()) == sorted(order)


def test_fp8_proxy_requantisation_matches_torch_cast():
    """The fp8 proxy: fp32 mean of the dequantised members, scale amax/448,
    codes by RNE; the codes must equal torch's cast of the same fp32 values."""
    x = small("fp8", L=16, H=4, d=8)
    for g in (2, 3, 4):
        q, qs, w = x.q[:g], x.q_scale[:g], x.w[:g]
        pq, psc, pw = oracle.proxy("fp8", q, qs, w)
        deq = torch.from_numpy(q).view(torch.float8_e4m3fn).float() * torch.from_numpy(qs)[:, None, None]
        acc = deq[0].clone()
        for i in range(1, g):
            acc = acc + deq[i]
        mean = acc / float(g)
        sigma = (mean.abs().max() / 448.0).item()
        assert psc == np.float32(sigma)
        ref = (mean / torch.tensor(sigma, dtype=torch.float32)).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
        assert np.array_equal(pq, ref)
        wr = torch.from_numpy(w[0]).clone()
        for i in range(1, g):
            wr = wr + torch.from_numpy(w[i])
        assert np.array_equal(pw, (wr / float(g)).numpy())


@pytest.mark.parametrize("fmt", ["bf16", "fp8"])
def test_positive_scalings_and_head_permutation(fmt):
    x = small(fmt, L=64)
    m = 9
    base = run(x, oracle.DENSE, topk=m)["idx"]
    y = small(fmt, L=64)
    y.w *= np.float32(4.0)
    assert np.array_equal(run(y, oracle.DENSE, topk=m)["idx"], base)
    if fmt == "fp8":
        y = small(fmt, L=64)
        y.q_scale *= np.float32(0.5)
        assert np.array_equal(run(y, oracle.DENSE, topk=m)["idx"], base)
    perm = np.random.default_rng(0).permutation(x.q.shape[1])
    for t in (0, 31, 63):
        f0 = oracle.scores(fmt, x.q[t], 1.0 if x.q_scale is None else x.q_scale[t], x.w[t], x.k, x.k_scale, t)
        f1 = oracle.scores(fmt, x.q[t][perm], 1.0 if x.q_scale is None else x.q_scale[t], x.w[t][perm],
                           x.k, x.k_scale, t)
        assert np.allclose(f0, f1, rtol=1e-12, atol=0)


def test_negating_gates_reverses_order_of_active_keys():
    """One head: negating the gate negates every score, so the dense top-k over
    keys with a positive dot becomes the bottom of the order."""
    x = small("bf16", L=50, H=1, d=8)
    t = 49
    f = oracle.scores("bf16", x.q[t], 1.0, x.w[t], x.k, None, t)
    g = oracle.scores("bf16", x.q[t], 1.0, -x.w[t], x.k, None, t)
    assert np.array_equal(g, -f)


def test_group_count_and_ragged_tail():
    """Eq. 2: groups are runs of g from the call's first query; a short last
    group of one row is its own proxy, which gives the dense set truncated at
    its own position, i.e. the dense set."""
    x = small("fp8", L=45)
    dense = run(x, oracle.DENSE, topk=5)["idx"]
    r = run(x, oracle.REUSE, g=4, c=8, topk=5)["idx"]        # 45 = 11*4 + 1
    assert sorted(r[44].tolist()) == sorted(dense[44].tolist())
    chunked = np.concatenate([run(x, oracle.REUSE, g=4, c=8, topk=5, p0=p, n_q=min(16, 45 - p))["idx"]
                              for p in range(0, 45, 16)])
    assert np.array_equal(chunked, r)                         # chunks of a multiple of g


# ------------------------------------------------ App. B window, aggregation
def _topk_brute(f, pos, m):
    order = sorted(range(len(pos)), key=lambda i: (-f[i], pos[i]))[:m]
    return sorted(int(pos[i]) for i in order)


def _scores(x, t, pos):
    return oracle.scores_at(x.dtype, x.q[t], 1.0 if x.q_scale is None else x.q_scale[t], x.w[t], x.k, x.k_scale,
                            np.asarray(pos, dtype=np.int32))


@pytest.mark.parametrize("fmt", ["bf16", "fp8"])
@pytest.mark.parametrize("W", [1, 3, 6])
def test_prefill_window_with_full_budget_is_dense(fmt, W):
    """App. B: with the window, a candidate budget that covers the sequence
    makes Refine equal dense for every member, guardrail off (without the
    window the later members of a group could not reach (t0, t])."""
    x = small(fmt, L=48)
    g, m = 4, 6
    dense = run(x, oracle.DENSE, topk=m)["idx"]
    r = run(x, oracle.REFINE, g=g, c=48 + g, topk=m, dense_below=0, window=W)["idx"]
    assert np.array_equal(np.sort(r, 1), np.sort(dense, 1))
    plain = run(x, oracle.REFINE, g=g, c=48 + g, topk=m, dense_below=0)["idx"]
    assert not np.array_equal(np.sort(plain, 1), np.sort(dense, 1))


@pytest.mark.parametrize("fmt", ["bf16", "fp8"])
@pytest.mark.parametrize("W,g", [(2, 4), (4, 4), (5, 2), (4, 3)])
def test_prefill_window_brute_force(fmt, W, g):
    """App. B prefill, restated in Python: C = (proxy top-(c - w_g) over
    [0, t0 - W]) followed by the window union t0-W+1 .. t0+g-1 (w_g = W+g-1
    slots, -1 where no member reaches); member t re-scores C within [0, t]."""
    x = small(fmt, L=70)
    c, m = 20, 5
    res = run(x, oracle.REFINE, g=g, c=c, topk=m, dense_below=0, window=W, want_cand=True, want_proxy=True)
    wg = W + g - 1
    L = 70
    for j in range((L + g - 1) // g):
        t0, gs = j * g, min(g, L - j * g)
        fp = oracle.scores_at(x.dtype, res["pq"][j], res["psc"][j], res["pw"][j], x.k, x.k_scale,
                              np.arange(max(0, t0 - W + 1), dtype=np.int32))
        proxy = _topk_brute(fp, list(range(max(0, t0 - W + 1))), c - wg)
        proxy = proxy if len(proxy) == c - wg else proxy + [-1] * (c - wg - len(proxy))
        union = [p if 0 <= p <= t0 + gs - 1 else -1 for p in range(t0 - W + 1, t0 - W + 1 + wg)]
        cand = res["cand"][j]
        assert sorted(cand[:c - wg].tolist()) == sorted(proxy), j
        assert cand[c - wg:].tolist() == union, j
        for t in range(t0, t0 + gs):
            use = [int(p) for p in cand if 0 <= p <= t]
            exp = _topk_brute(_scores(x, t, use), use, m)
            got = sorted(v for v in res["idx"][t].tolist() if v >= 0)
            assert got == exp, (j, t)
            assert set(range(max(0, t - W + 1), t + 1)) <= set(use)   # its own window is in reach


@pytest.mark.parametrize("fmt", ["bf16", "fp8"])
@pytest.mark.parametrize("W,g", [(2, 2), (4, 2), (5, 3)])
def test_decode_window_brute_force(fmt, W, g):
    """App. B decode: the pool is the proxy top-c over [0, t0]; each query adds
    its own window [t-W+1, t] (duplicates removed); W >= g."""
    x = small(fmt, L=60)
    c, m = 12, 5
    p0 = 60 - g
    res = run(x, oracle.REFINE, g=g, c=c, topk=m, dense_below=0, window=W, window_kind=oracle.WINDOW_PER_QUERY,
              want_cand=True, want_proxy=True, p0=p0, n_q=g)
    cand = res["cand"][0]
    assert len(cand) == c + W + g - 1
    fp = oracle.scores_at(x.dtype, res["pq"][0], res["psc"][0], res["pw"][0], x.k, x.k_scale,
                          np.arange(p0 + 1, dtype=np.int32))
    pool = _topk_brute(fp, list(range(p0 + 1)), c)
    assert sorted(cand[:c].tolist()) == pool
    valid = cand[cand >= 0]
    assert len(set(valid.tolist())) == len(valid)                     # no position twice
    for i in range(g):
        t = p0 + i
        use = sorted(set(pool) | set(range(max(0, t - W + 1), t + 1)))
        exp = _topk_brute(_scores(x, t, use), use, m)
        assert sorted(v for v in res["idx"][i].tolist() if v >= 0) == exp, t


@pytest.mark.parametrize("fmt", ["bf16", "fp8"])
def test_window_zero_is_the_plain_candidate_set(fmt):
    x = small(fmt, L=64)
    for kind in (oracle.WINDOW_SHARED, oracle.WINDOW_PER_QUERY):
        a = run(x, oracle.REFINE, g=4, c=20, topk=6, window=0, window_kind=kind, want_cand=True)
        b = run(x, oracle.REFINE, g=4, c=20, topk=6, want_cand=True)
        assert np.array_equal(a["idx"], b["idx"]) and np.array_equal(a["cand"], b["cand"])


def test_window_argument_checks():
    x = small("fp8", L=32)
    with pytest.raises(ValueError):                    # Reuse has no refine step
        run(x, oracle.REUSE, g=4, c=16, topk=4, window=2)
    with pytest.raises(ValueError):                    # decode needs W >= g
        run(x, oracle.REFINE, g=4, c=16, topk=4, window=3, window_kind=oracle.WINDOW_PER_QUERY)
    with pytest.raises(ValueError):                    # prefill needs c >= W + g - 1
        run(x, oracle.REFINE, g=4, c=6, topk=4, window=4)


@pytest.mark.parametrize("fmt", ["bf16", "fp8"])
def test_first_and_last_member_aggregation(fmt):
    """The endpoint proxies of the aggregation ablation (Sec. 5.4): the proxy is
    that member's row unchanged, so Reuse hands every member the top-k of the
    first (last) member's own scores over [0, t0]."""
    x = small(fmt, L=50)
    g, m = 4, 5
    for agg, pick in ((oracle.AGG_FIRST, lambda t0, gs: t0), (oracle.AGG_LAST, lambda t0, gs: t0 + gs - 1)):
        res = run(x, oracle.REUSE, g=g, c=8, topk=m, dense_below=0, agg=agg, want_proxy=True)
        for j in range((50 + g - 1) // g):
            t0, gs = j * g, min(g, 50 - j * g)
            src = pick(t0, gs)
            assert np.array_equal(res["pq"][j], x.q[src]) and np.array_equal(res["pw"][j], x.w[src])
            exp = _topk_brute(_scores(x, src, list(range(t0 + 1))), list(range(t0 + 1)), m)
            for t in range(t0, t0 + gs):
                assert sorted(v for v in res["idx"][t].tolist() if v >= 0) == exp, (agg, t)


def _decode_case(fmt, g, W, copies):
    """A decode sequence of 60 keys whose key rows at the given positions are
    replaced by copies of chosen rows (so their scores tie with those rows)."""
    x = small(fmt, L=60)
    p0 = 60 - g
    pre = run(x, oracle.REFINE, g=g, c=4, topk=2, dense_below=0, want_proxy=True, p0=p0, n_q=g)
    fp = oracle.scores_at(x.dtype, pre["pq"][0], pre["psc"][0], pre["pw"][0], x.k, x.k_scale,
                          np.arange(p0 + 1, dtype=np.int32))
    order = [int(s) for s in np.argsort(-fp, kind="stable")]
    for dst, rank in copies:
        x.k[dst] = x.k[order[rank]]
        if x.k_scale is not None:
            x.k_scale[dst] = x.k_scale[order[rank]]
    return x, p0


@pytest.mark.parametrize("fmt", ["bf16", "fp8"])
def test_decode_window_removes_pool_duplicates(fmt):
    """The window's positions up to t0 carry the proxy's best key, so the pool
    holds them; the window part must not list them again."""
    g, W, c, m = 2, 4, 12, 6
    p0 = 60 - g
    x, p0 = _decode_case(fmt, g, W, [(p, 0) for p in range(p0 - W + 1, p0 + 1)])
    res = run(x, oracle.REFINE, g=g, c=c, topk=m, dense_below=0, window=W, window_kind=oracle.WINDOW_PER_QUERY,
              want_cand=True, p0=p0, n_q=g)
    cand = res["cand"][0]
    assert set(range(p0 - W + 1, p0 + 1)) <= set(cand[:c].tolist())      # the pool holds them
    valid = cand[cand >= 0]
    assert len(set(valid.tolist())) == len(valid)
    for i in range(g):
        row = res["idx"][i][res["idx"][i] >= 0]
        assert len(set(row.tolist())) == len(row)


@pytest.mark.parametrize("fmt", ["bf16", "fp8"])
def test_decode_window_is_per_query(fmt):
    """Two early positions carry the proxy's best key (the pool, c = 2); every
    window position carries its second best.  The last query may not use the
    union positions older than its own window, which would otherwise win the
    ties by lower position."""
    g, W, c, m = 3, 4, 2, 5
    p0 = 60 - g
    union = list(range(p0 - W + 1, p0 + g))
    x, p0 = _decode_case(fmt, g, W, [(5, 0), (6, 0)] + [(p, 1) for p in union])
    res = run(x, oracle.REFINE, g=g, c=c, topk=m, dense_below=0, window=W, window_kind=oracle.WINDOW_PER_QUERY,
              want_cand=True, p0=p0, n_q=g)
    pool = sorted(res["cand"][0][:c].tolist())
    assert pool == [5, 6]
    t = p0 + g - 1
    use = sorted(set(pool) | set(range(t - W + 1, t + 1)))
    exp = _topk_brute(_scores(x, g - 1 + p0, use), use, m)
    got = sorted(v for v in res["idx"][g - 1].tolist() if v >= 0)
    assert got == exp
    assert not set(got) & set(range(p0 - W + 1, t - W + 1))


# ------------------------------------------------ IndexCache composition (Sec. 5.1, Table 1 +IC)
def _layers(fmt, n_layers, L=64):
    """Distinct inputs per layer (the same positions, another seed each)."""
    xs = [small(fmt, L=L, seed=300 + l) for l in range(n_layers)]
    return xs, [(x.q, x.q_scale, x.w, x.k, x.k_scale) for x in xs]


def _own(x, mode, **kw):
    """The layer's own indexer result (Algorithm 1, pinned above)."""
    return run(x, mode, **kw)["idx"]


IC_KW = dict(g=4, c=12, topk=6)


@pytest.mark.parametrize("fmt", ["bf16", "fp8"])
@pytest.mark.parametrize("mode", [oracle.REUSE, oracle.REFINE, oracle.DENSE])
def test_indexcache_stride_one_is_per_layer(fmt, mode):
    """Every layer an anchor: each layer is indexed on its own inputs."""
    xs, layers = _layers(fmt, 3)
    kw = dict(IC_KW) if mode != oracle.DENSE else dict(topk=6)
    got = oracle.index_layers(fmt, layers, 0, 64, mode=mode, stride=1, **kw)
    for l, x in enumerate(xs):
        assert np.array_equal(got[l], _own(x, mode, **kw)), l


@pytest.mark.parametrize("fmt", ["bf16", "fp8"])
@pytest.mark.parametrize("stride", [2, 3])
def test_indexcache_followers_take_the_anchor_before_them(fmt, stride):
    """Stride r: layers l .. l+r-1 of a block all hold the anchor l's sets,
    which differ from what the followers' own inputs would give."""
    n_layers = 5
    xs, layers = _layers(fmt, n_layers)
    own = [_own(x, oracle.REFINE, **IC_KW) for x in xs]
    got = oracle.index_layers(fmt, layers, 0, 64, mode=oracle.REFINE, stride=stride, **IC_KW)
    differs = 0
    for l in range(n_layers):
        a = l - l % stride
        assert np.array_equal(got[l], own[a]), (l, a)
        differs += not np.array_equal(own[l], own[a])
    assert differs >= 1  # the inputs tell anchors and followers apart


@pytest.mark.parametrize("fmt", ["bf16", "fp8"])
def test_indexcache_explicit_anchor_pattern(fmt):
    """An irregular pattern: each follower takes the NEAREST anchor before it
    (not the first layer, not the next anchor)."""
    anchors = [1, 0, 0, 1, 0, 1]
    xs, layers = _layers(fmt, len(anchors))
    own = [_own(x, oracle.REUSE, **IC_KW) for x in xs]
    for l, a in enumerate(anchors):  # the followers' inputs are never read
        if not a:
            layers[l] = None
    got = oracle.index_layers(fmt, layers, 0, 64, mode=oracle.REUSE, anchors=anchors, **IC_KW)
    src = [0, 0, 0, 3, 3, 5]
    for l in range(len(anchors)):
        assert np.array_equal(got[l], own[src[l]]), l
    assert not np.array_equal(own[4], own[3]) or not np.array_equal(own[4], own[0])


def test_indexcache_stride_past_the_layers_and_identical_layers():
    """A stride beyond the layer count shares layer 0's sets everywhere; layers
    with identical inputs give the per-layer result for any stride."""
    xs, layers = _layers("fp8", 4)
    own0 = _own(xs[0], oracle.REFINE, **IC_KW)
    for out in oracle.index_layers("fp8", layers, 0, 64, mode=oracle.REFINE, stride=10, **IC_KW):
        assert np.array_equal(out, own0)
    same = [layers[0]] * 4
    for stride in (1, 2, 3):
        for out in oracle.index_layers("fp8", same, 0, 64, mode=oracle.REFINE, stride=stride, **IC_KW):
            assert np.array_equal(out, own0)


def test_indexcache_chunk_offset_and_guardrail():
    """A later chunk (queries 32 .. 63 against keys 0 .. 63) with the guardrail
    at c: the layer function passes the call's positions through."""
    xs, _ = _layers("fp8", 3)
    p0 = 32
    layers = [(x.q[p0:], x.q_scale[p0:], x.w[p0:], x.k, x.k_scale) for x in xs]
    got = oracle.index_layers("fp8", layers, p0, 64, mode=oracle.REFINE, stride=2, g=4, c=40, topk=6)
    for l in range(3):
        a = l - l % 2
        assert np.array_equal(got[l], _own(xs[a], oracle.REFINE, p0=p0, g=4, c=40, topk=6)), l


def test_indexcache_first_layer_must_be_an_anchor():
    _, layers = _layers("bf16", 2)
    with pytest.raises(ValueError):
        oracle.index_layers("bf16", layers, 0, 64, mode=oracle.REUSE, anchors=[0, 1], **IC_KW)
