"""Per-kernel GPU tests through the C ABI stage entry points."""
import zlib

import numpy as np
import pytest
import torch

import oracle
import paper_2607_24593_amd as pv
from gpu_util import dev, host, say
from workload.gen import encode_bf16, make_prefill

pytestmark = pytest.mark.gpu


def test_encode_e4m3_matches_oracle_rne():
    vals = np.array([oracle.e4m3_decode(c) for c in range(0x7F)])
    mids = (vals[:-1] + vals[1:]) / 2
    rng = np.random.default_rng(1)
    x = np.concatenate([vals, -vals, mids, -mids, rng.uniform(-448, 448, 50000),
                        rng.normal(0, 0.01, 50000), [0.0, -0.0]]).astype(np.float32)
    say("encode_e4m3", x.size)
    got = host(pv.pivot_encode_e4m3(dev(x)))
    ref = np.array([oracle.e4m3_encode(float(v)) for v in x], dtype=np.uint8)
    bad = np.nonzero(got != ref)[0]
    assert bad.size == 0, [(float(x[i]), int(got[i]), int(ref[i])) for i in bad[:8]]


@pytest.mark.parametrize("fmt", ["fp8", "bf16"])
@pytest.mark.parametrize("g", [1, 2, 3, 4, 5, 8, 9, 16, 37])
def test_proxy_rows_bit_exact(fmt, g):
    """Proxies of 37 rows in groups of g (ragged last group), bit for bit; the
    kernel reads members in batches of 8 (fp8) or 4 (bf16), so g = 5, 9, 16
    and 37 span several batches, some partial."""
    x = make_prefill(37, fmt, seed=100 + g, threads=1)
    say("proxy_rows", fmt, "g", g)
    pq, ps, pw = pv.pivot_proxy_rows(dev(x.q), dev(x.q_scale), dev(x.w), g)
    pq, ps, pw = host(pq), host(ps), host(pw)
    if fmt == "bf16":
        pq = pq.view(np.uint16)
    for j in range((37 + g - 1) // g):
        rows = slice(j * g, min(37, (j + 1) * g))
        oq, osc, ow = oracle.proxy(fmt, x.q[rows], None if x.q_scale is None else x.q_scale[rows], x.w[rows])
        assert np.array_equal(pq[j], oq), (j, np.nonzero(pq[j] != oq))
        assert ps[j] == np.float32(osc), j
        assert np.array_equal(pw[j], ow), j


@pytest.mark.parametrize("g", [2, 4])
def test_proxy_codes_at_ties_and_near_zero(g):
    """fp8 proxies whose mean / scale lands exactly on E4M3 midpoints (RNE
    ties), on values of either sign below the smallest subnormal, and on exact
    zeros.  The members of a group alternate between adjacent codes a and b of
    one sign, all with the scale 3/16; element 0 is 448 in every member, so the
    proxy's scale is 3/16 again and every quotient is (a + b) / 2 exactly.
    Group 1 spans 2^-11 .. 2^-8 of 448 sigma, where the quotient sits near the
    subnormal and zero boundaries."""
    rng = np.random.default_rng(11)
    H, d = 64, 128
    n_groups = 2
    q = np.zeros((n_groups * g, H, d), dtype=np.uint8)
    sc = np.float32(0.1875)
    for j in range(n_groups):
        lo = rng.integers(0, 0x7D, size=(H, d)) if j == 0 else rng.integers(0, 8, size=(H, d))
        sign = (rng.integers(0, 2, size=(H, d)) * 0x80).astype(np.uint8)
        a = (lo | sign).astype(np.uint8)
        b = ((lo + 1) | sign).astype(np.uint8)
        if j == 1:  # opposite signs cancel to zero
            b[::7] = a[::7] ^ 0x80
        for u in range(g):
            q[j * g + u] = a if u % 2 == 0 else b
            q[j * g + u, 0, 0] = 0x7E  # 448
    q_scale = np.full(n_groups * g, sc, dtype=np.float32)
    w = rng.standard_normal((n_groups * g, H)).astype(np.float32)
    say("proxy ties", g)
    pq, ps, pw = pv.pivot_proxy_rows(dev(q), dev(q_scale), dev(w), g)
    pq, ps = host(pq), host(ps)
    for j in range(n_groups):
        oq, osc, _ = oracle.proxy("fp8", q[j * g:(j + 1) * g], q_scale[j * g:(j + 1) * g], w[j * g:(j + 1) * g])
        assert osc == sc, osc
        assert np.array_equal(pq[j], oq), (j, np.count_nonzero(pq[j] != oq))
        assert ps[j] == np.float32(osc), j


@pytest.mark.parametrize("fmt", ["fp8", "bf16"])
@pytest.mark.parametrize("n_rows,lim0,step", [(1, 5000, 0), (2, 4999, 1), (3, 700, 7), (5, 33, 2),
                                              (16, 4100, 1), (40, 8300, 3), (64, 0, 130)])
def test_score_rows_match_oracle(fmt, n_rows, lim0, step):
    lim_max = lim0 + (n_rows - 1) * step
    L = lim_max + 1
    x = make_prefill(max(L, n_rows), fmt, seed=7, threads=4)
    q, qs, w = x.q[:n_rows], None if x.q_scale is None else x.q_scale[:n_rows], x.w[:n_rows]
    ld = lim_max + 1 + 13
    say("score_rows", fmt, n_rows, lim0, step)
    got = host(pv.pivot_score_rows(dev(q), dev(qs), dev(w), dev(x.k), dev(x.k_scale), lim0, step, ld=ld))
    # bf16: fp32 MFMA sums of exact bf16 products, so every element is within
    # a few fp32 ulps of the row's largest |score| (1e-5 of it); fp8 adds the
    # four-level linear term of the epilogue, whose residual is below 2^-16 of
    # max|u| per level chain, bounded here by 1e-4 of the row's largest |score|
    tol = 1e-5 if fmt == "bf16" else 1e-4
    for r in range(n_rows):
        lim = lim0 + r * step
        f = oracle.scores(fmt, q[r], 1.0 if qs is None else qs[r], w[r], x.k, x.k_scale, lim)
        scale = np.abs(f).max() + 1e-30
        err = np.abs(got[r, :lim + 1] - f) / scale
        assert err.max() < tol, (r, int(err.argmax()), float(err.max()))
        assert np.isnan(got[r, lim + 1:]).all(), r   # nothing written past the row's limit


def _expect_topk(row, n, m):
    return oracle.topk(row[:n].astype(np.float64), np.arange(n, dtype=np.int32), m)


@pytest.mark.parametrize("split", [False, True, "bf16"])
@pytest.mark.parametrize("case", ["normal", "ties", "signed_zeros", "short", "exact", "long2k", "long4k",
                                  "ragged", "constant", "sample_miss", "sample_ragged", "heavy_tail", "small_m",
                                  "unaligned", "m4k_normal", "slice_skew", "decode_shape", "many_rows",
                                  "wave_skew"])
def test_topk_rows_exact(case, split):
    """Rows of 16384+ scores with m <= 2048 take the sampled one-pass path; the
    sample_miss rows put the sample's largest keys where the rest of the row is
    low, so the pass finds fewer than m keys and falls back to two passes.
    split: with a workspace, calls of at most 256 rows split each long row over
    several workgroups; slice_skew puts every high score in the first slice,
    which overflows its share of the scratch and falls back.  Calls of more
    than 256 rows take one 512-thread workgroup per row, whose waves compact
    into segments of their own: wave_skew puts every high score in the columns
    wave 0 reads (elements e with e mod 2048 < 256), which overflows its
    segment and falls back."""
    rng = np.random.default_rng(zlib.crc32(case.encode()))
    n0, step, m = 5000, 0, 100
    if case == "normal":
        rows = rng.standard_normal((6, 5000))
    elif case == "ties":
        rows = rng.integers(0, 10, (6, 5000)).astype(np.float64)
    elif case == "signed_zeros":
        rows = rng.choice([-0.0, 0.0, 1.0, -1.0, 2.0], size=(3, 40000)); n0 = 40000
    elif case == "short":
        rows = rng.standard_normal((4, 64)); n0, m = 50, 100
    elif case == "exact":
        rows = rng.standard_normal((3, 100)); n0, m = 100, 100
    elif case == "long2k":
        rows = rng.standard_normal((2, 262144)); n0, m = 262144, 2048
    elif case == "long4k":
        rows = np.exp(rng.standard_normal((2, 131072)) * 3); n0, m = 131072, 4096
    elif case == "ragged":
        rows = rng.standard_normal((40, 3000)); n0, step, m = 17, 70, 64
    elif case == "sample_miss":
        rows = rng.standard_normal((2, 65536)) * 0.1
        sampled = (np.arange(65536) // 64) % 16 == 0        # every 16th 256-byte chunk
        rows[:, sampled] += 5.0; n0, m = 65536, 2048
    elif case == "sample_ragged":
        rows = rng.standard_normal((6, 70000)); n0, step, m = 16384, 10001, 2048
    elif case == "heavy_tail":
        rows = np.exp(rng.standard_normal((3, 131072)) * 3); n0, m = 131072, 2048
    elif case == "small_m":
        rows = rng.standard_normal((3, 100000)); n0, m = 100000, 16
    elif case == "unaligned":
        rows = rng.standard_normal((4, 40001)); n0, step, m = 39990, 3, 1000
    elif case == "m4k_normal":
        rows = rng.standard_normal((3, 70000)); n0, m = 70000, 4096
    elif case == "slice_skew":
        rows = rng.standard_normal((2, 131072)) * 0.1
        rows[:, :4096] += 5.0; n0, m = 131072, 2048
    elif case == "decode_shape":
        rows = rng.standard_normal((32, 131071)); n0, m = 131071, 4096
    elif case == "many_rows":
        rows = rng.standard_normal((300, 20000)); n0, step, m = 16384, 12, 2048
    elif case == "wave_skew":
        rows = rng.standard_normal((300, 32768)) * 0.1
        rows[:, np.arange(32768) % 2048 < 256] += 5.0; n0, m = 32768, 2048
    else:
        rows = np.full((2, 20000), 3.5); n0, m = 20000, 700
    rows = rows.astype(np.float32)
    say("topk_rows", case, rows.shape, n0, step, m, split)
    if split == "bf16":  # the rows the fp8 index paths rank: rounded to bf16 first
        bits = encode_bf16(rows)
        rows = (bits.astype(np.uint32) << 16).view(np.float32)
        got = host(pv.pivot_topk_rows_bf16(dev(bits), n0, step, m))
    elif split:
        got = host(pv.pivot_topk_rows_ws(dev(rows), n0, step, m))
    else:
        got = host(pv.pivot_topk_rows(dev(rows), n0, step, m))
    for r in range(rows.shape[0]):
        n = n0 + r * step
        exp = _expect_topk(rows[r], n, m)
        assert sorted(got[r].tolist()) == sorted(exp.tolist()), (case, r)
