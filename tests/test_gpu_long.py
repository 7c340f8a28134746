"""GPU parity past the named workloads' lengths: 2^20 keys per sequence (four
times the longest configuration, well inside the 2^27 limit).  Score rows of
a million entries take the select's long-row paths (the sampled threshold
declines rows whose expected candidate count would overflow its buffer, and
the row falls back to the exact two-pass select), and the score tiles split
the launch.  Decode (two sequences, an MTP step of g = 2) and a 512-query
prefill chunk at the end of a 2^20-token prefix are checked against the
oracle, the chunk on sampled groups."""
import numpy as np
import pytest
import torch

import oracle
import paper_2607_24593_amd as pv
from gpu_util import dev, host, say
from parity import check_pivot
from workload.gen import make_decode

pytestmark = pytest.mark.gpu

L = 1 << 20
MODES = {"dense": oracle.DENSE, "reuse": oracle.REUSE, "refine": oracle.REFINE}


@pytest.fixture(scope="module")
def dec():
    say("generate decode", 2, L)
    return make_decode(2, L, 2, "fp8", seed=71, threads=16)


@pytest.fixture(scope="module")
def chunk():
    say("generate chunk", 1, L, 512)
    return make_decode(1, L, 512, "fp8", seed=72, threads=16)


@pytest.mark.parametrize("mode", ["dense", "reuse", "refine"])
def test_decode_1m_keys(dec, mode):
    x = dec
    B, g, c, topk = 2, 2, 4096, 2048
    q, qs, w, k, ks = dev(x.q), dev(x.q_scale), dev(x.w), dev(x.k), dev(x.k_scale)
    say("decode 1M", mode)
    cand = None
    if mode == "dense":
        idx = pv.pivot_dense_index(q, qs, w, k, ks, [L - g] * B, [L] * B, topk)
    else:
        ct = torch.full((B, 1, c), -7, dtype=torch.int32, device="cuda") if mode == "refine" else None
        idx = pv.pivot_group_index(q, qs, w, k, ks, [L - g] * B, [L] * B, topk,
                                   mode=pv.PIVOT_REUSE if mode == "reuse" else pv.PIVOT_REFINE, g=g, c=c,
                                   out_cand=ct)
        cand = None if ct is None else host(ct)
    idx = host(idx)
    for b in range(B):
        check_pivot("fp8", x.q[b], x.q_scale[b], x.w[b], L - g, x.k[b], x.k_scale[b], L, mode=MODES[mode], g=g,
                    c=c, topk=topk, dense_below=-1, gpu_idx=idx[b], gpu_cand=None if cand is None else cand[b],
                    label=f"decode 1M {mode} b{b}")


@pytest.mark.parametrize("mode", ["dense", "reuse", "refine"])
def test_prefill_chunk_1m_keys(chunk, mode):
    x = chunk
    n_q, c, topk = 512, 4096, 2048
    g = 1 if mode == "dense" else 4
    p0 = L - n_q
    q, qs, w, k, ks = dev(x.q[0]), dev(x.q_scale[0]), dev(x.w[0]), dev(x.k[0]), dev(x.k_scale[0])
    say("prefill chunk 1M", mode)
    cand = None
    if mode == "dense":
        idx = pv.pivot_dense_index(q, qs, w, k, ks, p0, L, topk)
    else:
        ct = torch.full((1, n_q // g, c), -7, dtype=torch.int32, device="cuda") if mode == "refine" else None
        idx = pv.pivot_group_index(q, qs, w, k, ks, p0, L, topk,
                                   mode=pv.PIVOT_REUSE if mode == "reuse" else pv.PIVOT_REFINE, g=g, c=c,
                                   out_cand=ct)
        cand = None if ct is None else host(ct)[0]
    idx = host(idx)
    rng = np.random.default_rng(5)
    ng = n_q // g
    groups = sorted({0, ng - 1} | set(int(v) for v in rng.integers(0, ng, 2)))
    check_pivot("fp8", x.q[0], x.q_scale[0], x.w[0], p0, x.k[0], x.k_scale[0], L, mode=MODES[mode], g=g, c=c,
                topk=topk, dense_below=-1, gpu_idx=idx, gpu_cand=cand, groups=groups, label=f"chunk 1M {mode}")
