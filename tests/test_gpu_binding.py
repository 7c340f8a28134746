"""GPU tests of the Python binding's workspace handling: calls on two streams
at once use separate workspaces, and a call is sized for its own guardrail
setting (not the default one)."""
import numpy as np
import pytest
import torch

import paper_2607_24593_amd as pv
from gpu_util import dev, host, say
from parity import check_pivot
from workload.gen import make_prefill

import oracle

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def two_prefills():
    return make_prefill(6000, "fp8", seed=71, threads=8), make_prefill(6000, "fp8", seed=72, threads=8)


def _call(x, mode, stream, out):
    n = 6000
    p0, n_q = n - 2000, 2000
    sl = slice(p0, p0 + n_q)
    args = (dev(x.q[sl]), dev(x.q_scale[sl]), dev(x.w[sl]), dev(x.k), dev(x.k_scale), p0, n, 256)
    torch.cuda.synchronize()
    return args, lambda: pv.pivot_group_index(*args, mode=mode, g=4, c=1024, out=out, stream=stream)


def test_two_streams_do_not_share_a_workspace(two_prefills):
    """Refine on one stream and Reuse on another, issued back to back so they
    overlap on the GPU, give the same sets as the same calls one at a time on
    the current stream."""
    xa, xb = two_prefills
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
    ref_a = torch.empty((2000, 256), dtype=torch.int32, device="cuda")
    ref_b = torch.empty_like(ref_a)
    _, fa = _call(xa, pv.PIVOT_REFINE, None, ref_a)
    _, fb = _call(xb, pv.PIVOT_REUSE, None, ref_b)
    say("binding: one stream")
    fa()
    fb()
    ra, rb = host(ref_a), host(ref_b)
    out_a, out_b = torch.empty_like(ref_a), torch.empty_like(ref_b)
    _, ga = _call(xa, pv.PIVOT_REFINE, s1, out_a)
    _, gb = _call(xb, pv.PIVOT_REUSE, s2, out_b)
    say("binding: two streams")
    for _ in range(3):
        torch.cuda.synchronize()
        ga()
        gb()
        torch.cuda.synchronize()
        assert np.array_equal(np.sort(host(out_a), 1), np.sort(ra, 1))
        assert np.array_equal(np.sort(host(out_b), 1), np.sort(rb, 1))


def test_guardrail_off_short_chunk_fresh_stream():
    """dense_below = 0 on a chunk with every group below c: the call needs a
    proxy and re-score region that a workspace sized for the default guardrail
    (every group dense) lacks.  A new stream starts with an empty workspace
    cache, so the size the binding asks for is the one the call gets."""
    L, g, c, topk = 900, 4, 1024, 64
    x = make_prefill(L, "fp8", seed=73, threads=4)
    s = torch.cuda.Stream()
    out = torch.empty((L, topk), dtype=torch.int32, device="cuda")
    cand = torch.full((1, (L + g - 1) // g, c), -7, dtype=torch.int32, device="cuda")
    args = (dev(x.q), dev(x.q_scale), dev(x.w), dev(x.k), dev(x.k_scale), 0, L, topk)
    torch.cuda.synchronize()
    say("binding: dense_below=0 short chunk")
    with torch.cuda.stream(s):
        pv.pivot_group_index(*args, mode=pv.PIVOT_REFINE, g=g, c=c, dense_below=0, out=out, out_cand=cand,
                             stream=s)
    s.synchronize()
    check_pivot("fp8", x.q, x.q_scale, x.w, 0, x.k, x.k_scale, L, mode=oracle.REFINE, g=g, c=c, topk=topk,
                dense_below=0, gpu_idx=host(out), gpu_cand=host(cand)[0], groups=[0, 1, 2, 100, (L - 1) // g],
                label="db0 short")
