"""Index calls captured into a HIP graph (torch.cuda.CUDAGraph) and replayed:
the library allocates, copies and clears nothing inside a call, so a call
captures whole.  Each replay, with other eager work and synchronisations
between replays, must give the eager call's sets."""
import numpy as np
import pytest
import torch

import paper_2607_24593_amd as pv
from gpu_util import dev, host, say
from workload.gen import make_decode

pytestmark = pytest.mark.gpu

B, L, G, C, TOPK = 4, 32768, 2, 4096, 2048


@pytest.fixture(scope="module")
def inputs():
    x = make_decode(B, L, G, "fp8", seed=91, threads=16)
    return [dev(a) for a in (x.q, x.q_scale, x.w, x.k, x.k_scale)]


def _sets(t):
    return np.sort(host(t), axis=-1)


@pytest.mark.parametrize("mode", ["dense", "reuse", "refine", "refine_window"])
def test_graph_replays_match_eager(inputs, mode):
    q, qs, w, k, ks = inputs
    pos, nk = [L - G] * B, [L] * B
    out = torch.full((B, G, TOPK), -7, dtype=torch.int32, device="cuda")

    def call(ws=None):
        if mode == "dense":
            return pv.pivot_dense_index(q, qs, w, k, ks, pos, nk, TOPK, out=out, ws=ws)
        if mode == "refine_window":
            return pv.pivot_group_index_opts(q, qs, w, k, ks, pos, nk, TOPK, mode=pv.PIVOT_REFINE, g=G, c=C,
                                             window=4, window_kind=pv.PIVOT_WINDOW_PER_QUERY, out=out, ws=ws)
        m = pv.PIVOT_REUSE if mode == "reuse" else pv.PIVOT_REFINE
        return pv.pivot_group_index(q, qs, w, k, ks, pos, nk, TOPK, mode=m, g=G, c=C, out=out, ws=ws)

    say("graph eager", mode)
    call()
    want = _sets(out)
    ws = pv.workspace(0, q.device)
    graph = torch.cuda.CUDAGraph()
    say("graph capture", mode)
    with torch.cuda.graph(graph):
        call(ws)
    for rep in range(3):
        out.fill_(-7)
        # other eager work between replays: a dense call on shifted positions into another buffer
        pv.pivot_dense_index(q, qs, w, k, ks, [L - G - 1 - rep] * B, [L - 1 - rep] * B, TOPK)
        torch.cuda.synchronize()
        say("graph replay", mode, rep)
        graph.replay()
        got = _sets(out)
        assert np.array_equal(got, want), (mode, rep)
