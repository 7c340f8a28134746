"""GPU test of pivot_group_index_noalloc, the entry point that allocates
nothing (its scratch is an array the library holds per device): called
through the C ABI, its index sets equal those of pivot_group_index_opts on
the same inputs, over consecutive calls whose second is smaller than the
first (the scratch keeps the previous call's contents)."""
import ctypes

import numpy as np
import pytest
import torch

import paper_2607_24593_amd as pv
from gpu_util import dev, host, say
from workload.gen import make_decode, make_prefill

pytestmark = pytest.mark.gpu


def _compare(label, q, qs, w, k, ks, pos, nk, topk, mode, g, c):
    shape = tuple(q.shape[:-2]) + (topk,)
    say("noalloc", label, "existing entry point")
    ref = pv.pivot_group_index_opts(q, qs, w, k, ks, pos, nk, topk, mode=mode, g=g, c=c)
    out = torch.full(shape, -7, dtype=torch.int32, device="cuda")
    a = pv.make_args(q, qs, w, k, ks, pos, nk, topk, out)
    a.workspace, a.workspace_bytes = None, 0  # ignored by the no-alloc entry point
    o = pv.group_opts(mode, g, c, -1)
    torch.cuda.synchronize()
    say("noalloc", label, "no-alloc entry point")
    st = pv.lib().pivot_group_index_noalloc(ctypes.byref(a), ctypes.byref(o))
    assert st == pv.PIVOT_OK, (st, pv.last_error())
    got, exp = host(out), host(ref)
    assert np.array_equal(np.sort(got, -1), np.sort(exp, -1)), label


def test_noalloc_matches_group_index_on_consecutive_calls():
    B, L, g = 8, 20000, 2
    x = make_decode(B, L, g, "fp8", seed=91, threads=6)
    _compare("decode 8x20000 refine", dev(x.q), dev(x.q_scale), dev(x.w), dev(x.k), dev(x.k_scale), [L - g] * B,
             [L] * B, 256, pv.PIVOT_REFINE, g, 1024)
    B, L = 3, 9000  # smaller: the scratch still holds the first call's data
    x = make_decode(B, L, g, "fp8", seed=92, threads=6)
    _compare("decode 3x9000 refine", dev(x.q), dev(x.q_scale), dev(x.w), dev(x.k), dev(x.k_scale), [L - g] * B,
             [L] * B, 256, pv.PIVOT_REFINE, g, 1024)
    L, p0 = 12048, 10000
    x = make_prefill(L, "fp8", seed=93, threads=8)
    sl = slice(p0, L)
    _compare("prefill chunk reuse", dev(x.q[sl]), dev(x.q_scale[sl]), dev(x.w[sl]), dev(x.k), dev(x.k_scale), p0, L,
             2048, pv.PIVOT_REUSE, 4, 4096)
    _compare("prefill chunk refine", dev(x.q[sl]), dev(x.q_scale[sl]), dev(x.w[sl]), dev(x.k), dev(x.k_scale), p0,
             L, 2048, pv.PIVOT_REFINE, 4, 4096)


def test_noalloc_rejects_calls_beyond_its_scratch():
    """An 8192-query Refine chunk at 131072 keys needs more than the scratch:
    the call returns PIVOT_ERR_WORKSPACE and leaves the output untouched."""
    L, n = 131072, 8192
    q = torch.zeros((n, 64, 128), dtype=torch.uint8, device="cuda")
    qs = torch.ones(n, dtype=torch.float32, device="cuda")
    w = torch.zeros((n, 64), dtype=torch.float32, device="cuda")
    k = torch.zeros((L, 128), dtype=torch.uint8, device="cuda")
    ks = torch.ones(L, dtype=torch.float32, device="cuda")
    out = torch.full((n, 2048), -7, dtype=torch.int32, device="cuda")
    a = pv.make_args(q, qs, w, k, ks, L - n, L, 2048, out)
    o = pv.group_opts(pv.PIVOT_REFINE, 4, 4096, -1)
    torch.cuda.synchronize()
    assert pv.lib().pivot_group_index_noalloc(ctypes.byref(a), ctypes.byref(o)) == pv.PIVOT_ERR_WORKSPACE
    assert "no-alloc scratch" in pv.last_error()
    assert bool((out == -7).all())
