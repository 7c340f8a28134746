"""GPU parity of PIVOT composed with IndexCache (pivot_index_layers; Sec. 5.1
"Baselines", the +IC rows of Table 1): the anchor layers against the oracle's
layer function, the followers entry for entry against the anchor they share,
and an anchor layer against the single-layer entry point."""
import numpy as np
import pytest
import torch

import oracle
import paper_2607_24593_amd as pv
from gpu_util import dev, host, say
from parity import check_pivot
from workload.gen import WORKLOADS, make, make_decode, make_prefill

pytestmark = pytest.mark.gpu

MODES = {None: oracle.DENSE, pv.PIVOT_REUSE: oracle.REUSE, pv.PIVOT_REFINE: oracle.REFINE}


@pytest.fixture(scope="module")
def layer_inputs():
    """Four layers of a 6000-token fp8 prefill with inputs of their own."""
    return [make_prefill(6000, "fp8", seed=500 + l, threads=8) for l in range(4)]


def _run(xs, p0, n, mode, g, c, topk, stride=1, anchors=None, drop_followers=False):
    sl = slice(p0, p0 + n)
    layers = []
    for l, x in enumerate(xs):
        is_anchor = anchors[l] if anchors is not None else l % stride == 0
        if drop_followers and not is_anchor:
            layers.append(None)
        else:
            layers.append((dev(x.q[sl]), dev(x.q_scale[sl]), dev(x.w[sl]), dev(x.k[:p0 + n]),
                           dev(x.k_scale[:p0 + n])))
    say("index_layers", "mode", mode, "stride", stride, "anchors", anchors, "p0", p0, "n", n)
    outs = pv.pivot_index_layers(layers, p0, p0 + n, topk, stride=stride, anchors=anchors, mode=mode, g=g, c=c)
    return [host(o) for o in outs]


def _single_cand(args, B, n, g, c, topk):
    """Refine's candidate sets for the two-stage parity check: the layer call
    has no candidate output, so the single-layer call on the same inputs gives
    them, and the test requires its index sets to equal the layer's."""
    ng = (n + g - 1) // g
    ct = torch.full((B, ng, c), -7, dtype=torch.int32, device="cuda")
    idx = pv.pivot_group_index(*args, topk, mode=pv.PIVOT_REFINE, g=g, c=c, out_cand=ct)
    return host(idx), host(ct)


@pytest.mark.parametrize("mode", [pv.PIVOT_REFINE, pv.PIVOT_REUSE, None])
@pytest.mark.parametrize("stride,anchors", [(2, None), (1, [1, 0, 0, 1])])
def test_layers_match_oracle(layer_inputs, mode, stride, anchors):
    xs = layer_inputs
    p0, n, g, c, topk = 4000, 2000, 4, 1024, 256
    outs = _run(xs, p0, n, mode, g, c, topk, stride, anchors, drop_followers=True)
    anc = oracle.layer_anchors(len(xs), stride) if anchors is None else np.asarray(anchors, np.uint8)
    rng = np.random.default_rng(3)
    gg = g if mode is not None else 1
    ng = (n + gg - 1) // gg
    groups = sorted({0, ng - 1} | set(int(v) for v in rng.integers(0, ng, 6)))
    src = 0
    for l, x in enumerate(xs):
        if anc[l]:
            src = l
            sl = slice(p0, p0 + n)
            cand = None
            if mode == pv.PIVOT_REFINE:
                args = (dev(x.q[sl]), dev(x.q_scale[sl]), dev(x.w[sl]), dev(x.k[:p0 + n]), dev(x.k_scale[:p0 + n]),
                        p0, p0 + n)
                one, cand = _single_cand(args, 1, n, g, c, topk)
                assert np.array_equal(np.sort(one, 1), np.sort(outs[l], 1)), l
                cand = cand[0]
            check_pivot("fp8", x.q[sl], x.q_scale[sl], x.w[sl], p0, x.k[:p0 + n], x.k_scale[:p0 + n], p0 + n,
                        mode=MODES[mode], g=gg, c=c, topk=topk, dense_below=-1, gpu_idx=outs[l], gpu_cand=cand,
                        groups=groups, label=f"layer {l}")
        else:
            # the oracle's layer function gives a follower its anchor's sets
            # (pinned on the CPU), so the follower passes exactly when it
            # holds the GPU anchor's sets, entry for entry
            assert np.array_equal(outs[l], outs[src]), (l, src)


def test_anchor_equals_single_layer_call(layer_inputs):
    """An anchor layer is exactly the single-layer pivot_group_index call."""
    xs = layer_inputs
    p0, n = 4000, 2000
    outs = _run(xs, p0, n, pv.PIVOT_REFINE, 4, 1024, 256, stride=2)
    sl = slice(p0, p0 + n)
    for l in (0, 2):
        x = xs[l]
        one = pv.pivot_group_index(dev(x.q[sl]), dev(x.q_scale[sl]), dev(x.w[sl]), dev(x.k[:p0 + n]),
                                   dev(x.k_scale[:p0 + n]), p0, p0 + n, 256, mode=pv.PIVOT_REFINE, g=4, c=1024)
        assert np.array_equal(np.sort(host(one), 1), np.sort(outs[l], 1)), l
    assert not np.array_equal(np.sort(outs[0], 1), np.sort(outs[2], 1))


def test_many_followers_and_decode_batch():
    """More followers than one copy launch takes (17 after the anchor), over a
    decode batch (B sequences, one MTP group each)."""
    B, L, g = 3, 5000, 2
    x = make_decode(B, L, g, "fp8", seed=77, threads=6)
    q, qs, w, k, ks = dev(x.q), dev(x.q_scale), dev(x.w), dev(x.k), dev(x.k_scale)
    n_layers = 18
    layers = [(q, qs, w, k, ks)] + [None] * (n_layers - 1)
    say("index_layers decode", n_layers)
    outs = pv.pivot_index_layers(layers, [L - g] * B, [L] * B, 256, stride=n_layers, mode=pv.PIVOT_REFINE, g=g,
                                 c=1024)
    ref = host(outs[0])
    for l in range(1, n_layers):
        assert np.array_equal(host(outs[l]), ref), l
    one, cand = _single_cand((q, qs, w, k, ks, [L - g] * B, [L] * B), B, g, g, 1024, 256)
    assert np.array_equal(np.sort(one, -1), np.sort(ref, -1))
    for b in range(B):
        check_pivot("fp8", x.q[b], x.q_scale[b], x.w[b], L - g, x.k[b], x.k_scale[b], L, mode=oracle.REFINE, g=g,
                    c=1024, topk=256, dense_below=-1, gpu_idx=ref[b], gpu_cand=cand[b], label=f"ic decode b{b}")


def test_prefill_128k_two_layers_stride_two():
    """The full-size shape: the last 8192-query chunk of the 128K prefill for
    two layers at stride 2 (the second layer takes the first's sets)."""
    wl = WORKLOADS["prefill-128k-fp8"]
    say("generate", wl.name)
    x = make(wl, threads=16)
    p0, n = wl.L - wl.chunk, wl.chunk
    sl = slice(p0, p0 + n)
    layer = (dev(x.q[sl]), dev(x.q_scale[sl]), dev(x.w[sl]), dev(x.k), dev(x.k_scale))
    say("index_layers 128k")
    outs = pv.pivot_index_layers([layer, None], p0, p0 + n, wl.topk, stride=2, mode=pv.PIVOT_REFINE, g=4, c=wl.c)
    a, f = host(outs[0]), host(outs[1])
    assert np.array_equal(a, f)
    one, cand = _single_cand(layer + (p0, p0 + n), 1, n, 4, wl.c, wl.topk)
    assert np.array_equal(np.sort(one, 1), np.sort(a, 1))
    rng = np.random.default_rng(12)
    groups = sorted({0, n // 4 - 1} | set(int(v) for v in rng.integers(0, n // 4, 5)))
    check_pivot("fp8", x.q[sl], x.q_scale[sl], x.w[sl], p0, x.k, x.k_scale, wl.L, mode=oracle.REFINE, g=4,
                c=wl.c, topk=wl.topk, dense_below=-1, gpu_idx=a, gpu_cand=cand[0], groups=groups, label="128k ic")
    del layer
    torch.cuda.empty_cache()
