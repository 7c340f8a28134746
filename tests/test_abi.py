"""C ABI of libpivot.so on the CPU: the library loads, exports every function
include/pivot.h declares, and rejects bad arguments with the documented status
before launching anything (no call here reaches a kernel)."""
import ctypes
import os
import re

import pytest
import torch

import paper_2607_24593_amd as pv

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "pivot.h")

pytestmark = pytest.mark.skipif(not os.path.exists(pv.LIB_PATH), reason="libpivot.so not built")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"^[A-Za-z_][\w\s\*]*?\b(pivot_\w+)\s*\(", text, flags=re.M)))


def test_every_declared_symbol_is_exported():
    names = declared_functions()
    assert len(names) >= 10, names
    L = pv.lib()
    for n in names:
        assert hasattr(L, n), n
    assert sorted(names) == sorted(pv.EXPORTED)


def test_status_strings_and_version():
    assert pv.status_string(0) == "ok"
    assert "workspace" in pv.status_string(3)
    assert pv.status_string(99) == "unknown status"
    assert pv.version().startswith("pivot-gfx950")


FAKE = 1 << 40  # a non-null address the library must never dereference before launching


def args(dtype=pv.PIVOT_DT_FP8_E4M3, B=1, n_q=64, q_pos0=0, n_k=None, topk=8, heads=64, dim=128,
         scales=True, ws_bytes=0, ws_addr=FAKE):
    a = pv.pivot_args()
    a.dtype, a.heads, a.dim, a.batch, a.n_q = dtype, heads, dim, B, n_q
    pos = [q_pos0] * max(B, 1)
    nk = [q_pos0 + n_q if n_k is None else n_k] * max(B, 1)
    a._pos = (ctypes.c_int32 * len(pos))(*pos)
    a._nk = (ctypes.c_int32 * len(nk))(*nk)
    a.q_pos0 = ctypes.cast(a._pos, ctypes.POINTER(ctypes.c_int32))
    a.n_k = ctypes.cast(a._nk, ctypes.POINTER(ctypes.c_int32))
    a.q = a.w = a.k = a.out_idx = FAKE
    a.q_scale = a.k_scale = FAKE if scales else None
    a.k_seq_stride = max(nk + [0])
    a.topk = topk
    a.workspace = ws_addr
    a.workspace_bytes = ws_bytes
    a.stream = None
    return a


def dense(a):
    return pv.lib().pivot_dense_index(ctypes.byref(a))


def group(a, mode=pv.PIVOT_REFINE, g=4, c=16, db=-1):
    return pv.lib().pivot_group_index(ctypes.byref(a), mode, g, c, db, None)


def test_null_args():
    assert pv.lib().pivot_dense_index(None) == pv.PIVOT_ERR_INVALID_ARG
    assert pv.lib().pivot_workspace_size(None, -1, 1, 0) == 0


@pytest.mark.parametrize("kw,status", [
    (dict(heads=32), pv.PIVOT_ERR_UNSUPPORTED),
    (dict(dim=64), pv.PIVOT_ERR_UNSUPPORTED),
    (dict(dtype=5), pv.PIVOT_ERR_UNSUPPORTED),
    (dict(topk=0), pv.PIVOT_ERR_INVALID_ARG),
    (dict(n_q=-1), pv.PIVOT_ERR_INVALID_ARG),
    (dict(B=0), pv.PIVOT_ERR_INVALID_ARG),
    (dict(q_pos0=10, n_k=70), pv.PIVOT_ERR_INVALID_ARG),      # n_k < q_pos0 + n_q
    (dict(q_pos0=-3), pv.PIVOT_ERR_INVALID_ARG),
    (dict(scales=False), pv.PIVOT_ERR_INVALID_ARG),          # fp8 without scales
    (dict(q_pos0=pv.PIVOT_MAX_KEYS - 63, n_q=64), pv.PIVOT_ERR_UNSUPPORTED),  # n_k past the key limit
])
def test_dense_validation(kw, status):
    a = args(**kw)
    assert dense(a) == status
    assert pv.last_error() != ""


def test_missing_pointer():
    a = args()
    a.k = None
    assert dense(a) == pv.PIVOT_ERR_INVALID_ARG


def test_bf16_needs_no_scales():
    a = args(dtype=pv.PIVOT_DT_BF16, scales=False, ws_bytes=0)
    assert dense(a) == pv.PIVOT_ERR_WORKSPACE  # passes validation, stops at the workspace check


@pytest.mark.parametrize("mode,g,c,status", [
    (pv.PIVOT_REFINE, 0, 16, pv.PIVOT_ERR_INVALID_ARG),
    (pv.PIVOT_REFINE, 4, 4, pv.PIVOT_ERR_INVALID_ARG),        # c < k
    (pv.PIVOT_REFINE, 4, 16384, pv.PIVOT_ERR_UNSUPPORTED),    # c beyond the LDS budget
    (7, 4, 16, pv.PIVOT_ERR_INVALID_ARG),
    (pv.PIVOT_REUSE, 4, -1, pv.PIVOT_ERR_INVALID_ARG),
])
def test_group_validation(mode, g, c, status):
    assert group(args(), mode, g, c) == status


def opts(mode=pv.PIVOT_REFINE, g=4, c=16, db=-1, window=0, kind=pv.PIVOT_WINDOW_SHARED, agg=pv.PIVOT_AGG_MEAN,
         path=pv.PIVOT_REFINE_AUTO):
    return pv.group_opts(mode, g, c, db, window, kind, agg, refine_path=path)


def group_opts(a, o):
    return pv.lib().pivot_group_index_opts(ctypes.byref(a), ctypes.byref(o))


@pytest.mark.parametrize("kw,status", [
    (dict(window=-1), pv.PIVOT_ERR_INVALID_ARG),
    (dict(window=2, mode=pv.PIVOT_REUSE), pv.PIVOT_ERR_INVALID_ARG),              # the window is Refine only
    (dict(window=14, c=16), pv.PIVOT_ERR_INVALID_ARG),                            # shared: c < W + g - 1
    (dict(window=3, kind=pv.PIVOT_WINDOW_PER_QUERY), pv.PIVOT_ERR_INVALID_ARG),   # per-query: W < g
    (dict(window=4, kind=2), pv.PIVOT_ERR_INVALID_ARG),
    (dict(agg=3), pv.PIVOT_ERR_INVALID_ARG),
    (dict(agg=-1), pv.PIVOT_ERR_INVALID_ARG),
    (dict(c=4, window=8, kind=pv.PIVOT_WINDOW_PER_QUERY), pv.PIVOT_ERR_WORKSPACE),  # 4 + 11 >= topk: valid
    (dict(c=4), pv.PIVOT_ERR_INVALID_ARG),                                         # c < topk, no window
    (dict(c=8100, window=100, kind=pv.PIVOT_WINDOW_PER_QUERY), pv.PIVOT_ERR_UNSUPPORTED),  # 8203 slots
    (dict(c=16, window=13), pv.PIVOT_ERR_WORKSPACE),                               # c == W + g - 1: valid
    (dict(mode=pv.PIVOT_DENSE), pv.PIVOT_ERR_INVALID_ARG),
    (dict(path=3), pv.PIVOT_ERR_INVALID_ARG),
    (dict(path=-1), pv.PIVOT_ERR_INVALID_ARG),
    (dict(path=pv.PIVOT_REFINE_FUSED), pv.PIVOT_ERR_WORKSPACE),                    # valid: reaches the workspace check
    (dict(path=pv.PIVOT_REFINE_SPLIT), pv.PIVOT_ERR_WORKSPACE),
])
def test_group_opts_validation(kw, status):
    assert group_opts(args(ws_bytes=0), opts(**kw)) == status
    assert pv.last_error() != ""


def test_group_opts_null_and_plain_equivalence():
    L = pv.lib()
    assert L.pivot_group_index_opts(ctypes.byref(args()), None) == pv.PIVOT_ERR_INVALID_ARG
    assert L.pivot_cand_width(None) == 0
    assert L.pivot_group_workspace_size(None, ctypes.byref(opts())) == 0
    assert L.pivot_group_workspace_size(ctypes.byref(args()), None) == 0
    # without window and with the mean, the opts form sizes exactly as pivot_group_index
    a = args(n_q=100, q_pos0=900)
    for mode in (pv.PIVOT_REUSE, pv.PIVOT_REFINE):
        assert pv.pivot_group_workspace_size(a, opts(mode=mode, db=16)) == pv.pivot_workspace_size(a, mode, 4, 16)


def test_cand_width_and_window_workspace():
    assert pv.pivot_cand_width(opts(c=16)) == 16
    assert pv.pivot_cand_width(opts(c=16, window=5)) == 16                       # shared: inside c
    assert pv.pivot_cand_width(opts(c=16, window=5, kind=pv.PIVOT_WINDOW_PER_QUERY)) == 16 + 5 + 3
    up = lambda n: (n + 255) // 256 * 256  # noqa: E731
    a = args(n_q=100, q_pos0=900)
    base = pv.pivot_group_workspace_size(a, opts(db=16))
    per_q = pv.pivot_group_workspace_size(a, opts(db=16, window=5, kind=pv.PIVOT_WINDOW_PER_QUERY))
    ng, width = 25, 24
    # the candidate rows and the members' re-scores grow from c to c + W + g - 1 slots
    assert per_q - base == (up(ng * width * 4) + up(ng * 4 * width * 2)) - (up(ng * 16 * 4) + up(ng * 4 * 16 * 2))
    assert pv.pivot_group_workspace_size(a, opts(db=16, window=5)) == base
    assert pv.pivot_group_workspace_size(a, opts(window=3, kind=pv.PIVOT_WINDOW_PER_QUERY)) == 0  # invalid


def layout(cu_q=None, page_size=0, pool_keys=0, max_pages=0, table=False):
    lo = pv.pivot_layout()
    if cu_q is not None:
        lo._cu = (ctypes.c_int32 * len(cu_q))(*cu_q)
        lo.cu_q = ctypes.cast(lo._cu, ctypes.POINTER(ctypes.c_int32))
    if table:
        lo.block_table = FAKE
        lo.max_pages, lo.page_size, lo.pool_keys = max_pages, page_size, pool_keys
    return lo


def dense_layout(a, lo):
    return pv.lib().pivot_dense_index_layout(ctypes.byref(a), ctypes.byref(lo))


@pytest.mark.parametrize("kw,status", [
    (dict(cu_q=[1, 64]), pv.PIVOT_ERR_INVALID_ARG),                          # cu_q[0] != 0
    (dict(cu_q=[0, 40, 30]), pv.PIVOT_ERR_INVALID_ARG),                      # decreasing
    (dict(cu_q=[0, 40, 80]), pv.PIVOT_ERR_INVALID_ARG),                      # run 2 needs n_k >= 40
    (dict(table=True, page_size=24, pool_keys=96, max_pages=4), pv.PIVOT_ERR_INVALID_ARG),   # not a power of 2
    (dict(table=True, page_size=8, pool_keys=96, max_pages=8), pv.PIVOT_ERR_INVALID_ARG),    # below 16
    (dict(table=True, page_size=16, pool_keys=100, max_pages=4), pv.PIVOT_ERR_INVALID_ARG),  # not a multiple
    (dict(table=True, page_size=16, pool_keys=64, max_pages=2), pv.PIVOT_ERR_INVALID_ARG),   # n_k=64 > 2 pages
    (dict(table=True, page_size=16, pool_keys=64, max_pages=0), pv.PIVOT_ERR_INVALID_ARG),
    (dict(table=True, page_size=16, pool_keys=(1 << 24) + 16, max_pages=4), pv.PIVOT_ERR_UNSUPPORTED),  # > 2^31 B
    (dict(table=True, page_size=16, pool_keys=64, max_pages=4), pv.PIVOT_ERR_WORKSPACE),     # valid
    (dict(cu_q=[0, 64], table=True, page_size=64, pool_keys=128, max_pages=1), pv.PIVOT_ERR_WORKSPACE),
])
def test_layout_validation(kw, status):
    B = len(kw["cu_q"]) - 1 if "cu_q" in kw else 1
    a = args(B=B, ws_bytes=0)
    if B == 2:
        a._pos = (ctypes.c_int32 * 2)(0, 0)
        a._nk = (ctypes.c_int32 * 2)(64, 30)
        a.q_pos0 = ctypes.cast(a._pos, ctypes.POINTER(ctypes.c_int32))
        a.n_k = ctypes.cast(a._nk, ctypes.POINTER(ctypes.c_int32))
    lo = layout(**kw)
    assert dense_layout(a, lo) == status
    assert pv.lib().pivot_group_index_layout(ctypes.byref(a), ctypes.byref(lo), ctypes.byref(opts())) == status


def test_layout_workspace_sizes():
    """A one-run varlen layout sizes as the padded call; a ragged batch sizes its
    candidate rows by the sum of its runs' groups."""
    up = lambda n: (n + 255) // 256 * 256  # noqa: E731
    a = args(n_q=100, q_pos0=900)
    lo = layout(cu_q=[0, 100])
    L = pv.lib()
    for o in (None, opts(db=16), opts(mode=pv.PIVOT_REUSE, db=16)):
        ob = None if o is None else ctypes.byref(o)
        ref = pv.pivot_workspace_size(a, pv.PIVOT_DENSE) if o is None else pv.pivot_group_workspace_size(a, o)
        assert L.pivot_workspace_size_layout(ctypes.byref(a), ctypes.byref(lo), ob) == ref
    assert L.pivot_workspace_size_layout(ctypes.byref(a), None, None) == pv.pivot_workspace_size(a, pv.PIVOT_DENSE)
    # two runs of 10 and 7 rows: 3 + 2 groups of 4, 17 query rows; the score
    # tile holds both sequences' 3 group rows of ld(910) = 960 bf16 scores
    lin = lambda rows: up(rows * 512) + up(rows * 16)  # noqa: E731
    b = args(B=2, n_q=10, q_pos0=900)
    ragged = L.pivot_workspace_size_layout(ctypes.byref(b), ctypes.byref(layout(cu_q=[0, 10, 17])),
                                           ctypes.byref(opts(db=16)))
    ng = 5
    proxies = up(ng * 64 * 128) + up(ng * 4) + up(ng * 64 * 4)
    cand = up(ng * 16 * 4) + up(ng * 4 * 16 * 2)
    assert ragged == lin(17) + lin(ng) + proxies + cand + 2 * 3 * 960 * 2


def test_empty_runs_need_no_workspace():
    a = args(B=2, ws_bytes=0, ws_addr=None)
    lo = layout(cu_q=[0, 0, 0])
    assert dense_layout(a, lo) == pv.PIVOT_OK
    assert pv.lib().pivot_group_index_layout(ctypes.byref(a), ctypes.byref(lo), ctypes.byref(opts())) == pv.PIVOT_OK


def test_workspace_checks():
    a = args(ws_bytes=0)
    assert dense(a) == pv.PIVOT_ERR_WORKSPACE
    need = pv.pivot_workspace_size(a, pv.PIVOT_DENSE)
    assert need > 0
    a = args(ws_bytes=need, ws_addr=FAKE + 4)
    assert dense(a) == pv.PIVOT_ERR_INVALID_ARG                # misaligned
    a = args(ws_bytes=need // 8)
    assert dense(a) == pv.PIVOT_ERR_WORKSPACE
    a = args(ws_bytes=need, ws_addr=None)
    assert dense(a) == pv.PIVOT_ERR_WORKSPACE


def test_empty_call_is_ok_without_workspace():
    a = args(n_q=0, q_pos0=5, n_k=5, ws_bytes=0, ws_addr=None)
    assert dense(a) == pv.PIVOT_OK
    assert group(a) == pv.PIVOT_OK


def test_workspace_size_closed_form():
    up = lambda n: (n + 255) // 256 * 256  # noqa: E731
    lin = lambda rows: up(rows * 512) + up(rows * 16)  # noqa: E731  (fp8 epilogue's linear term)
    ld = lambda n: (((n + 63) // 64) | 1) * 64  # noqa: E731  (row stride: an odd multiple of 64 floats)
    assert ld(1000) == 1088 and ld(1024) == 1088 and ld(1088) == 1088
    # dense, one sequence: 100 rows x ld(1000)=1088 scores, bf16 for fp8
    # inputs, fp32 for bf16 inputs
    a = args(n_q=100, q_pos0=900)
    assert pv.pivot_workspace_size(a, pv.PIVOT_DENSE) == lin(100) + 100 * ld(1000) * 2
    b = args(n_q=100, q_pos0=900, dtype=pv.PIVOT_DT_BF16, scales=False)
    assert pv.pivot_workspace_size(b, pv.PIVOT_DENSE) == 100 * ld(1000) * 4
    # Refine, g=4, c=16, guardrail at c: all 25 groups start at t0 >= 900 >= c;
    # members need the linear term (Refine re-scores them), and so do proxies
    ng = 25
    proxies = up(ng * 64 * 128) + up(ng * 4) + up(ng * 64 * 4)
    cand = up(ng * 16 * 4) + up(ng * 4 * 16 * 2)   # candidate sets + members' re-scores
    assert pv.pivot_workspace_size(a, pv.PIVOT_REFINE, 4, 16) == \
        lin(100) + lin(ng) + proxies + cand + ng * ld(1000) * 2
    # Reuse: no candidate buffer, no member rows to re-score
    assert pv.pivot_workspace_size(a, pv.PIVOT_REUSE, 4, 16) == lin(ng) + proxies + ng * ld(1000) * 2
    # long prefix: score tiles stay near 1 GiB, plus the split select's scratch
    # for up to 256 long rows (16000 (key, position) pairs, 16 counts and a
    # threshold each)
    split = lambda rows: rows * (16000 * 8 + 16 * 4 + 4)  # noqa: E731
    a = args(n_q=16384, q_pos0=262144 - 16384)
    assert pv.pivot_workspace_size(a, pv.PIVOT_DENSE) == lin(16384) + split(256) + (1 << 30)
    assert pv.pivot_topk_rows_workspace_size(32) == split(32)
    assert pv.pivot_topk_rows_workspace_size(256) == split(256)
    assert pv.pivot_topk_rows_workspace_size(257) == 0 and pv.pivot_topk_rows_workspace_size(0) == 0


def test_stage_validation():
    L = pv.lib()
    assert L.pivot_score_rows(1, 64, 128, 4, FAKE, FAKE, FAKE, FAKE, FAKE, 10, 1, FAKE, 5, FAKE, 1 << 20, None) == \
        pv.PIVOT_ERR_INVALID_ARG                               # ld < lim + 1
    assert L.pivot_score_rows(1, 32, 128, 4, FAKE, FAKE, FAKE, FAKE, FAKE, 10, 1, FAKE, 64, FAKE, 1 << 20, None) == \
        pv.PIVOT_ERR_UNSUPPORTED
    assert L.pivot_score_rows(1, 64, 128, 4, FAKE, FAKE, FAKE, FAKE, FAKE, 10, 1, FAKE, pv.PIVOT_MAX_KEYS + 64,
                              FAKE, 1 << 20, None) == pv.PIVOT_ERR_UNSUPPORTED  # ld past the key limit
    need = pv.score_rows_workspace(4)
    assert L.pivot_score_rows(1, 64, 128, 4, FAKE, FAKE, FAKE, FAKE, FAKE, 10, 1, FAKE, 64, FAKE, need - 1, None) == \
        pv.PIVOT_ERR_WORKSPACE
    assert L.pivot_topk_rows(2, FAKE, 10, 8, 4, 4, FAKE, None) == pv.PIVOT_ERR_INVALID_ARG  # 12 > ld
    assert L.pivot_topk_rows(0, None, 0, 0, 0, 4, None, None) == pv.PIVOT_OK
    assert L.pivot_topk_rows_ws(2, FAKE, 64, 8, 4, 4, FAKE, FAKE + 4, 1 << 20, None) == \
        pv.PIVOT_ERR_INVALID_ARG                               # misaligned workspace
    assert L.pivot_topk_rows_ws(2, FAKE, 10, 8, 4, 4, FAKE, FAKE, 1 << 20, None) == pv.PIVOT_ERR_INVALID_ARG
    assert L.pivot_proxy_rows(1, 64, 128, 8, 0, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, None) == \
        pv.PIVOT_ERR_INVALID_ARG
    assert L.pivot_encode_e4m3(None, None, 0, None) == pv.PIVOT_OK


def test_binding_fails_loudly_without_library(monkeypatch, tmp_path):
    monkeypatch.setattr(pv, "LIB_PATH", str(tmp_path / "missing.so"))
    monkeypatch.setattr(pv, "_lib", None)
    with pytest.raises(RuntimeError, match="HIP library missing"):
        pv.lib()


def test_profile_kind_mask():
    """pivot_profile_begin_kinds: empty or out-of-range masks are rejected, a
    valid one starts a profile that ends with no launches counted."""
    L = pv.lib()
    assert L.pivot_profile_begin_kinds(0) == pv.PIVOT_ERR_INVALID_ARG
    assert L.pivot_profile_begin_kinds(1 << len(pv.KERNELS)) == pv.PIVOT_ERR_INVALID_ARG
    pv.pivot_profile_begin(["score", "select"])
    assert L.pivot_profile_begin() == pv.PIVOT_ERR_INVALID_ARG     # one profile at a time
    prof = pv.pivot_profile_end()
    assert all(n == 0 for n, _ in prof.values())


def layers_call(layers, stride=1, anchors=None, o=None):
    arr = (pv.pivot_args * len(layers))(*layers)
    anc = None if anchors is None else (ctypes.c_uint8 * len(anchors))(*anchors)
    return pv.lib().pivot_index_layers(arr, len(layers), stride, anc, None if o is None else ctypes.byref(o))


def _mismatch(field, value):
    b = args(ws_bytes=0)
    setattr(b, field, value)
    return [args(ws_bytes=0), b]


@pytest.mark.parametrize("make,kw,status", [
    (lambda: [args()], dict(stride=0), pv.PIVOT_ERR_INVALID_ARG),                   # stride < 1, no anchors
    (lambda: [args(), args()], dict(anchors=[0, 1]), pv.PIVOT_ERR_INVALID_ARG),     # layer 0 not an anchor
    (lambda: _mismatch("n_q", 32), {}, pv.PIVOT_ERR_INVALID_ARG),
    (lambda: _mismatch("topk", 4), {}, pv.PIVOT_ERR_INVALID_ARG),
    (lambda: _mismatch("dtype", pv.PIVOT_DT_BF16), {}, pv.PIVOT_ERR_INVALID_ARG),
    (lambda: [args(), args(q_pos0=1, n_k=65)], {}, pv.PIVOT_ERR_INVALID_ARG),       # positions differ
    (lambda: _mismatch("out_idx", None), dict(stride=2), pv.PIVOT_ERR_INVALID_ARG),  # follower without output
    (lambda: [args(ws_bytes=0), args(ws_bytes=0)], dict(stride=2), pv.PIVOT_ERR_WORKSPACE),
    (lambda: [args(ws_bytes=0), args(ws_bytes=0)], dict(stride=1), pv.PIVOT_ERR_WORKSPACE),
    (lambda: [args(topk=0), args(topk=0)], dict(stride=2), pv.PIVOT_ERR_INVALID_ARG),  # anchor's own check
])
def test_index_layers_validation(make, kw, status):
    """Every layer is checked before a launch; a follower's inputs may be NULL."""
    assert layers_call(make(), **kw) == status
    assert pv.last_error() != ""


def test_index_layers_follower_inputs_unread_and_opts_checked():
    L = pv.lib()
    assert L.pivot_index_layers(None, 1, 1, None, None) == pv.PIVOT_ERR_INVALID_ARG
    follower = args(ws_bytes=0)
    follower.q = follower.w = follower.k = follower.q_scale = follower.k_scale = None
    # validation reaches layer 0's workspace check: the NULL follower inputs are accepted
    assert layers_call([args(ws_bytes=0), follower], stride=2, o=opts()) == pv.PIVOT_ERR_WORKSPACE
    # the same NULL inputs on an anchor layer are rejected
    assert layers_call([args(ws_bytes=0), follower], stride=1, o=opts()) == pv.PIVOT_ERR_INVALID_ARG
    o = opts()
    o.out_cand = FAKE
    assert layers_call([args(), args()], stride=1, o=o) == pv.PIVOT_ERR_INVALID_ARG
    assert layers_call([args(ws_bytes=0)], stride=1, o=opts(g=0)) == pv.PIVOT_ERR_INVALID_ARG


def test_noalloc_size_check_precedes_the_device():
    """pivot_group_index_noalloc checks its arguments and its scratch budget
    before any HIP call: these fail the same way with no GPU."""
    L = pv.lib()
    assert L.pivot_group_index_noalloc(None, ctypes.byref(opts())) == pv.PIVOT_ERR_INVALID_ARG
    assert L.pivot_group_index_noalloc(ctypes.byref(args()), None) == pv.PIVOT_ERR_INVALID_ARG
    big = args(n_q=8192, q_pos0=131072 - 8192, topk=2048)
    o = opts(mode=pv.PIVOT_REFINE, g=4, c=4096)
    assert L.pivot_group_index_noalloc(ctypes.byref(big), ctypes.byref(o)) == pv.PIVOT_ERR_WORKSPACE
    assert "no-alloc scratch" in pv.last_error()
    empty = args(n_q=0)
    assert L.pivot_group_index_noalloc(ctypes.byref(empty), ctypes.byref(o)) == pv.PIVOT_OK
