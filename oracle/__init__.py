"""CPU oracle for the PIVOT indexer path (test infrastructure only).

Only the test suite, the package smoke check and the benchmark's CPU-baseline
leg may import this package.  It wraps `pivot_oracle.c`, a plain fp64 C
restatement of the lightning-indexer score (Sec. 3.1 Eq. 1, App. A), TopK, and
Algorithm 1 of App. E (grouping Eqs. 2-3, proxy Eq. 4, proxy scan Eq. 5,
Reuse Eq. 6, Refine Eqs. 7-9, short-group guardrail), and its composition with
IndexCache across layers (Sec. 5.1 "Baselines").  The library is built
with gcc; nothing here touches the GPU path.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "pivot_oracle.c")
_LIB = os.environ.get("PIVOT_ORACLE_LIB") or os.path.join(_HERE, "libpivot_oracle.so")

DENSE, REUSE, REFINE = 0, 1, 2
FMT = {"bf16": 0, "fp8": 1}
WINDOW_SHARED, WINDOW_PER_QUERY = 0, 1     # App. B: prefill and decode readings
AGG_MEAN, AGG_FIRST, AGG_LAST = 0, 1, 2    # Eq. 4 mean, or one member's row


def compile_source(src: str, out: str) -> str:
    """gcc -O2 with OpenMP and no FMA contraction (the proxy's fp32 steps are
    rounded one operation at a time)."""
    tmp = out + ".tmp"
    subprocess.check_call(["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-fopenmp",
                           "-ffp-contract=off", "-fno-fast-math", "-Wall", "-Wextra",
                           "-Wno-unused-parameter", src, "-o", tmp, "-lm"])
    os.replace(tmp, out)
    return out


def build(force: bool = True) -> str:
    """Compile the oracle library next to its source."""
    if force or not os.path.exists(_LIB):
        compile_source(_SRC, _LIB)
    return _LIB


_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build()
        L = ctypes.CDLL(_LIB)
        P, I, I64, F = ctypes.c_void_p, ctypes.c_int, ctypes.c_int64, ctypes.c_float
        L.oracle_e4m3_decode.restype = ctypes.c_double
        L.oracle_e4m3_decode.argtypes = [ctypes.c_uint8]
        L.oracle_e4m3_encode.restype = ctypes.c_uint8
        L.oracle_e4m3_encode.argtypes = [F]
        L.oracle_bf16_decode.restype = ctypes.c_double
        L.oracle_bf16_decode.argtypes = [ctypes.c_uint16]
        L.oracle_bf16_encode.restype = ctypes.c_uint16
        L.oracle_bf16_encode.argtypes = [F]
        L.oracle_topk.argtypes = [P, P, I64, I, P]
        L.oracle_proxy.argtypes = [I, I, I, P, P, P, I, P, P, P]
        L.oracle_scores.argtypes = [I, I, I, P, F, P, P, P, I64, P]
        L.oracle_scores_at.argtypes = [I, I, I, P, F, P, P, P, P, I64, P]
        L.oracle_refine_on.argtypes = [I, I, I, P, P, P, I, P, P, P, I64, I, P]
        L.oracle_index.argtypes = [I, I, I, P, P, P, I, I64, P, P, I64,
                                   I, I, I, I, I, P, I, P, P, P, P, P]
        L.oracle_index_ex.argtypes = [I, I, I, P, P, P, I, I64, P, P, I64,
                                      I, I, I, I, I, I, I, I, P, I, P, P, P, P, P]
        L.oracle_index_layers.argtypes = [I, I, I, I, P, P, P, P, I, I64, P, P, I64, I, I, I, I, I, P]
        L.oracle_num_threads.restype = I
        _lib = L
    return _lib


def _p(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _c(a, dt):
    return None if a is None else np.ascontiguousarray(a, dtype=dt)


def _code_dtype(fmt: str):
    return np.uint8 if fmt == "fp8" else np.uint16


def num_threads() -> int:
    return lib().oracle_num_threads()


# ---------------------------------------------------------------- codecs
def e4m3_decode(code: int) -> float:
    return lib().oracle_e4m3_decode(int(code))


def e4m3_encode(x: float) -> int:
    return lib().oracle_e4m3_encode(float(x))


def bf16_decode(bits: int) -> float:
    return lib().oracle_bf16_decode(int(bits))


def bf16_encode(x: float) -> int:
    return lib().oracle_bf16_encode(float(x))


# ---------------------------------------------------------------- steps
def topk(f, pos, m: int) -> np.ndarray:
    f = _c(f, np.float64)
    pos = _c(pos, np.int32)
    out = np.empty(m, dtype=np.int32)
    lib().oracle_topk(_p(f), _p(pos), len(f), m, _p(out))
    return out


def proxy(fmt: str, q, q_scale, w):
    """Eq. 4 proxy of the members q [gs,H,d], q_scale [gs], w [gs,H]."""
    q = _c(q, _code_dtype(fmt))
    gs, H, d = q.shape
    qs = _c(q_scale, np.float32) if fmt == "fp8" else None
    w = _c(w, np.float32)
    pq = np.empty((H, d), dtype=_code_dtype(fmt))
    psc = np.zeros(1, dtype=np.float32)
    pw = np.empty(H, dtype=np.float32)
    rc = lib().oracle_proxy(FMT[fmt], H, d, _p(q), _p(qs), _p(w), gs, _p(pq), _p(psc), _p(pw))
    assert rc == 0
    return pq, float(psc[0]), pw


def scores(fmt: str, q_row, sq, w_row, k, k_scale, lim: int) -> np.ndarray:
    """Scores of one row (H,d codes) over key positions [0, lim], in fp64."""
    q_row = _c(q_row, _code_dtype(fmt))
    H, d = q_row.shape
    w_row = _c(w_row, np.float32)
    k = _c(k, _code_dtype(fmt))
    ks = _c(k_scale, np.float32) if fmt == "fp8" else None
    out = np.empty(lim + 1, dtype=np.float64)
    lib().oracle_scores(FMT[fmt], H, d, _p(q_row), float(sq if fmt == "fp8" else 1.0), _p(w_row),
                        _p(k), _p(ks), lim, _p(out))
    return out


def scores_at(fmt: str, q_row, sq, w_row, k, k_scale, pos) -> np.ndarray:
    q_row = _c(q_row, _code_dtype(fmt))
    H, d = q_row.shape
    w_row = _c(w_row, np.float32)
    k = _c(k, _code_dtype(fmt))
    ks = _c(k_scale, np.float32) if fmt == "fp8" else None
    pos = _c(pos, np.int32)
    out = np.empty(len(pos), dtype=np.float64)
    lib().oracle_scores_at(FMT[fmt], H, d, _p(q_row), float(sq if fmt == "fp8" else 1.0),
                           _p(w_row), _p(k), _p(ks), _p(pos), len(pos), _p(out))
    return out


def refine_on(fmt: str, q, q_scale, w, k, k_scale, cand, m: int) -> np.ndarray:
    """Eqs. 8-9: members q [gs,H,d] re-score the given candidates, top-m each."""
    q = _c(q, _code_dtype(fmt))
    gs, H, d = q.shape
    qs = _c(q_scale, np.float32) if fmt == "fp8" else None
    w = _c(w, np.float32)
    k = _c(k, _code_dtype(fmt))
    ks = _c(k_scale, np.float32) if fmt == "fp8" else None
    cand = _c(cand, np.int32)
    cand = cand[cand >= 0]
    out = np.empty((gs, m), dtype=np.int32)
    lib().oracle_refine_on(FMT[fmt], H, d, _p(q), _p(qs), _p(w), gs, _p(k), _p(ks),
                           _p(cand), len(cand), m, _p(out))
    return out


def cand_width(c: int, g: int, window: int = 0, window_kind: int = WINDOW_SHARED) -> int:
    """Candidate slots per group: c, or c + W + g - 1 with the decode window."""
    return c + window + g - 1 if (window > 0 and window_kind == WINDOW_PER_QUERY) else c


def index(fmt: str, q, q_scale, w, p0: int, k, k_scale, n_k: int, *, mode: int, g: int = 1,
          c: int = 0, topk: int, dense_below: int | None = None, groups=None,
          want_cand: bool = False, want_proxy: bool = False, window: int = 0,
          window_kind: int = WINDOW_SHARED, agg: int = AGG_MEAN):
    """Algorithm 1 over one sequence's queries q [n_q,H,d] at positions p0.. .

    mode DENSE / REUSE / REFINE.  dense_below defaults to c (the guardrail of
    Algorithm 1); 0 disables it.  window / window_kind: App. B's local window
    (Refine only).  agg: proxy aggregation.  groups: optional list of group
    indices to compute (rows of other groups are returned as -2).  Returns a
    dict with 'idx' [n_q, topk] and, if asked, 'cand' [n_groups, width] and the
    proxies."""
    q = _c(q, _code_dtype(fmt))
    n_q, H, d = q.shape
    qs = _c(q_scale, np.float32) if fmt == "fp8" else None
    w = _c(w, np.float32)
    k = _c(k, _code_dtype(fmt))
    ks = _c(k_scale, np.float32) if fmt == "fp8" else None
    if mode == DENSE:
        g = 1
    if dense_below is None:
        dense_below = c if mode != DENSE else 0
    n_groups = (n_q + g - 1) // g
    sel = None if groups is None else np.ascontiguousarray(groups, dtype=np.int32)
    out = np.full((n_q, topk), -2, dtype=np.int32)
    width = cand_width(c, g, window, window_kind)
    cand = np.full((n_groups, width), -2, dtype=np.int32) if (want_cand and mode == REFINE) else None
    pq = np.zeros((n_groups, H, d), dtype=_code_dtype(fmt)) if want_proxy else None
    psc = np.zeros(n_groups, dtype=np.float32) if want_proxy else None
    pw = np.zeros((n_groups, H), dtype=np.float32) if want_proxy else None
    rc = lib().oracle_index_ex(FMT[fmt], H, d, _p(q), _p(qs), _p(w), n_q, int(p0), _p(k), _p(ks),
                               int(n_k), mode, g, c, topk, dense_below, int(window), int(window_kind),
                               int(agg), _p(sel), 0 if sel is None else len(sel),
                               _p(out), _p(cand), _p(pq), _p(psc), _p(pw))
    if rc != 0:
        raise ValueError("oracle_index rejected its arguments")
    res = {"idx": out}
    if cand is not None:
        res["cand"] = cand
    if want_proxy:
        res.update(pq=pq, psc=psc, pw=pw)
    return res


def layer_anchors(n_layers: int, stride: int) -> np.ndarray:
    """Anchor layers every `stride` layers from layer 0."""
    return (np.arange(n_layers) % stride == 0).astype(np.uint8)


def index_layers(fmt: str, layers, p0: int, n_k: int, *, mode: int, g: int = 1, c: int = 0, topk: int,
                 dense_below: int | None = None, stride: int | None = None, anchors=None):
    """PIVOT (or the dense indexer) composed with IndexCache over consecutive
    layers.  layers: a list of (q [n_q,H,d], q_scale, w, k, k_scale), one per
    layer (entries of non-anchor layers may be None).  Anchors: `anchors`
    (one flag per layer) or every `stride`-th layer from 0.  Returns one
    [n_q, topk] index array per layer."""
    n_layers = len(layers)
    anc = layer_anchors(n_layers, stride) if anchors is None else np.asarray(anchors, dtype=np.uint8)
    if dense_below is None:
        dense_below = c if mode != DENSE else 0
    ref = next(L for L in layers if L is not None)
    n_q, H, d = ref[0].shape
    keep, qp, sp, wp, kp, ksp, outs = [], [], [], [], [], [], []
    for L in layers:
        if L is None:
            L = (None, None, None, None, None)
        q, qs, w, k, ks = L
        arrs = (_c(q, _code_dtype(fmt)), _c(qs, np.float32) if fmt == "fp8" else None, _c(w, np.float32),
                _c(k, _code_dtype(fmt)), _c(ks, np.float32) if fmt == "fp8" else None)
        keep.append(arrs)
        for lst, a in zip((qp, sp, wp, kp, ksp), arrs):
            lst.append(None if a is None else a.ctypes.data)
        outs.append(np.full((n_q, topk), -2, dtype=np.int32))
    P = ctypes.c_void_p
    arr = lambda xs: (P * n_layers)(*xs)  # noqa: E731
    anc = np.ascontiguousarray(anc)
    if anc.shape != (n_layers,):
        raise ValueError("one anchor flag per layer")
    rc = lib().oracle_index_layers(FMT[fmt], H, d, n_layers, _p(anc), arr(qp),
                                   arr(sp) if fmt == "fp8" else None, arr(wp), n_q, int(p0), arr(kp),
                                   arr(ksp) if fmt == "fp8" else None, int(n_k), mode, g, c, topk,
                                   dense_below, (P * n_layers)(*[o.ctypes.data for o in outs]))
    if rc != 0:
        raise ValueError("oracle_index_layers rejected its arguments")
    return outs
