"""MI355X (gfx950) PIVOT indexer: thin Python binding of libpivot.so.

Every function marshals torch tensors (device memory) and the current HIP
stream into the C ABI declared in include/pivot.h and calls it; all arithmetic
runs in the library's HIP kernels.  The binding allocates the workspace the
library asks for (the library itself never allocates).  Importing works without
a GPU; calling needs the built library and a gfx950 device, and fails loudly
otherwise.
"""
from __future__ import annotations

import ctypes
import os

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libpivot.so")

PIVOT_OK, PIVOT_ERR_INVALID_ARG, PIVOT_ERR_UNSUPPORTED, PIVOT_ERR_WORKSPACE, PIVOT_ERR_HIP = range(5)
PIVOT_DT_BF16, PIVOT_DT_FP8_E4M3 = 0, 1
PIVOT_REUSE, PIVOT_REFINE = 0, 1
PIVOT_DENSE = -1
PIVOT_MAX_KEYS = 1 << 27
PIVOT_NOALLOC_SCRATCH_BYTES = 64 << 20
PIVOT_WINDOW_SHARED, PIVOT_WINDOW_PER_QUERY = 0, 1
PIVOT_AGG_MEAN, PIVOT_AGG_FIRST, PIVOT_AGG_LAST = 0, 1, 2
PIVOT_REFINE_AUTO, PIVOT_REFINE_FUSED, PIVOT_REFINE_SPLIT = 0, 1, 2
H, D = 64, 128

EXPORTED = ["pivot_workspace_size", "pivot_dense_index", "pivot_group_index", "pivot_cand_width",
            "pivot_group_workspace_size", "pivot_group_index_opts", "pivot_dense_index_layout",
            "pivot_group_index_layout", "pivot_workspace_size_layout", "pivot_proxy_rows",
            "pivot_score_rows", "pivot_topk_rows", "pivot_topk_rows_workspace_size", "pivot_topk_rows_ws",
            "pivot_topk_rows_bf16",
            "pivot_encode_e4m3", "pivot_profile_begin", "pivot_profile_begin_kinds", "pivot_index_layers",
            "pivot_group_index_noalloc",
            "pivot_profile_end", "pivot_status_string", "pivot_last_error", "pivot_version"]
KERNELS = ["proxy", "score", "select", "refine", "fill", "lin", "copy"]


class PivotError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__(f"{where}: {status_string(status)} ({last_error()})")


class pivot_profile(ctypes.Structure):
    _fields_ = [("launches", ctypes.c_int64 * 7), ("total_ms", ctypes.c_double * 7)]


class pivot_args(ctypes.Structure):
    _fields_ = [
        ("dtype", ctypes.c_int32), ("heads", ctypes.c_int32), ("dim", ctypes.c_int32),
        ("batch", ctypes.c_int32), ("n_q", ctypes.c_int32),
        ("q_pos0", ctypes.POINTER(ctypes.c_int32)), ("n_k", ctypes.POINTER(ctypes.c_int32)),
        ("q", ctypes.c_void_p), ("q_scale", ctypes.c_void_p), ("w", ctypes.c_void_p),
        ("k", ctypes.c_void_p), ("k_scale", ctypes.c_void_p), ("k_seq_stride", ctypes.c_int64),
        ("topk", ctypes.c_int32), ("out_idx", ctypes.c_void_p),
        ("workspace", ctypes.c_void_p), ("workspace_bytes", ctypes.c_size_t),
        ("stream", ctypes.c_void_p),
    ]


class pivot_group_opts(ctypes.Structure):
    _fields_ = [
        ("mode", ctypes.c_int32), ("g", ctypes.c_int32), ("c", ctypes.c_int32),
        ("dense_below", ctypes.c_int32), ("window", ctypes.c_int32), ("window_kind", ctypes.c_int32),
        ("aggregate", ctypes.c_int32), ("out_cand", ctypes.c_void_p), ("refine_path", ctypes.c_int32),
    ]


class pivot_layout(ctypes.Structure):
    _fields_ = [
        ("cu_q", ctypes.POINTER(ctypes.c_int32)), ("block_table", ctypes.c_void_p),
        ("max_pages", ctypes.c_int32), ("page_size", ctypes.c_int32), ("pool_keys", ctypes.c_int64),
    ]


def make_layout(cu_q=None, block_table=None, page_size=0, pool_keys=0) -> pivot_layout:
    """cu_q: host ints [B+1] (packed query runs) or None; block_table: dev int32
    [B, max_pages] (paged keys) or None."""
    lo = pivot_layout()
    if cu_q is not None:
        lo._cu = (ctypes.c_int32 * len(cu_q))(*[int(v) for v in cu_q])
        lo.cu_q = ctypes.cast(lo._cu, ctypes.POINTER(ctypes.c_int32))
    if block_table is not None:
        if block_table.dtype != torch.int32 or block_table.dim() != 2 or not block_table.is_contiguous():
            raise ValueError("block_table must be a contiguous int32 [B, max_pages] tensor")
        lo.block_table = _ptr(block_table)
        lo.max_pages = block_table.shape[1]
        lo.page_size = int(page_size)
        lo.pool_keys = int(pool_keys)
        lo._bt = block_table
    return lo


def group_opts(mode, g, c, dense_below=-1, window=0, window_kind=PIVOT_WINDOW_SHARED,
               aggregate=PIVOT_AGG_MEAN, out_cand=None, refine_path=PIVOT_REFINE_AUTO) -> pivot_group_opts:
    o = pivot_group_opts()
    o.mode, o.g, o.c, o.dense_below = int(mode), int(g), int(c), int(dense_below)
    o.window, o.window_kind, o.aggregate = int(window), int(window_kind), int(aggregate)
    o.out_cand = _ptr(out_cand)
    o.refine_path = int(refine_path)
    o._keep = out_cand
    return o


_lib = None


def lib():
    """Load libpivot.so (built by __graft_entry__.build() / paper_2607_24593_amd.build)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"HIP library missing: {LIB_PATH}; build it with paper_2607_24593_amd.build")
        L = ctypes.CDLL(LIB_PATH)
        A = ctypes.POINTER(pivot_args)
        I32, I64, P = ctypes.c_int32, ctypes.c_int64, ctypes.c_void_p
        L.pivot_workspace_size.restype = ctypes.c_size_t
        L.pivot_workspace_size.argtypes = [A, I32, I32, I32]
        L.pivot_dense_index.restype = I32
        L.pivot_dense_index.argtypes = [A]
        L.pivot_group_index.restype = I32
        L.pivot_group_index.argtypes = [A, I32, I32, I32, I32, P]
        O = ctypes.POINTER(pivot_group_opts)
        L.pivot_cand_width.restype = I32
        L.pivot_cand_width.argtypes = [O]
        L.pivot_group_workspace_size.restype = ctypes.c_size_t
        L.pivot_group_workspace_size.argtypes = [A, O]
        L.pivot_group_index_opts.restype = I32
        L.pivot_group_index_opts.argtypes = [A, O]
        Lo = ctypes.POINTER(pivot_layout)
        L.pivot_dense_index_layout.restype = I32
        L.pivot_dense_index_layout.argtypes = [A, Lo]
        L.pivot_group_index_layout.restype = I32
        L.pivot_group_index_layout.argtypes = [A, Lo, O]
        L.pivot_workspace_size_layout.restype = ctypes.c_size_t
        L.pivot_workspace_size_layout.argtypes = [A, Lo, O]
        L.pivot_group_index_noalloc.restype = I32
        L.pivot_group_index_noalloc.argtypes = [A, O]
        L.pivot_index_layers.restype = I32
        L.pivot_index_layers.argtypes = [A, I32, I32, P, O]
        L.pivot_proxy_rows.restype = I32
        L.pivot_proxy_rows.argtypes = [I32, I32, I32, I32, I32, P, P, P, P, P, P, P]
        L.pivot_score_rows.restype = I32
        L.pivot_score_rows.argtypes = [I32, I32, I32, I32, P, P, P, P, P, I64, I32, P, I64, P, ctypes.c_size_t, P]
        L.pivot_topk_rows.restype = I32
        L.pivot_topk_rows.argtypes = [I32, P, I64, I64, I32, I32, P, P]
        L.pivot_topk_rows_bf16.restype = I32
        L.pivot_topk_rows_bf16.argtypes = [I32, P, I64, I64, I32, I32, P, P]
        L.pivot_topk_rows_workspace_size.restype = ctypes.c_size_t
        L.pivot_topk_rows_workspace_size.argtypes = [I32]
        L.pivot_topk_rows_ws.restype = I32
        L.pivot_topk_rows_ws.argtypes = [I32, P, I64, I64, I32, I32, P, P, ctypes.c_size_t, P]
        L.pivot_encode_e4m3.restype = I32
        L.pivot_encode_e4m3.argtypes = [P, P, I64, P]
        L.pivot_profile_begin.restype = I32
        L.pivot_profile_begin.argtypes = []
        L.pivot_profile_begin_kinds.restype = I32
        L.pivot_profile_begin_kinds.argtypes = [ctypes.c_uint32]
        L.pivot_profile_end.restype = I32
        L.pivot_profile_end.argtypes = [ctypes.POINTER(pivot_profile)]
        L.pivot_status_string.restype = ctypes.c_char_p
        L.pivot_status_string.argtypes = [I32]
        L.pivot_last_error.restype = ctypes.c_char_p
        L.pivot_last_error.argtypes = []
        L.pivot_version.restype = ctypes.c_char_p
        L.pivot_version.argtypes = []
        _lib = L
    return _lib


def status_string(status: int) -> str:
    return lib().pivot_status_string(int(status)).decode()


def last_error() -> str:
    return lib().pivot_last_error().decode()


def version() -> str:
    return lib().pivot_version().decode()


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream):
    if stream is None:
        return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    if isinstance(stream, torch.cuda.Stream):
        return ctypes.c_void_p(stream.cuda_stream)
    return ctypes.c_void_p(int(stream))


def _dtype_code(q) -> int:
    if q.element_size() == 1:
        return PIVOT_DT_FP8_E4M3
    if q.element_size() == 2:
        return PIVOT_DT_BF16
    raise ValueError("q must hold fp8 codes (1 byte) or bf16 (2 bytes)")


def _check(status: int, where: str):
    if status != PIVOT_OK:
        raise PivotError(status, where)


_WS = {}


def _torch_stream(stream, device):
    """The torch stream object for a call's `stream` argument (None: current)."""
    dev = torch.device(device)
    if stream is None:
        return torch.cuda.current_stream(dev)
    if isinstance(stream, torch.cuda.Stream):
        return stream
    return torch.cuda.ExternalStream(int(stream), device=dev)


def workspace(nbytes: int, device, stream=None) -> torch.Tensor:
    """A cached device buffer of at least nbytes (256-byte aligned by torch) for
    calls on `stream` (None: the current stream).  There is one buffer per
    (device, stream): calls on one stream run in order, so they may share it,
    while calls on two streams would write one buffer concurrently.  The buffer
    is allocated with that stream current, so torch's caching allocator orders
    its reuse after the work already queued on the stream when it is replaced."""
    dev = torch.device(device)
    s = _torch_stream(stream, dev)
    key = (dev.type, dev.index, s.cuda_stream)
    buf = _WS.get(key)
    if buf is None or buf.numel() < nbytes:
        _WS.pop(key, None)
        with torch.cuda.stream(s):
            buf = torch.empty(max(nbytes, 256), dtype=torch.uint8, device=dev)
        _WS[key] = buf
    return buf


def make_args(q, q_scale, w, k, k_scale, q_pos0, n_k, topk, out_idx, k_seq_stride=None, stream=None):
    """pivot_args for q [B, n_q, H, d] (or [n_q, H, d]), w [B, n_q, H], k [B, S, d]
    (or [S, d]); q_pos0 / n_k are ints or per-sequence lists."""
    if q.dim() == 3:
        q = q.unsqueeze(0)
        w = w.unsqueeze(0)
        q_scale = None if q_scale is None else q_scale.unsqueeze(0)
    if k.dim() == 2:
        k = k.unsqueeze(0)
        k_scale = None if k_scale is None else k_scale.unsqueeze(0)
    B, n_q = q.shape[0], q.shape[1]
    pos = [int(q_pos0)] * B if isinstance(q_pos0, int) else [int(v) for v in q_pos0]
    nk = [int(n_k)] * B if isinstance(n_k, int) else [int(v) for v in n_k]
    for t in (q, w, k, out_idx) + tuple(x for x in (q_scale, k_scale) if x is not None):
        if not t.is_contiguous():
            raise ValueError("tensors must be contiguous")
    a = pivot_args()
    a.dtype = _dtype_code(q)
    a.heads, a.dim = q.shape[2], q.shape[3]
    a.batch, a.n_q = B, n_q
    a._pos = (ctypes.c_int32 * B)(*pos)
    a._nk = (ctypes.c_int32 * B)(*nk)
    a.q_pos0 = ctypes.cast(a._pos, ctypes.POINTER(ctypes.c_int32))
    a.n_k = ctypes.cast(a._nk, ctypes.POINTER(ctypes.c_int32))
    a.q, a.q_scale, a.w = _ptr(q), _ptr(q_scale), _ptr(w)
    a.k, a.k_scale = _ptr(k), _ptr(k_scale)
    a.k_seq_stride = k.shape[1] if k_seq_stride is None else int(k_seq_stride)
    a.topk = int(topk)
    a.out_idx = _ptr(out_idx)
    a.stream = _stream(stream)
    a._keep = (q, q_scale, w, k, k_scale, out_idx)
    return a


def pivot_workspace_size(a: pivot_args, mode: int = PIVOT_DENSE, g: int = 1, c: int = 0) -> int:
    return int(lib().pivot_workspace_size(ctypes.byref(a), int(mode), int(g), int(c)))


def _attach_workspace(a, mode, g, c, ws, device, stream=None):
    need = pivot_workspace_size(a, mode, g, c)
    if need == 0 and a.n_q > 0:
        return  # invalid shapes: the entry point reports the reason
    buf = ws if ws is not None else workspace(need, device, stream)
    a.workspace = _ptr(buf)
    a.workspace_bytes = buf.numel() * buf.element_size()
    a._ws = buf


def pivot_dense_index(q, q_scale, w, k, k_scale, q_pos0, n_k, topk, out=None, ws=None, stream=None):
    """Dense lightning indexer: returns int32 [B, n_q, topk] (or [n_q, topk])."""
    squeeze = q.dim() == 3
    shape = (q.shape[0], topk) if squeeze else (q.shape[0], q.shape[1], topk)
    out = torch.empty(shape, dtype=torch.int32, device=q.device) if out is None else out
    a = make_args(q, q_scale, w, k, k_scale, q_pos0, n_k, topk, out, stream=stream)
    _attach_workspace(a, PIVOT_DENSE, 1, 0, ws, q.device, stream)
    _check(lib().pivot_dense_index(ctypes.byref(a)), "pivot_dense_index")
    return out


def pivot_group_index(q, q_scale, w, k, k_scale, q_pos0, n_k, topk, mode, g, c, dense_below=-1,
                      out=None, out_cand=None, ws=None, stream=None):
    """PIVOT Reuse / Refine (Algorithm 1): returns int32 [B, n_q, topk] (or [n_q, topk])."""
    squeeze = q.dim() == 3
    shape = (q.shape[0], topk) if squeeze else (q.shape[0], q.shape[1], topk)
    out = torch.empty(shape, dtype=torch.int32, device=q.device) if out is None else out
    a = make_args(q, q_scale, w, k, k_scale, q_pos0, n_k, topk, out, stream=stream)
    # sized for this call's guardrail (pivot_workspace_size assumes dense_below = c)
    o = group_opts(mode, g, c, dense_below)
    _attach(a, pivot_group_workspace_size(a, o), ws, q.device, stream)
    _check(lib().pivot_group_index(ctypes.byref(a), int(mode), int(g), int(c), int(dense_below),
                                   _ptr(out_cand)), "pivot_group_index")
    return out


def pivot_cand_width(o: pivot_group_opts) -> int:
    return int(lib().pivot_cand_width(ctypes.byref(o)))


def pivot_group_workspace_size(a: pivot_args, o: pivot_group_opts) -> int:
    return int(lib().pivot_group_workspace_size(ctypes.byref(a), ctypes.byref(o)))


def pivot_group_index_opts(q, q_scale, w, k, k_scale, q_pos0, n_k, topk, mode, g, c, dense_below=-1,
                           window=0, window_kind=PIVOT_WINDOW_SHARED, aggregate=PIVOT_AGG_MEAN,
                           out=None, out_cand=None, ws=None, stream=None, refine_path=PIVOT_REFINE_AUTO):
    """PIVOT with App. B's local window and the first / last proxy aggregation;
    out_cand, when given, is int32 [B, n_groups, pivot_cand_width(opts)];
    refine_path: PIVOT_REFINE_AUTO / _FUSED / _SPLIT (same results)."""
    squeeze = q.dim() == 3
    shape = (q.shape[0], topk) if squeeze else (q.shape[0], q.shape[1], topk)
    out = torch.empty(shape, dtype=torch.int32, device=q.device) if out is None else out
    a = make_args(q, q_scale, w, k, k_scale, q_pos0, n_k, topk, out, stream=stream)
    o = group_opts(mode, g, c, dense_below, window, window_kind, aggregate, out_cand, refine_path)
    _attach(a, pivot_group_workspace_size(a, o), ws, q.device, stream)
    _check(lib().pivot_group_index_opts(ctypes.byref(a), ctypes.byref(o)), "pivot_group_index_opts")
    return out


def pivot_index_layers(layers, q_pos0, n_k, topk, *, stride=1, anchors=None, mode=None, g=1, c=0, dense_below=-1,
                       window=0, window_kind=PIVOT_WINDOW_SHARED, aggregate=PIVOT_AGG_MEAN, outs=None, ws=None,
                       stream=None):
    """PIVOT (mode PIVOT_REUSE / PIVOT_REFINE) or the dense indexer (mode None)
    composed with IndexCache over consecutive layers.  layers: one (q, q_scale,
    w, k, k_scale) per layer, shaped as for pivot_dense_index; a non-anchor
    layer's entry may be None (its inputs are not read).  Anchors: `anchors`
    (one flag per layer) or every `stride`-th layer from 0.  Returns one int32
    index tensor per layer (or fills `outs`)."""
    n_layers = len(layers)
    ref = layers[0]
    if ref is None:
        raise ValueError("layer 0 is an anchor and needs its inputs")
    q0 = ref[0]
    squeeze = q0.dim() == 3
    shape = (q0.shape[0], topk) if squeeze else (q0.shape[0], q0.shape[1], topk)
    if outs is None:
        outs = [torch.empty(shape, dtype=torch.int32, device=q0.device) for _ in range(n_layers)]
    arr = (pivot_args * n_layers)()
    keep = []
    for l, L in enumerate(layers):
        src = ref if L is None else L
        a = make_args(*src, q_pos0, n_k, topk, outs[l], stream=stream)
        if L is None:
            a.q = a.q_scale = a.w = a.k = a.k_scale = None
        arr[l] = a
        keep.append(a)
    o = None if mode is None else group_opts(mode, g, c, dense_below, window, window_kind, aggregate)
    need = int(lib().pivot_workspace_size_layout(ctypes.byref(arr[0]), None, None if o is None else ctypes.byref(o)))
    if need > 0:
        buf = ws if ws is not None else workspace(need, q0.device, stream)
        arr[0].workspace = _ptr(buf)
        arr[0].workspace_bytes = buf.numel() * buf.element_size()
        keep.append(buf)
    anc = None
    if anchors is not None:
        anc = (ctypes.c_uint8 * n_layers)(*[1 if v else 0 for v in anchors])
    _check(lib().pivot_index_layers(arr, n_layers, int(stride), anc, None if o is None else ctypes.byref(o)),
           "pivot_index_layers")
    return outs


def make_args_batch(q, q_scale, w, k, k_scale, q_pos0, n_k, topk, out_idx, stream=None):
    """pivot_args for packed query rows q [rows, H, d] / w [rows, H] of len(q_pos0)
    sequences (their runs given by a layout's cu_q) and keys k: a page pool
    [keys, d] (with a layout's block_table), or contiguous sequences [B, S, d]."""
    for t in (q, w, k, out_idx) + tuple(x for x in (q_scale, k_scale) if x is not None):
        if not t.is_contiguous():
            raise ValueError("tensors must be contiguous")
    B = len(q_pos0)
    a = pivot_args()
    a.dtype = _dtype_code(q)
    a.heads, a.dim = q.shape[1], q.shape[2]
    a.batch, a.n_q = B, 0
    a._pos = (ctypes.c_int32 * B)(*[int(v) for v in q_pos0])
    a._nk = (ctypes.c_int32 * B)(*[int(v) for v in n_k])
    a.q_pos0 = ctypes.cast(a._pos, ctypes.POINTER(ctypes.c_int32))
    a.n_k = ctypes.cast(a._nk, ctypes.POINTER(ctypes.c_int32))
    a.q, a.q_scale, a.w = _ptr(q), _ptr(q_scale), _ptr(w)
    a.k, a.k_scale = _ptr(k), _ptr(k_scale)
    a.k_seq_stride = k.shape[1] if k.dim() == 3 else k.shape[0]  # [B, S, d]: contiguous sequences of S keys
    a.topk = int(topk)
    a.out_idx = _ptr(out_idx)
    a.stream = _stream(stream)
    a._keep = (q, q_scale, w, k, k_scale, out_idx)
    return a


def pivot_workspace_size_layout(a: pivot_args, lo: pivot_layout, o=None) -> int:
    return int(lib().pivot_workspace_size_layout(ctypes.byref(a), ctypes.byref(lo),
                                                 None if o is None else ctypes.byref(o)))


def _attach(a, need, ws, device, stream=None):
    if need > 0:
        buf = ws if ws is not None else workspace(need, device, stream)
        a.workspace = _ptr(buf)
        a.workspace_bytes = buf.numel() * buf.element_size()
        a._ws = buf


def pivot_dense_index_layout(q, q_scale, w, k, k_scale, q_pos0, n_k, topk, layout, out=None, ws=None,
                             stream=None):
    """Dense index of packed query runs (layout.cu_q) over contiguous or paged keys:
    returns int32 [rows, topk]."""
    out = torch.empty((q.shape[0], topk), dtype=torch.int32, device=q.device) if out is None else out
    a = make_args_batch(q, q_scale, w, k, k_scale, q_pos0, n_k, topk, out, stream=stream)
    _attach(a, pivot_workspace_size_layout(a, layout), ws, q.device, stream)
    _check(lib().pivot_dense_index_layout(ctypes.byref(a), ctypes.byref(layout)), "pivot_dense_index_layout")
    return out


def pivot_group_index_layout(q, q_scale, w, k, k_scale, q_pos0, n_k, topk, layout, mode, g, c, dense_below=-1,
                             window=0, window_kind=PIVOT_WINDOW_SHARED, aggregate=PIVOT_AGG_MEAN, out=None,
                             out_cand=None, ws=None, stream=None, refine_path=PIVOT_REFINE_AUTO):
    """PIVOT over packed query runs (groups restart at every run) and contiguous or
    paged keys: returns int32 [rows, topk]."""
    out = torch.empty((q.shape[0], topk), dtype=torch.int32, device=q.device) if out is None else out
    a = make_args_batch(q, q_scale, w, k, k_scale, q_pos0, n_k, topk, out, stream=stream)
    o = group_opts(mode, g, c, dense_below, window, window_kind, aggregate, out_cand, refine_path)
    _attach(a, pivot_workspace_size_layout(a, layout, o), ws, q.device, stream)
    _check(lib().pivot_group_index_layout(ctypes.byref(a), ctypes.byref(layout), ctypes.byref(o)),
           "pivot_group_index_layout")
    return out


def pivot_proxy_rows(q, q_scale, w, g, stream=None):
    """Eq. 4 proxies of runs of g rows of one sequence: (q_proxy, scale, w_proxy)."""
    n_q = q.shape[0]
    ng = (n_q + g - 1) // g
    pq = torch.empty((ng,) + tuple(q.shape[1:]), dtype=q.dtype, device=q.device)
    ps = torch.empty(ng, dtype=torch.float32, device=q.device)
    pw = torch.empty((ng, w.shape[1]), dtype=torch.float32, device=q.device)
    _check(lib().pivot_proxy_rows(_dtype_code(q), q.shape[1], q.shape[2], n_q, int(g), _ptr(q), _ptr(q_scale),
                                  _ptr(w), _ptr(pq), _ptr(ps), _ptr(pw), _stream(stream)), "pivot_proxy_rows")
    return pq, ps, pw


def score_rows_workspace(n_rows: int) -> int:
    """PIVOT_SCORE_ROWS_WORKSPACE of include/pivot.h."""
    return (n_rows * 512 + 255) // 256 * 256 + n_rows * 16


def pivot_score_rows(q, q_scale, w, k, k_scale, lim0, lim_step, ld=None, out=None, stream=None):
    """Scores of rows q [n, H, d] over keys 0 .. lim0 + r * lim_step: fp32 [n, ld]."""
    n = q.shape[0]
    lim_max = lim0 + (n - 1) * lim_step
    ld = lim_max + 1 if ld is None else ld
    out = torch.full((n, ld), float("nan"), dtype=torch.float32, device=q.device) if out is None else out
    nbytes = score_rows_workspace(n) if _dtype_code(q) == PIVOT_DT_FP8_E4M3 else 0
    ws = workspace(nbytes, q.device, stream) if nbytes else None
    _check(lib().pivot_score_rows(_dtype_code(q), q.shape[1], q.shape[2], n, _ptr(q), _ptr(q_scale), _ptr(w),
                                  _ptr(k), _ptr(k_scale), int(lim0), int(lim_step), _ptr(out), int(ld), _ptr(ws),
                                  nbytes, _stream(stream)), "pivot_score_rows")
    return out


def pivot_topk_rows(scores, n0, n_step, m, out=None, stream=None):
    """Top-m positions of rows of scores [n, ld] with n0 + r * n_step valid entries."""
    n, ld = scores.shape
    out = torch.empty((n, m), dtype=torch.int32, device=scores.device) if out is None else out
    _check(lib().pivot_topk_rows(n, _ptr(scores), ld, int(n0), int(n_step), int(m), _ptr(out), _stream(stream)),
           "pivot_topk_rows")
    return out


def pivot_topk_rows_bf16(scores, n0, n_step, m, out=None, stream=None):
    """pivot_topk_rows over bf16 score rows (an int16 / bfloat16 tensor [n, ld] of bf16 bits)."""
    n, ld = scores.shape
    if scores.element_size() != 2:
        raise ValueError("bf16 rows hold 2-byte scores")
    out = torch.empty((n, m), dtype=torch.int32, device=scores.device) if out is None else out
    _check(lib().pivot_topk_rows_bf16(n, _ptr(scores), ld, int(n0), int(n_step), int(m), _ptr(out),
                                      _stream(stream)), "pivot_topk_rows_bf16")
    return out


def pivot_topk_rows_workspace_size(n_rows: int) -> int:
    return int(lib().pivot_topk_rows_workspace_size(int(n_rows)))


def pivot_topk_rows_ws(scores, n0, n_step, m, out=None, ws=None, stream=None):
    """pivot_topk_rows with a workspace (few long rows are split over several workgroups)."""
    n, ld = scores.shape
    out = torch.empty((n, m), dtype=torch.int32, device=scores.device) if out is None else out
    need = pivot_topk_rows_workspace_size(n)
    if ws is None and need > 0:
        ws = workspace(need, scores.device, stream)
    nbytes = 0 if ws is None else ws.numel() * ws.element_size()
    _check(lib().pivot_topk_rows_ws(n, _ptr(scores), ld, int(n0), int(n_step), int(m), _ptr(out), _ptr(ws),
                                    nbytes, _stream(stream)), "pivot_topk_rows_ws")
    return out


def pivot_profile_begin(kinds=None):
    """Time every kernel kind, or only the names in `kinds` (from KERNELS)."""
    if kinds is None:
        _check(lib().pivot_profile_begin(), "pivot_profile_begin")
        return
    mask = 0
    for name in kinds:
        mask |= 1 << KERNELS.index(name)
    _check(lib().pivot_profile_begin_kinds(mask), "pivot_profile_begin_kinds")


def pivot_profile_end() -> dict:
    """{kernel: (launches, total_ms)} since pivot_profile_begin()."""
    p = pivot_profile()
    _check(lib().pivot_profile_end(ctypes.byref(p)), "pivot_profile_end")
    return {name: (int(p.launches[i]), float(p.total_ms[i])) for i, name in enumerate(KERNELS)}


def pivot_encode_e4m3(x, out=None, stream=None):
    out = torch.empty(x.shape, dtype=torch.uint8, device=x.device) if out is None else out
    _check(lib().pivot_encode_e4m3(_ptr(x), _ptr(out), x.numel(), _stream(stream)), "pivot_encode_e4m3")
    return out
