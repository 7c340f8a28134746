#!/usr/bin/env python
"""Benchmark of the PIVOT indexer hot path on one MI355X (gfx950).

One step = one PIVOT-Refine pass (g=4, c=4096, k=2048) over a whole 131072-token
fp8 prefill, issued as 16 calls of 8192 queries against their full causal
prefix: grouping and guardrail planning, proxy aggregation, proxy scan, proxy
top-c, and the per-member gather / re-score / top-k.  Inputs are synthetic
(workload.gen, the 128K prefill recipe) and resident in HBM before timing.

Reported besides the headline queries/s: the dense indexer and PIVOT-Reuse on
the same prefill (speedup), a group-size sweep, Refine with App. B's local
window (W=4), the bf16 scoring kernel's MFMA fraction (the 128K prefill in bf16), MTP decode (32 x 131072 cached keys, g=2, also with the
per-query window; each call launched eagerly and replayed from a captured HIP graph), the batch layouts (paged decode keys, a packed batch of
four prefill requests), per-kernel times from HIP events recorded around each launch
inside the timed steps, the roofline fraction of the dominant kernel, and the
CPU oracle timed on a sample of the same workload.

    python bench.py [--gpus 1] [--steps K] [--warmup W]
"""
from __future__ import annotations

import argparse
import gc
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK = {"fp8": 5000.0, "bf16": 2500.0}  # dense MFMA TFLOP/s (MI355X)
HBM_PEAK = 8000.0                        # GB/s
FLOP_PER_PAIR = 2 * 64 * 128             # one (row, key) score: 64 heads x 128-dim dot


def log(*a):
    print("[bench]", *a, file=sys.stderr, flush=True)


# ---------------------------------------------------------------- accounting
def plan_chunk(p0, n_q, g, c, mode):
    """Rows of one call as the library plans them (Algorithm 1 guardrail at c)."""
    ng = (n_q + g - 1) // g
    if mode == "dense":
        return n_q, []
    gap = c - p0
    J = 0 if gap <= 0 else min(-(-gap // g), ng)
    dense_rows = min(J * g, n_q)
    proxies = [(p0 + j * g, min(g, n_q - j * g)) for j in range(J, ng)]
    return dense_rows, proxies


LIN_ROW_BYTES = 4 * 128 + 4 * 4


def units(chunks, mode, g, c, topk, eb_q=1, eb_k=1):
    """Algorithmic work per pass: score pairs, select bytes, refine bytes and flops, proxy bytes.
    The library stores score rows as bf16 for fp8 inputs (2 bytes per score
    read by the select) and as fp32 for bf16 inputs."""
    row_q = 64 * 128 * eb_q + 4 + 4 * 64
    eb_s = 2 if eb_q == 1 else 4
    pairs = sel_bytes = ref_bytes = ref_flops = prox_bytes = 0
    for p0, n_q in chunks:
        dense_rows, proxies = plan_chunk(p0, n_q, g, c, mode)
        dp = sum(p0 + i + 1 for i in range(dense_rows))
        pairs += dp
        sel_bytes += eb_s * dp + 4 * topk * dense_rows
        for t0, gs in proxies:
            n = t0 + 1
            pairs += n
            m = topk if mode == "reuse" else c
            fan = gs if mode == "reuse" else 1
            sel_bytes += eb_s * n + 4 * min(m, n) * fan
            prox_bytes += (gs + 1) * row_q if gs > 1 else 0
            if eb_q == 1:  # fp8: the epilogue's linear terms (4 x 128 codes + 4 scales) of the
                # proxy, and for Refine of the members, written by the proxy kernel
                prox_bytes += LIN_ROW_BYTES * (1 + (gs if mode == "refine" else 0))
            if mode == "refine":
                nc = min(c, n)
                ref_bytes += nc * (128 * eb_k + 4) + 4 * nc + gs * row_q + 4 * gs * topk
                ref_flops += gs * nc * FLOP_PER_PAIR
    return dict(pairs=pairs, score_flops=pairs * FLOP_PER_PAIR, select_bytes=sel_bytes,
                refine_bytes=ref_bytes, refine_flops=ref_flops, proxy_bytes=prox_bytes)


# ---------------------------------------------------------------- runs
class Prefill:
    def __init__(self, wl, threads, score_tile_mb=None):
        import torch
        from workload.gen import make
        t = time.time()
        x = make(wl, threads=threads)
        log(f"generated {wl.name} in {time.time() - t:.1f}s")
        self.wl, self.x = wl, x
        d = lambda a: None if a is None else torch.from_numpy(a.view("int16") if a.dtype.name == "uint16" else a).cuda()  # noqa
        self.q, self.qs, self.w, self.k, self.ks = d(x.q), d(x.q_scale), d(x.w), d(x.k), d(x.k_scale)
        L = wl.L
        self.chunks = [(p0, min(wl.chunk, L - p0)) for p0 in range(0, L, wl.chunk)]
        self.out = torch.empty((L, wl.topk), dtype=torch.int32, device="cuda")
        import paper_2607_24593_amd as pv
        self.pv = pv
        p0, n = self.chunks[-1]
        need = 0
        for g in wl.g:
            a = pv.make_args(self.q[p0:p0 + n], self.qs[p0:p0 + n] if self.qs is not None else None,
                             self.w[p0:p0 + n], self.k[:p0 + n], None if self.ks is None else self.ks[:p0 + n],
                             p0, p0 + n, wl.topk, self.out[p0:p0 + n])
            for mode in (pv.PIVOT_DENSE, pv.PIVOT_REUSE, pv.PIVOT_REFINE):
                need = max(need, pv.pivot_workspace_size(a, mode, g, wl.c))
        if score_tile_mb is not None:
            # the library tiles score rows to fit the workspace: replace the
            # default ~1 GiB score tile by the requested size
            need = need - (1 << 30) + int(score_tile_mb) * (1 << 20)
        self.ws = torch.empty(need, dtype=torch.uint8, device="cuda")
        log(f"workspace {need / 2**30:.2f} GiB")

    def run(self, mode, g, window=0):
        pv, wl = self.pv, self.wl
        for p0, n in self.chunks:
            sl = slice(p0, p0 + n)
            args = (self.q[sl], None if self.qs is None else self.qs[sl], self.w[sl], self.k[:p0 + n],
                    None if self.ks is None else self.ks[:p0 + n], p0, p0 + n, wl.topk)
            if mode == "dense":
                pv.pivot_dense_index(*args, out=self.out[sl], ws=self.ws)
            elif window:  # App. B's prefill window (Refine)
                pv.pivot_group_index_opts(*args, mode=pv.PIVOT_REFINE, g=g, c=wl.c, window=window,
                                          window_kind=pv.PIVOT_WINDOW_SHARED, out=self.out[sl], ws=self.ws)
            else:
                pv.pivot_group_index(*args, mode=pv.PIVOT_REUSE if mode == "reuse" else pv.PIVOT_REFINE,
                                     g=g, c=wl.c, out=self.out[sl], ws=self.ws)


def run_two_streams(pf, mode, g):
    """One pass with the chunk calls alternating over two streams, each with
    its own workspace: the chunks are independent calls (disjoint queries and
    outputs, read-only keys), so one call's kernels fill the GPU while the
    other's launch ramps or drains.  Every stream keeps the default priority."""
    import torch
    pv, wl = pf.pv, pf.wl
    if not hasattr(pf, "second"):  # freed with pf
        pf.second = (torch.cuda.Stream(), torch.empty_like(pf.ws))
    s1, (s2, ws2) = torch.cuda.current_stream(), pf.second
    s2.wait_stream(s1)
    for i, (p0, n) in enumerate(pf.chunks):
        s, ws = (s1, pf.ws) if i % 2 == 0 else (s2, ws2)
        sl = slice(p0, p0 + n)
        args = (pf.q[sl], None if pf.qs is None else pf.qs[sl], pf.w[sl], pf.k[:p0 + n],
                None if pf.ks is None else pf.ks[:p0 + n], p0, p0 + n, wl.topk)
        with torch.cuda.stream(s):
            if mode == "dense":
                pv.pivot_dense_index(*args, out=pf.out[sl], ws=ws, stream=s)
            else:
                pv.pivot_group_index(*args, mode=pv.PIVOT_REUSE if mode == "reuse" else pv.PIVOT_REFINE, g=g,
                                     c=wl.c, out=pf.out[sl], ws=ws, stream=s)
    s1.wait_stream(s2)


class no_gc:
    """Python's cyclic collector paused around a timed loop: a full collection
    over the interpreter's heap (torch, the workload's arrays) takes tens of ms
    on the host and would show up as an idle GPU inside the timed region."""

    def __enter__(self):
        gc.collect()
        gc.disable()

    def __exit__(self, *exc):
        gc.enable()


def timed(fn, reps):
    import torch
    torch.cuda.synchronize()
    with no_gc():
        t = time.perf_counter()
        for _ in range(reps):
            fn()
        torch.cuda.synchronize()
        return (time.perf_counter() - t) / reps


def kernel_roofline(prof, u, K, dtype):
    """Per-kernel times of K passes (pivot_profile_end()) against the algorithmic
    units of one pass (units()): the dominant kernel and its roofline."""
    kern = {}
    for name, (n, ms) in prof.items():
        if n == 0:
            continue
        e = {"launches_per_pass": n / K, "ms_per_pass": ms / K, "avg_launch_ms": ms / n}
        if name == "score":
            e.update(bound="mfma", achieved=u["score_flops"] * K / (ms * 1e-3) / 1e12, unit="TFLOP/s",
                     peak=PEAK[dtype])
        elif name == "select":
            e.update(bound="hbm", achieved=u["select_bytes"] * K / (ms * 1e-3) / 1e9, unit="GB/s", peak=HBM_PEAK)
        elif name == "refine" and u["refine_bytes"]:
            e.update(bound="hbm", achieved=u["refine_bytes"] * K / (ms * 1e-3) / 1e9, unit="GB/s", peak=HBM_PEAK,
                     mfma_TFLOPs=u["refine_flops"] * K / (ms * 1e-3) / 1e12)
        elif name == "proxy" and u["proxy_bytes"]:
            e.update(bound="hbm", achieved=u["proxy_bytes"] * K / (ms * 1e-3) / 1e9, unit="GB/s", peak=HBM_PEAK)
        if "achieved" in e:
            e["frac"] = e["achieved"] / e["peak"]
        kern[name] = e
    dom = max(kern, key=lambda n: kern[n]["ms_per_pass"])
    d = kern[dom]
    return kern, {"kernel": dom, "bound": d.get("bound"), "achieved": d.get("achieved"), "peak": d.get("peak"),
                  "unit": d.get("unit"), "frac": d.get("frac")}


def workload_bench(name, modes, reps):
    """A named workload timed pass by pass (all its chunks, inputs resident):
    queries/s and speedup over the dense pass per mode, and each mode's
    per-kernel breakdown from a separate profiled pass with the dominant
    kernel's roofline."""
    import torch
    from workload.gen import WORKLOADS
    wl = WORKLOADS[name]
    pf = Prefill(wl, threads=16)
    g = wl.g[0]
    eb = 1 if wl.dtype == "fp8" else 2
    res = {"workload": name, "L": wl.L, "chunk": wl.chunk, "g": g, "c": wl.c, "topk": wl.topk, "dtype": wl.dtype}
    for mode in modes:
        fn = lambda: pf.run(mode, g)  # noqa: E731
        fn()
        sec = timed(fn, reps)
        with no_gc():
            pf.pv.pivot_profile_begin()
            fn()
            torch.cuda.synchronize()
            prof = pf.pv.pivot_profile_end()
        u = units(pf.chunks, mode, g if mode != "dense" else 1, wl.c, wl.topk, eb, eb)
        kern, roof = kernel_roofline(prof, u, 1, wl.dtype)
        res[mode] = {"ms_per_pass": sec * 1e3, "queries_per_s": wl.L / sec, "roofline": roof, "kernels": kern}
        log(f"{name} {mode}: {sec * 1e3:.2f} ms ({wl.L / sec:.3g} q/s); dominant {roof['kernel']} "
            f"frac {roof['frac']}")
    for mode in modes:
        if mode != "dense" and "dense" in res:
            res[mode]["speedup_vs_dense"] = res["dense"]["ms_per_pass"] / res[mode]["ms_per_pass"]
    del pf
    gc.collect()
    torch.cuda.empty_cache()
    return res


def indexcache_bench(pf, g, reps, n_layers=4, stride=2):
    """PIVOT-Refine composed with IndexCache (Sec. 5.1, Table 1 +IC) over
    n_layers layers of the 128K prefill: anchors every `stride` layers run
    PIVOT on inputs of their own (a second layer of inputs from another seed),
    followers take the anchor's sets.  Against every layer running PIVOT
    (stride 1).  Layer-queries/s counts every layer's queries."""
    import torch
    from workload.gen import make_prefill
    pv, wl = pf.pv, pf.wl
    t = time.time()
    xb = make_prefill(wl.L, wl.dtype, seed=0x1C0 + 2, rho=0.9, threads=16)
    log(f"generated a second 128K layer in {time.time() - t:.1f}s")
    d = lambda a: torch.from_numpy(a).cuda()  # noqa: E731
    B = (d(xb.q), d(xb.q_scale), d(xb.w), d(xb.k), d(xb.k_scale))
    A = (pf.q, pf.qs, pf.w, pf.k, pf.ks)
    srcs = [A if (l // stride) % 2 == 0 else B for l in range(n_layers)]
    outs = [torch.empty((wl.L, wl.topk), dtype=torch.int32, device="cuda") for _ in range(n_layers)]

    def run(st):
        for p0, n in pf.chunks:
            sl = slice(p0, p0 + n)
            layers = []
            for l, (q, qs, w, k, ks) in enumerate(srcs):
                layers.append((q[sl], qs[sl], w[sl], k[:p0 + n], ks[:p0 + n]) if l % st == 0 else None)
            pv.pivot_index_layers(layers, p0, p0 + n, wl.topk, stride=st, mode=pv.PIVOT_REFINE, g=g, c=wl.c,
                                  outs=[o[sl] for o in outs], ws=pf.ws)
    res = {"layers": n_layers, "stride": stride, "mode": f"refine g={g} c={wl.c} k={wl.topk}",
           "workload": wl.name}
    for st in (stride, 1):
        run(st)
        sec = timed(lambda: run(st), reps)
        res[f"stride{st}"] = {"ms_per_pass": sec * 1e3, "layer_queries_per_s": n_layers * wl.L / sec}
        log(f"IndexCache {n_layers} layers stride {st}: {sec * 1e3:.2f} ms")
    res["speedup_vs_every_layer_pivot"] = res["stride1"]["ms_per_pass"] / res[f"stride{stride}"]["ms_per_pass"]
    return res


def decode_bench(reps):
    import torch
    import paper_2607_24593_amd as pv
    from workload.gen import WORKLOADS, make
    wl = WORKLOADS["decode-32x128k-fp8"]
    t = time.time()
    x = make(wl, threads=16)
    log(f"generated {wl.name} in {time.time() - t:.1f}s")
    B, L, g = wl.batch, wl.L, wl.g[0]
    d = lambda a: torch.from_numpy(a).cuda()  # noqa: E731
    q, qs, w, k, ks = d(x.q), d(x.q_scale), d(x.w), d(x.k), d(x.k_scale)
    pos, nk = [L - g] * B, [L] * B
    out = torch.empty((B, g, wl.topk), dtype=torch.int32, device="cuda")
    res = {}

    def call(mode, ws=None):
        if mode == "dense":
            return lambda: pv.pivot_dense_index(q, qs, w, k, ks, pos, nk, wl.topk, out=out, ws=ws)
        if mode == "refine_W4":  # App. B's per-query window, W = 4
            return lambda: pv.pivot_group_index_opts(q, qs, w, k, ks, pos, nk, wl.topk, mode=pv.PIVOT_REFINE, g=g,
                                                     c=wl.c, window=4, window_kind=pv.PIVOT_WINDOW_PER_QUERY,
                                                     out=out, ws=ws)
        m = pv.PIVOT_REUSE if mode == "reuse" else pv.PIVOT_REFINE
        return lambda: pv.pivot_group_index(q, qs, w, k, ks, pos, nk, wl.topk, mode=m, g=g, c=wl.c, out=out,
                                            ws=ws)

    modes = ("dense", "reuse", "refine", "refine_W4")
    for mode in modes:
        fn = call(mode)
        fn()
        sec = timed(fn, reps)
        res[mode] = {"us_per_step": sec * 1e6, "queries_per_s": B * g / sec}
    # the same calls replayed from a HIP graph captured once per mode (the
    # library makes no allocation, copy or memset inside a call, so a call
    # captures whole): the chain's launch gaps without host work per step
    ws = pv.workspace(0, q.device)  # the cached workspace, sized by the calls above
    for mode in modes:
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            call(mode, ws)()
        graph.replay()
        res[mode]["graph_us_per_step"] = timed(graph.replay, reps) * 1e6
        del graph
    for mode in ("reuse", "refine", "refine_W4"):
        res[mode]["speedup_vs_dense"] = res["dense"]["us_per_step"] / res[mode]["us_per_step"]
        res[mode]["graph_speedup_vs_dense"] = res["dense"]["graph_us_per_step"] / res[mode]["graph_us_per_step"]
    key_bytes = B * L * (128 + 4)
    res["dense"]["key_stream_GBps"] = key_bytes / (res["dense"]["us_per_step"] * 1e-6) / 1e9
    res["workload"] = wl.name
    return res


def bf16_score_bench(reps, L=131072, chunk=8192):
    """The bf16 scoring kernel: dense indexer passes over an L-token bf16
    prefill (the 128K prefill recipe with bf16 queries and keys), in chunks of
    `chunk` queries against their causal prefix; the score kernel's time from
    HIP events on its launches, against the bf16 MFMA peak."""
    import torch
    import paper_2607_24593_amd as pv
    from workload.gen import make_prefill
    t = time.time()
    x = make_prefill(L, "bf16", seed=1, rho=0.9, threads=16)
    log(f"generated a {L}-token bf16 prefill in {time.time() - t:.1f}s")
    d = lambda a: torch.from_numpy(a.view("int16") if a.dtype.name == "uint16" else a).cuda()  # noqa: E731
    q, w, k = d(x.q), d(x.w), d(x.k)
    topk = 2048
    out = torch.empty((L, topk), dtype=torch.int32, device="cuda")
    chunks = [(p0, min(chunk, L - p0)) for p0 in range(0, L, chunk)]

    def run():
        for p0, n in chunks:
            pv.pivot_dense_index(q[p0:p0 + n], None, w[p0:p0 + n], k[:p0 + n], None, p0, p0 + n, topk,
                                 out=out[p0:p0 + n])
    run()
    torch.cuda.synchronize()
    with no_gc():
        pv.pivot_profile_begin(["score"])
        t = time.perf_counter()
        for _ in range(reps):
            run()
        torch.cuda.synchronize()
        sec = (time.perf_counter() - t) / reps
        prof = pv.pivot_profile_end()
    n_sc, ms_sc = prof["score"]
    flops = sum(p0 + i + 1 for p0, n in chunks for i in range(n)) * FLOP_PER_PAIR
    tf = flops * reps / (ms_sc * 1e-3) / 1e12
    return {"workload": f"prefill-{L // 1024}k-bf16 (dense, {len(chunks)} calls of {chunk} queries)",
            "ms_per_pass": sec * 1e3, "score_launches_per_pass": n_sc / reps,
            "score_ms_per_pass": ms_sc / reps, "score_TFLOPs": tf, "peak": PEAK["bf16"], "frac": tf / PEAK["bf16"]}


def layout_bench(reps):
    """The batch layouts: the 32 x 131072-key decode with keys in a paged pool
    (pages of 64 keys, shuffled) against the same keys contiguous, and a
    prefill batch of four requests (8K, 16K, 24K and 32K fp8 tokens, their
    last 4096 queries each) as one packed call against one call per request."""
    import numpy as np
    import torch
    import paper_2607_24593_amd as pv
    from workload.gen import WORKLOADS, make, make_prefill
    res = {}
    wl = WORKLOADS["decode-32x128k-fp8"]
    x = make(wl, threads=16)
    B, L, g = wl.batch, wl.L, wl.g[0]
    d = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()  # noqa: E731
    q, qs, w = d(x.q), d(x.q_scale), d(x.w)
    page = 64
    per = L // page
    perm = np.random.default_rng(0).permutation(B * per).astype(np.int32)
    table = perm.reshape(B, per)
    pool = np.empty((B * per * page, x.k.shape[2]), dtype=x.k.dtype)
    pool_s = np.empty(B * per * page, dtype=np.float32)
    kv = x.k.reshape(B, per, page, -1)
    sv = x.k_scale.reshape(B, per, page)
    for b in range(B):
        pool.reshape(B * per, page, -1)[table[b]] = kv[b]
        pool_s.reshape(B * per, page)[table[b]] = sv[b]
    k, ks, kp, ksp, bt = d(x.k), d(x.k_scale), d(pool), d(pool_s), d(table)
    lay = pv.make_layout(cu_q=[g * b for b in range(B + 1)], block_table=bt, page_size=page, pool_keys=pool.shape[0])
    pos, nk = [L - g] * B, [L] * B
    out = torch.empty((B, g, wl.topk), dtype=torch.int32, device="cuda")
    outf = out.view(B * g, wl.topk)
    qf, qsf, wf = q.view(B * g, 64, 128), qs.view(B * g), w.view(B * g, 64)
    dec = {}
    for mode in ("dense", "reuse", "refine"):
        if mode == "dense":
            fc = lambda: pv.pivot_dense_index(q, qs, w, k, ks, pos, nk, wl.topk, out=out)  # noqa: E731
            fp = lambda: pv.pivot_dense_index_layout(qf, qsf, wf, kp, ksp, pos, nk, wl.topk, lay, out=outf)  # noqa
        else:
            m = pv.PIVOT_REUSE if mode == "reuse" else pv.PIVOT_REFINE
            fc = lambda m=m: pv.pivot_group_index(q, qs, w, k, ks, pos, nk, wl.topk, mode=m, g=g, c=wl.c,  # noqa
                                                  out=out)
            fp = lambda m=m: pv.pivot_group_index_layout(qf, qsf, wf, kp, ksp, pos, nk, wl.topk, lay, mode=m,  # noqa
                                                         g=g, c=wl.c, out=outf)
        fc(); fp()  # noqa: E702
        tc, tp = timed(fc, reps), timed(fp, reps)
        dec[mode] = {"contiguous_us": tc * 1e6, "paged_us": tp * 1e6, "paged_over_contiguous": tp / tc}
    res["decode_paged"] = dec
    # a prefill batch of four requests
    lens = [8192, 16384, 24576, 32768]
    n_last = 4096
    xs = [make_prefill(Lr, "fp8", seed=123 + i, threads=16) for i, Lr in enumerate(lens)]
    qp = d(np.concatenate([xr.q[Lr - n_last:] for xr, Lr in zip(xs, lens)]))
    qsp = d(np.concatenate([xr.q_scale[Lr - n_last:] for xr, Lr in zip(xs, lens)]))
    wp = d(np.concatenate([xr.w[Lr - n_last:] for xr, Lr in zip(xs, lens)]))
    S = max(lens)
    kb = np.zeros((len(lens), S, 128), dtype=np.uint8)
    kbs = np.zeros((len(lens), S), dtype=np.float32)
    for i, (xr, Lr) in enumerate(zip(xs, lens)):
        kb[i, :Lr] = xr.k
        kbs[i, :Lr] = xr.k_scale
    kb_t, kbs_t = d(kb), d(kbs)
    cu = [n_last * i for i in range(len(lens) + 1)]
    lay2 = pv.make_layout(cu_q=cu)
    pos2, nk2 = [Lr - n_last for Lr in lens], lens
    outp = torch.empty((n_last * len(lens), 2048), dtype=torch.int32, device="cuda")

    def packed():
        pv.pivot_group_index_layout(qp, qsp, wp, kb_t, kbs_t, pos2, nk2, 2048, lay2, mode=pv.PIVOT_REFINE, g=4,
                                    c=4096, out=outp)

    def separate():
        for i, Lr in enumerate(lens):
            sl = slice(cu[i], cu[i + 1])
            pv.pivot_group_index(qp[sl], qsp[sl], wp[sl], kb_t[i, :Lr], kbs_t[i, :Lr], Lr - n_last, Lr, 2048,
                                 mode=pv.PIVOT_REFINE, g=4, c=4096, out=outp[sl])
    packed(); separate()  # noqa: E702
    tpk, tsep = timed(packed, reps), timed(separate, reps)
    res["prefill_batch"] = {"requests": lens, "queries_each": n_last, "mode": "refine g=4 c=4096 k=2048",
                            "packed_ms": tpk * 1e3, "per_request_calls_ms": tsep * 1e3,
                            "packed_queries_per_s": n_last * len(lens) / tpk}
    return res


def cpu_baseline(pf, g, budget_s=12.0, max_groups=4096):
    """The oracle (C, fp64, OpenMP) on a sample of PIVOT-Refine groups of the same
    prefill: groups at uniformly random positions past the guardrail, drawn until
    about budget_s seconds of CPU work."""
    import numpy as np
    import oracle
    oracle.build(force=False)
    wl, x = pf.wl, pf.x
    rng = np.random.default_rng(0)
    lo = wl.c  # first position past the guardrail
    fp8 = wl.dtype == "fp8"
    t0s = []
    t = time.perf_counter()
    while time.perf_counter() - t < budget_s and len(t0s) < max_groups:
        t0 = int(rng.integers(lo, wl.L - g)) // g * g
        oracle.index(wl.dtype, x.q[t0:t0 + g], x.q_scale[t0:t0 + g] if fp8 else None, x.w[t0:t0 + g], t0,
                     x.k[:t0 + g], x.k_scale[:t0 + g] if fp8 else None, t0 + g, mode=oracle.REFINE, g=g, c=wl.c,
                     topk=wl.topk)
        t0s.append(t0)
    sec = time.perf_counter() - t
    t0s.sort()
    pairs_sample = sum(t0 + 1 + g * wl.c for t0 in t0s)
    full = units(pf.chunks, "refine", g, wl.c, wl.topk)
    pairs_full = full["pairs"] + full["refine_flops"] // FLOP_PER_PAIR
    return {"value": len(t0s) * g / sec, "unit": "queries/s", "cores": oracle.num_threads(), "kind": "oracle",
            "cpu_model": cpu_model(),
            "sample": f"{len(t0s)} PIVOT-Refine groups (g={g}, c={wl.c}, k={wl.topk}) at random positions "
                      f"{t0s[0]}..{t0s[-1]} of {wl.name}, {sec:.1f}s",
            "full_config_s_extrapolated": sec * pairs_full / pairs_sample}


def cpu_model():
    """The host CPU's model name (first processor in /proc/cpuinfo)."""
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    import platform
    return platform.processor() or "unknown"


# The paper's own indexer speedups (NVIDIA H20, DeepSeek-V3.2 / GLM-5.1
# activations): reported beside this library's numbers as context, not as a
# target (other hardware, other inputs).
PAPER_CONTEXT = {
    "hardware": "NVIDIA H20",
    "indexer_speedup_up_to": 4.0,
    "indexer_kernel_speedup_longest_context": 4.8,
    "reuse_kernel_speedup": "about 4x, 16K-256K, prefill and decode",
    "refine_kernel_speedup_16k": {"prefill": 0.93, "decode": 1.40},
    "refine_kernel_speedup_256k": {"prefill": 3.87, "decode": 3.42},
    "settings": "g=4, k=2048, c=4096; decode g=4 (MTP depth 3)",
    "source": "Abstract; Sec. 5.3 (Fig. 4); App. D",
    "note": "context only: different GPU, different inputs; absolute latencies are in the paper's figures only",
}


def recorded_traffic(kernel):
    """HBM bytes per launch of the score kernel from the committed counter
    summary, or None when its sources changed since the counters were taken."""
    import hashlib
    if kernel != "score":
        return None
    path = os.path.join(ROOT, "profiles", "score_kernel_traffic.txt")
    if not os.path.exists(path):
        return None
    rec = {}
    for line in open(path):
        if line.strip() and not line.startswith("#"):
            key, val = line.split()
            rec[key] = val
    csrc = os.path.join(ROOT, "paper_2607_24593_amd", "csrc")
    src = b"".join(open(os.path.join(csrc, f), "rb").read()
                   for f in ("score.hip", "mfma_tile.h", "device_common.h", "api.hip"))
    if hashlib.sha256(src).hexdigest() != rec.get("sources_sha256"):
        return None
    return float(rec["read_bytes_per_launch"]) + float(rec["written_bytes_per_launch"])


def calibrate_copy(nbytes=1 << 30, reps=3):
    """A plain elementwise copy of nbytes (reads nbytes, writes nbytes): the
    reference for scaling FETCH_SIZE / WRITE_SIZE counter readings."""
    import torch
    x = torch.ones(nbytes // 4, dtype=torch.float32, device="cuda")
    y = torch.empty_like(x)
    for _ in range(reps):
        torch.mul(x, 1.0, out=y)
    torch.cuda.synchronize()
    print(json.dumps({"calibration": "elementwise copy", "bytes_read": nbytes, "bytes_written": nbytes,
                      "dispatches": reps}), flush=True)


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=3)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--workload", default="prefill-128k-fp8")
    ap.add_argument("--g", type=int, default=4)
    ap.add_argument("--reps", type=int, default=2, help="passes per mode for the comparison table")
    ap.add_argument("--no-sweep", action="store_true")
    ap.add_argument("--no-decode", action="store_true")
    ap.add_argument("--no-layouts", action="store_true", help="skip the paged / packed-batch measurement")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-compare", action="store_true", help="skip the dense / Reuse / sweep passes")
    ap.add_argument("--score-tile-mb", type=int, default=None,
                    help="score-tile budget in MiB (default: the library's recommended workspace)")
    ap.add_argument("--decode-only", action="store_true", help="only the decode measurement")
    ap.add_argument("--no-configs", action="store_true",
                    help="skip the timed passes of the 2K bf16, 32K fp8 and 256K fp8 workloads")
    ap.add_argument("--no-indexcache", action="store_true", help="skip the multi-layer IndexCache measurement")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="only run a plain 1 GiB device copy kernel (HBM counter calibration)")
    args = ap.parse_args()
    if args.calibrate_copy:
        calibrate_copy()
        return
    if args.decode_only:
        import paper_2607_24593_amd as pv
        pv.lib()
        print(json.dumps({"decode": decode_bench(reps=50)}), flush=True)
        return
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(f"bench.py measures one GPU: this library has no multi-GPU path (asked for {max(args.gpus, world)})",
              file=sys.stderr)
        sys.exit(2)

    import torch
    import paper_2607_24593_amd as pv
    from workload.gen import WORKLOADS
    assert torch.cuda.is_available(), "bench.py needs a GPU"
    pv.lib()
    wl = WORKLOADS[args.workload]
    g = args.g
    pf = Prefill(wl, threads=16, score_tile_mb=args.score_tile_mb)

    # ---- headline: PIVOT-Refine steps
    for _ in range(args.warmup):
        pf.run("refine", g)
    torch.cuda.synchronize()
    # Events bracket only the scoring launches in the timed steps (each event
    # pair between dependent launches adds a gap); the breakdown over every
    # kernel comes from a separate profiled pass below.
    with no_gc():
        pv.pivot_profile_begin(["score"])
        t = time.perf_counter()
        for _ in range(args.steps):
            pf.run("refine", g)
        torch.cuda.synchronize()
        step_s = (time.perf_counter() - t) / args.steps
        prof_timed = pv.pivot_profile_end()
    log(f"refine g={g}: {step_s * 1e3:.2f} ms/step; score kernel {prof_timed['score']}")
    qps = wl.L / step_s
    KB = max(2, min(args.steps, 3))
    with no_gc():
        pv.pivot_profile_begin()
        for _ in range(KB):
            pf.run("refine", g)
        torch.cuda.synchronize()
        prof = pv.pivot_profile_end()
    log(f"kernel breakdown over {KB} profiled steps: {prof}")

    eb = 1 if wl.dtype == "fp8" else 2
    u = units(pf.chunks, "refine", g, wl.c, wl.topk, eb, eb)
    kern = {}
    for name, (n, ms) in prof.items():
        if n == 0:
            continue
        K = KB
        if name == "score":  # the timed steps' own events
            (n, ms), K = prof_timed["score"], args.steps
        e = {"launches_per_step": n / K, "ms_per_step": ms / K, "avg_launch_ms": ms / n}
        if name == "score":
            e.update(bound="mfma", achieved=u["score_flops"] * K / (ms * 1e-3) / 1e12, unit="TFLOP/s",
                     peak=PEAK[wl.dtype])
        elif name == "select":
            e.update(bound="hbm", achieved=u["select_bytes"] * K / (ms * 1e-3) / 1e9, unit="GB/s", peak=HBM_PEAK)
        elif name == "refine":
            e.update(bound="hbm", achieved=u["refine_bytes"] * K / (ms * 1e-3) / 1e9, unit="GB/s", peak=HBM_PEAK,
                     mfma_TFLOPs=u["refine_flops"] * K / (ms * 1e-3) / 1e12)
        elif name == "proxy":
            e.update(bound="hbm", achieved=u["proxy_bytes"] * K / (ms * 1e-3) / 1e9, unit="GB/s", peak=HBM_PEAK)
        if "achieved" in e:
            e["frac"] = e["achieved"] / e["peak"]
        kern[name] = e
    dom = max(kern, key=lambda n: kern[n]["ms_per_step"])
    dk = kern[dom]
    roofline = {"kernel": dom, "bound": dk.get("bound"), "achieved": dk.get("achieved"), "peak": dk.get("peak"),
                "unit": dk.get("unit"), "frac": dk.get("frac"), "traffic": recorded_traffic(dom),
                "traffic_unit": "HBM bytes per launch (FETCH_SIZE + WRITE_SIZE, copy-calibrated)",
                "units_per_step": {"score_pairs": u["pairs"], "score_flops": u["score_flops"],
                                   "select_bytes": u["select_bytes"], "refine_bytes": u["refine_bytes"]}}

    # ---- comparison: dense, Reuse, g sweep
    modes = {}
    dense_s = None if args.no_compare else timed(lambda: pf.run("dense", g), args.reps)
    ud = units(pf.chunks, "dense", 1, wl.c, wl.topk, eb, eb)
    if dense_s is not None:
        modes["dense"] = {"ms_per_pass": dense_s * 1e3, "queries_per_s": wl.L / dense_s,
                          "score_TFLOPs_incl_select": ud["score_flops"] / dense_s / 1e12}
        log(f"dense: {dense_s * 1e3:.2f} ms")
    sweep = () if args.no_compare else (wl.g if not args.no_sweep else (g,))
    for gg in sweep:
        for mode in ("reuse", "refine"):
            s = step_s if (mode == "refine" and gg == g) else timed(lambda: pf.run(mode, gg), args.reps)
            modes[f"{mode}_g{gg}"] = {"ms_per_pass": s * 1e3, "queries_per_s": wl.L / s,
                                      "speedup_vs_dense": dense_s / s}
            log(f"{mode} g={gg}: {s * 1e3:.2f} ms ({dense_s / s:.2f}x)")
    if not args.no_compare:  # App. B's local window at the paper's W = 4
        s = timed(lambda: pf.run("refine", g, window=4), args.reps)
        modes[f"refine_g{g}_W4"] = {"ms_per_pass": s * 1e3, "queries_per_s": wl.L / s,
                                    "speedup_vs_dense": dense_s / s}
        log(f"refine g={g} W=4: {s * 1e3:.2f} ms ({dense_s / s:.2f}x)")

    two = None
    if not args.no_compare:  # independent chunk calls overlapped on two streams
        run_two_streams(pf, "refine", g)
        r2 = timed(lambda: run_two_streams(pf, "refine", g), args.reps)
        d2 = timed(lambda: run_two_streams(pf, "dense", g), args.reps)
        two = {"refine_ms_per_pass": r2 * 1e3, "queries_per_s": wl.L / r2, "dense_ms_per_pass": d2 * 1e3,
               "speedup_vs_dense": d2 / r2, "vs_one_stream": step_s / r2}
        log(f"two streams: refine {r2 * 1e3:.2f} ms, dense {d2 * 1e3:.2f} ms ({step_s / r2:.3f}x one stream)")
    ic = None if args.no_indexcache else indexcache_bench(pf, g, reps=args.reps)
    bf16 = None if args.no_compare else bf16_score_bench(reps=args.reps)
    if bf16 is not None:
        log(f"bf16 score kernel: {bf16['score_TFLOPs']:.0f} TFLOP/s ({100 * bf16['frac']:.1f}% of peak)")
    dec = None if args.no_decode else decode_bench(reps=50)
    if dec is not None:
        log("decode us/step (eager | graph): " + ", ".join(
            f"{m} {dec[m]['us_per_step']:.1f} | {dec[m]['graph_us_per_step']:.1f}" for m in ("dense", "reuse", "refine")))
    layouts = None if args.no_layouts else layout_bench(reps=20)
    cpu = None if args.no_cpu_baseline else cpu_baseline(pf, g)
    ws_bytes = int(pf.ws.numel())
    del pf
    gc.collect()
    torch.cuda.empty_cache()
    configs = None
    if not args.no_configs:
        configs = {
            "prefill-2k-bf16": workload_bench("prefill-2k-bf16", ("dense", "reuse", "refine"), reps=20),
            "prefill-32k-fp8": workload_bench("prefill-32k-fp8", ("dense", "reuse", "refine"), reps=args.reps),
            "prefill-256k-fp8-pareto": workload_bench("prefill-256k-fp8-pareto", ("dense", "refine"), reps=1),
        }

    line = {
        "metric": "indexed queries/s and speedup vs dense indexer at 128K prefill; MFMA % of peak",
        "value": qps,
        "unit": "queries/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": step_s * 1e3,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": wl.dtype,
        "data": "synthetic",
        "config": {"workload": wl.name, "L": wl.L, "H": wl.H, "d": wl.d, "topk": wl.topk, "c": wl.c, "g": g,
                   "chunk": wl.chunk, "mode": "refine", "guardrail": "t0 < c -> dense",
                   "workspace_bytes": ws_bytes},
        "speedup_vs_dense": None if dense_s is None else dense_s / step_s,
        "mfma_frac_score_kernel": kern.get("score", {}).get("frac"),
        "score_bf16": bf16,
        "roofline": roofline,
        "kernels": kern,
        "kernels_note": f"score: HIP events of the {args.steps} timed steps; other kernels: a separate pass of "
                        f"{KB} steps with events around every launch",
        "modes": modes,
        "two_streams": two,
        "decode": dec,
        "layouts": layouts,
        "indexcache": ic,
        "configs": configs,
        "paper_context": PAPER_CONTEXT,
        "cpu_baseline": cpu,
    }
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
