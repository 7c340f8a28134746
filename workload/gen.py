"""Synthetic indexer inputs with the shape and structure of the paper's workloads.

The paper times its indexer on model activations (DeepSeek-V3.2 on long-context
suites), which are not available here. These generators stand in for them and
are built to show the two properties the method relies on (Sec. 3.2): nearby
queries are similar (O1: an AR(1) process along the query axis) and the score
distribution is long-tailed along the key axis (O3: a small set of keys shifted
or boosted along one shared direction).

Recipe (every array is float32 before encoding):
  * keys      k[s] ~ N(0, I/d); then either round(0.02 L) distinct positions get
              +3 u ("shift"), or round(0.01 L) positions get +A_s u with
              A_s = 1 + Lomax(alpha) ("pareto", i.e. classic Pareto with x_m = 1);
              u is a random unit vector.
  * queries   per head, q[t] = rho q[t-1] + eps_t, eps_t ~ N(0, I/d), with the
              stationary start q[0] ~ N(0, I/(d (1 - rho^2))).
  * gates     w[t, h] ~ N(0, 1/H).
  * encoding  bf16: round-to-nearest-even.  fp8 (OCP E4M3FN): per-token scale
              amax/448 (queries: amax over all H*d values of the token, keys: over
              d), codes = RNE(x / scale).  The casts are torch's CPU casts.

Random streams come from numpy's PCG64 seeded through SeedSequence; query
innovations are drawn in fixed blocks of QBLOCK rows, each from its own spawned
stream, so the values do not depend on the thread count.
"""
from __future__ import annotations

import math
from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass, field

import numpy as np
import torch

H_DEFAULT = 64
D_DEFAULT = 128
QBLOCK = 2048          # rows per independent query-innovation stream
SEED_BASE = 0x50495654
E4M3_MAX = 448.0


@dataclass(frozen=True)
class Workload:
    """One named workload.  `g` lists the group sizes it is run with."""
    name: str
    wid: int
    kind: str              # "prefill" or "decode"
    dtype: str             # "bf16" or "fp8"
    L: int                 # prefill length, or cached context per decode sequence
    topk: int
    c: int
    g: tuple
    chunk: int             # queries per library call (prefill)
    rho: float
    boost: tuple           # ("shift", frac, amplitude) or ("pareto", frac, alpha)
    batch: int = 1
    H: int = H_DEFAULT
    d: int = D_DEFAULT
    modes: tuple = ("dense", "reuse", "refine")

    @property
    def seed(self) -> int:
        return SEED_BASE + self.wid


WORKLOADS = {
    w.name: w
    for w in [
        Workload("prefill-2k-bf16", 0, "prefill", "bf16", 2048, 256, 512, (4,), 2048,
                 0.95, ("shift", 0.02, 3.0)),
        Workload("prefill-32k-fp8", 1, "prefill", "fp8", 32768, 2048, 4096, (4,), 32768,
                 0.95, ("shift", 0.02, 3.0)),
        Workload("prefill-128k-fp8", 2, "prefill", "fp8", 131072, 2048, 4096, (2, 4, 8), 8192,
                 0.9, ("shift", 0.02, 3.0)),
        Workload("decode-32x128k-fp8", 3, "decode", "fp8", 131072, 2048, 4096, (2,), 2,
                 0.95, ("shift", 0.02, 3.0), batch=32),
        Workload("prefill-256k-fp8-pareto", 4, "prefill", "fp8", 262144, 2048, 4096, (8,), 16384,
                 0.95, ("pareto", 0.01, 1.5), modes=("dense", "refine")),
    ]
}


def workload(name: str) -> Workload:
    return WORKLOADS[name]


@dataclass
class Inputs:
    """Encoded indexer inputs.  Prefill: q [L,H,d], w [L,H], k [L,d].
    Decode: q [B,g,H,d], w [B,g,H], k [B,L,d].  fp8 arrays hold E4M3FN codes
    (uint8) with float32 per-token scales; bf16 arrays hold raw bits (uint16)."""
    dtype: str
    q: np.ndarray
    q_scale: np.ndarray | None
    w: np.ndarray
    k: np.ndarray
    k_scale: np.ndarray | None
    meta: dict = field(default_factory=dict)


# ----------------------------------------------------------------- encodings
def encode_fp8_rows(x: np.ndarray):
    """Per-row (first axis) E4M3FN encoding: scale = amax/448, codes = RNE(x/scale)."""
    flat = x.reshape(x.shape[0], -1)
    amax = np.abs(flat).max(axis=1).astype(np.float32)
    scale = amax / np.float32(E4M3_MAX)
    scale[amax == 0] = np.float32(1.0)
    y = flat / scale[:, None]
    codes = torch.from_numpy(np.ascontiguousarray(y)).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    return codes.reshape(x.shape), scale.astype(np.float32)


def encode_bf16(x: np.ndarray) -> np.ndarray:
    t = torch.from_numpy(np.ascontiguousarray(x)).to(torch.bfloat16)
    return t.view(torch.int16).numpy().view(np.uint16)


def _encode(x: np.ndarray, dtype: str):
    if dtype == "fp8":
        return encode_fp8_rows(x)
    if dtype == "bf16":
        return encode_bf16(x), None
    raise ValueError(dtype)


# ----------------------------------------------------------------- draws
def _draw_keys(ss: np.random.SeedSequence, L: int, d: int, boost: tuple) -> np.ndarray:
    rng = np.random.Generator(np.random.PCG64(ss))
    u = rng.standard_normal(d)
    u /= np.linalg.norm(u)
    k = rng.standard_normal((L, d), dtype=np.float32)
    k *= np.float32(1.0 / math.sqrt(d))
    kind, frac, par = boost
    n = int(round(frac * L))
    if n > 0:
        pos = rng.choice(L, size=n, replace=False)
        if kind == "shift":
            amp = np.full(n, float(par))
        elif kind == "pareto":
            amp = 1.0 + rng.pareto(float(par), size=n)
        else:
            raise ValueError(kind)
        k[pos] += (amp[:, None] * u[None, :]).astype(np.float32)
    return k


def _innovations(ss: np.random.SeedSequence, rows: int, width: int, scale: float) -> np.ndarray:
    rng = np.random.Generator(np.random.PCG64(ss))
    e = rng.standard_normal((rows, width), dtype=np.float32)
    e *= np.float32(scale)
    return e


def _queries_encoded(ss: np.random.SeedSequence, L: int, H: int, d: int, rho: float,
                     dtype: str, threads: int):
    """AR(1) queries along t, encoded block by block (bounded memory)."""
    nblk = (L + QBLOCK - 1) // QBLOCK
    children = ss.spawn(nblk)
    width = H * d
    sig = 1.0 / math.sqrt(d)
    q_codes = np.empty((L, H, d), dtype=np.uint8 if dtype == "fp8" else np.uint16)
    q_scale = np.empty(L, dtype=np.float32) if dtype == "fp8" else None
    carry = None
    r32 = np.float32(rho)
    start_gain = np.float32(1.0 / math.sqrt(1.0 - rho * rho))

    def rows_of(b):
        return min(QBLOCK, L - b * QBLOCK)

    with ThreadPoolExecutor(max_workers=max(1, threads)) as ex:
        window = max(1, threads)
        futs = {}
        for b in range(min(window, nblk)):
            futs[b] = ex.submit(_innovations, children[b], rows_of(b), width, sig)
        for b in range(nblk):
            x = futs.pop(b).result()
            nxt = b + window
            if nxt < nblk:
                futs[nxt] = ex.submit(_innovations, children[nxt], rows_of(nxt), width, sig)
            if carry is None:
                x[0] *= start_gain
            else:
                x[0] += r32 * carry
            for t in range(1, x.shape[0]):
                x[t] += r32 * x[t - 1]
            carry = x[-1].copy()
            lo = b * QBLOCK
            codes, sc = _encode(x.reshape(-1, H, d), dtype)
            q_codes[lo:lo + x.shape[0]] = codes
            if q_scale is not None:
                q_scale[lo:lo + x.shape[0]] = sc
    return q_codes, q_scale


def _gates(ss: np.random.SeedSequence, rows: int, H: int) -> np.ndarray:
    rng = np.random.Generator(np.random.PCG64(ss))
    w = rng.standard_normal((rows, H), dtype=np.float32)
    w *= np.float32(1.0 / math.sqrt(H))
    return w


# ----------------------------------------------------------------- public API
def make_prefill(L: int, dtype: str, *, seed: int, rho: float = 0.95,
                 boost: tuple = ("shift", 0.02, 3.0), H: int = H_DEFAULT, d: int = D_DEFAULT,
                 threads: int = 8) -> Inputs:
    """One prefill sequence of L positions (queries and keys at every position)."""
    ks, qs, ws = np.random.SeedSequence(seed).spawn(3)
    kf = _draw_keys(ks, L, d, boost)
    k_codes, k_scale = _encode(kf, dtype)
    del kf
    q_codes, q_scale = _queries_encoded(qs, L, H, d, rho, dtype, threads)
    w = _gates(ws, L, H)
    return Inputs(dtype, q_codes, q_scale, w, k_codes, k_scale,
                  meta=dict(kind="prefill", L=L, H=H, d=d, rho=rho, boost=boost, seed=seed))


def make_decode(B: int, L: int, g: int, dtype: str, *, seed: int, rho: float = 0.95,
                boost: tuple = ("shift", 0.02, 3.0), H: int = H_DEFAULT, d: int = D_DEFAULT,
                threads: int = 8) -> Inputs:
    """B decode sequences, each with L cached keys; the g queries of one MTP step
    sit at positions L-g .. L-1 of their sequence."""
    per_seq = np.random.SeedSequence(seed).spawn(B)
    kdt = np.uint8 if dtype == "fp8" else np.uint16
    k = np.empty((B, L, d), dtype=kdt)
    k_scale = np.empty((B, L), dtype=np.float32) if dtype == "fp8" else None
    q = np.empty((B, g, H, d), dtype=kdt)
    q_scale = np.empty((B, g), dtype=np.float32) if dtype == "fp8" else None
    w = np.empty((B, g, H), dtype=np.float32)

    def one(b):
        ks, qs, ws = per_seq[b].spawn(3)
        kc, kscale = _encode(_draw_keys(ks, L, d, boost), dtype)
        qc, qscale = _queries_encoded(qs, g, H, d, rho, dtype, threads=1)
        k[b] = kc
        q[b] = qc
        w[b] = _gates(ws, g, H)
        if dtype == "fp8":
            k_scale[b] = kscale
            q_scale[b] = qscale

    with ThreadPoolExecutor(max_workers=max(1, threads)) as ex:
        list(ex.map(one, range(B)))
    return Inputs(dtype, q, q_scale, w, k, k_scale,
                  meta=dict(kind="decode", B=B, L=L, g=g, H=H, d=d, rho=rho, boost=boost, seed=seed))


def make(wl: Workload, threads: int = 8) -> Inputs:
    """Inputs of a named workload at its full size."""
    if wl.kind == "prefill":
        return make_prefill(wl.L, wl.dtype, seed=wl.seed, rho=wl.rho, boost=wl.boost,
                            H=wl.H, d=wl.d, threads=threads)
    return make_decode(wl.batch, wl.L, wl.g[0], wl.dtype, seed=wl.seed, rho=wl.rho,
                       boost=wl.boost, H=wl.H, d=wl.d, threads=threads)
