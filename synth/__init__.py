"""Seeded synthetic Re-Prefill workloads, Qwen2.5-shaped.

Shared input source for the GPU path's tests, the oracle's tests, the smoke check
and the benchmark.  It draws random tensors and the planted "heavy chunk" sets
and rounds to bf16; it computes nothing of the method itself (no logits, no
softmax, no pooling, no selection).

The paper evaluates on few-shot SST-2 / SubJ / TREC / RTE prefixes run through
Qwen2.5-7B/14B/32B; neither the datasets nor the weights are used here.  These
tensors stand in for post-RoPE Q/K/V of such prefixes: every KV head g of a
layer gets a random unit direction u_g; every query head of g's group gets
``+1.0*u_g``; the keys of the layer's heavy chunks get ``+alpha*u_g``, so those
chunks draw more attention and the top-k set has known members.  Heavy sets
drift from layer to layer by resampling a fraction of their members, standing in
for the paper's observation that important-chunk indices are similar across
layers (Sec. 4.3.1).

Random streams: numpy PCG64 seeded by SeedSequence([seed, cfg_id, layer,
tensor_id]), one independent stream per (layer, tensor), so layers can be
generated in any order or in parallel with identical results.
"""
from __future__ import annotations

import math
from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass, replace
from typing import Optional

import numpy as np

# tensor ids of the random streams
_T_Q, _T_KP, _T_VP, _T_KS, _T_VS, _T_U, _T_HEAVY = range(7)


@dataclass(frozen=True)
class Workload:
    name: str
    cfg_id: int
    n_layers: int
    n_prefix: int
    n_suffix: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    chunk_size: int
    keep_ratio: float
    dtype: str  # "f32" or "bf16"
    seed: int
    alpha: float  # key boost of heavy chunks along u
    heavy: str  # "planted3", "uniform" or "runs"
    heavy_frac: float = 0.05
    resample_frac: float = 0.0
    host_resident: bool = False
    sm_scale: float = 0.0

    @property
    def n_chunks(self) -> int:
        return -(-self.n_prefix // self.chunk_size)

    @property
    def group(self) -> int:
        return self.n_q_heads // self.n_kv_heads

    @property
    def elem_bytes(self) -> int:
        return 4 if self.dtype == "f32" else 2

    def scaled(self, **kw) -> "Workload":
        """Same recipe at other sizes (used for small parity cases)."""
        return replace(self, **kw)


# The five workloads: shapes of Qwen2.5-0.5B/7B/14B/32B attention layers (GQA
# head counts and head_dim of those models), prefix/suffix lengths, chunk
# sizes and keep ratios of the stated configurations.  Seeds: 0 for the small
# fp32 case, 42 (the paper's fixed seed) for the rest.
WORKLOADS = {
    "c1_f32_1k": Workload("c1_f32_1k", 1, 1, 1024, 32, 4, 1, 64, 16, 0.25, "f32", 0, 2.0,
                          "planted3"),
    "c2_qwen05b_8k": Workload("c2_qwen05b_8k", 2, 24, 8192, 128, 14, 2, 64, 16, 0.20, "bf16",
                              42, 1.5, "uniform", 0.05, 0.10),
    "c3_qwen7b_32k": Workload("c3_qwen7b_32k", 3, 28, 32768, 256, 28, 4, 128, 32, 0.10, "bf16",
                              42, 1.5, "uniform", 0.05, 0.15),
    "c4_qwen14b_64k_c8": Workload("c4_qwen14b_64k_c8", 4, 48, 65536, 512, 40, 8, 128, 8, 0.15,
                                  "bf16", 42, 1.5, "runs", 0.05, 0.15),
    "c4_qwen14b_64k_c16": Workload("c4_qwen14b_64k_c16", 4, 48, 65536, 512, 40, 8, 128, 16, 0.15,
                                   "bf16", 42, 1.5, "runs", 0.05, 0.15),
    "c4_qwen14b_64k_c32": Workload("c4_qwen14b_64k_c32", 4, 48, 65536, 512, 40, 8, 128, 32, 0.15,
                                   "bf16", 42, 1.5, "runs", 0.05, 0.15),
    "c4_qwen14b_64k_c64": Workload("c4_qwen14b_64k_c64", 4, 48, 65536, 512, 40, 8, 128, 64, 0.15,
                                   "bf16", 42, 1.5, "runs", 0.05, 0.15),
    "c5_qwen32b_128k_host": Workload("c5_qwen32b_128k_host", 5, 64, 131072, 1024, 40, 8, 128, 32,
                                     0.10, "bf16", 42, 1.5, "uniform", 0.05, 0.15,
                                     host_resident=True),
}


def _rng(w: Workload, layer: int, tensor: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence(
        [w.seed, w.cfg_id, layer, tensor])))


def to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 to bf16 (round to nearest, ties to even); returns uint16 bits."""
    u = np.ascontiguousarray(x, np.float32).view(np.uint32)
    bias = ((u >> 16) & 1) + np.uint32(0x7FFF)
    return ((u + bias) >> 16).astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (np.ascontiguousarray(b, np.uint16).astype(np.uint32) << 16).view(np.float32)


def _normal(rng: np.random.Generator, shape) -> np.ndarray:
    return rng.standard_normal(shape, dtype=np.float32)


def _runs_layout(rng: np.random.Generator, m: int, target: int, max_run: int = 8):
    """Non-overlapping runs of 1..max_run consecutive chunks until >= target chunks."""
    taken = np.zeros(m, bool)
    runs = []
    total = 0
    attempts = 0
    while total < target and attempts < 100000:
        attempts += 1
        length = int(rng.integers(1, max_run + 1))
        start = int(rng.integers(0, m - length + 1))
        lo, hi = max(0, start - 1), min(m, start + length + 1)  # keep a gap between runs
        if taken[lo:hi].any():
            continue
        taken[start:start + length] = True
        runs.append((start, length))
        total += length
    return runs, taken


def heavy_sets(w: Workload) -> list:
    """Per-layer heavy chunk index sets (sorted int64 arrays)."""
    m = w.n_chunks
    rng = _rng(w, 0, _T_HEAVY)
    out = []
    if w.heavy == "planted3":
        base = np.sort(rng.choice(m, size=min(3, m), replace=False))
        return [base.copy() for _ in range(w.n_layers)]
    if w.heavy == "uniform":
        h = max(1, int(round(w.heavy_frac * m)))
        cur = rng.choice(m, size=h, replace=False)
        out.append(np.sort(cur))
        n_swap = int(round(w.resample_frac * h))
        for _ in range(1, w.n_layers):
            cur = cur.copy()
            victims = rng.choice(h, size=n_swap, replace=False)
            pool = np.setdiff1d(np.arange(m), cur)
            cur[victims] = rng.choice(pool, size=n_swap, replace=False)
            out.append(np.sort(cur))
        return out
    if w.heavy == "runs":
        target = max(1, int(math.ceil(w.heavy_frac * m)))
        runs, taken = _runs_layout(rng, m, target)
        out.append(np.flatnonzero(taken))
        for _ in range(1, w.n_layers):
            n_swap = int(round(w.resample_frac * len(runs)))
            victims = set(int(v) for v in rng.choice(len(runs), size=n_swap, replace=False))
            keep = [r for i, r in enumerate(runs) if i not in victims]
            taken = np.zeros(m, bool)
            for s, L in keep:
                taken[s:s + L] = True
            new_runs = list(keep)
            placed = 0
            attempts = 0
            while placed < n_swap and attempts < 100000:
                attempts += 1
                length = int(rng.integers(1, 9))
                start = int(rng.integers(0, m - length + 1))
                lo, hi = max(0, start - 1), min(m, start + length + 1)
                if taken[lo:hi].any():
                    continue
                taken[start:start + length] = True
                new_runs.append((start, length))
                placed += 1
            runs = new_runs
            out.append(np.flatnonzero(taken))
        return out
    raise ValueError(w.heavy)


def layer_tensors(w: Workload, layer: int, heavy: Optional[np.ndarray] = None) -> dict:
    """Q [S][Hq][d], K/V prefix [n][Hkv][d], K/V suffix [S][Hkv][d] of one layer.

    float32 arrays for dtype f32, uint16 bf16 bit patterns for bf16.
    """
    if heavy is None:
        heavy = heavy_sets(w)[layer]
    n, S, Hq, Hkv, d, c = (w.n_prefix, w.n_suffix, w.n_q_heads, w.n_kv_heads, w.head_dim,
                           w.chunk_size)
    G = Hq // Hkv
    u = _normal(_rng(w, layer, _T_U), (Hkv, d)).astype(np.float64)
    u /= np.linalg.norm(u, axis=1, keepdims=True)
    u = u.astype(np.float32)
    q = _normal(_rng(w, layer, _T_Q), (S, Hq, d))
    q += np.repeat(u, G, axis=0)[None, :, :]
    kp = _normal(_rng(w, layer, _T_KP), (n, Hkv, d))
    tok = np.concatenate([np.arange(j * c, min((j + 1) * c, n)) for j in heavy]) if len(heavy) else \
        np.zeros(0, np.int64)
    kp[tok] += np.float32(w.alpha) * u[None, :, :]
    vp = _normal(_rng(w, layer, _T_VP), (n, Hkv, d))
    ks = _normal(_rng(w, layer, _T_KS), (S, Hkv, d))
    vs = _normal(_rng(w, layer, _T_VS), (S, Hkv, d))
    t = {"q": q, "k_prefix": kp, "v_prefix": vp, "k_suffix": ks, "v_suffix": vs}
    if w.dtype == "bf16":
        t = {k: to_bf16_bits(v) for k, v in t.items()}
    return t


def request_queries(w: Workload, layer: int, request: int) -> np.ndarray:
    """Suffix queries Q [S][Hq][d] of request `request` on the workload's shared
    prefix: layer_tensors' recipe for Q (noise plus the layer's per-group
    direction u), with request 0 giving layer_tensors' own Q and every other
    request drawing its noise from a stream of its own."""
    S, Hq, Hkv, d = w.n_suffix, w.n_q_heads, w.n_kv_heads, w.head_dim
    u = _normal(_rng(w, layer, _T_U), (Hkv, d)).astype(np.float64)
    u /= np.linalg.norm(u, axis=1, keepdims=True)
    u = u.astype(np.float32)
    rng = _rng(w, layer, _T_Q) if request == 0 else np.random.Generator(np.random.PCG64(
        np.random.SeedSequence([w.seed, w.cfg_id, layer, _T_Q, request])))
    q = _normal(rng, (S, Hq, d))
    q += np.repeat(u, Hq // Hkv, axis=0)[None, :, :]
    return to_bf16_bits(q) if w.dtype == "bf16" else q


def all_layers(w: Workload, layers=None, threads: int = 8) -> list:
    """layer_tensors for several layers, generated in parallel (same values)."""
    hs = heavy_sets(w)
    layers = list(range(w.n_layers)) if layers is None else list(layers)
    with ThreadPoolExecutor(max_workers=threads) as ex:
        return list(ex.map(lambda l: layer_tensors(w, l, hs[l]), layers))


def chunk_major(k_prefix: np.ndarray, v_prefix: np.ndarray, chunk_size: int) -> np.ndarray:
    """Host store layout of one layer: chunk j is one span [K rows; V rows] of
    chunk_size rows each (rows past n of the last chunk are zero padding).
    Returns an array of shape [m][2][c][Hkv][d]."""
    n, Hkv, d = k_prefix.shape
    m = -(-n // chunk_size)
    out = np.zeros((m, 2, chunk_size, Hkv, d), k_prefix.dtype)
    pad = m * chunk_size - n
    kk = np.concatenate([k_prefix, np.zeros((pad, Hkv, d), k_prefix.dtype)]) if pad else k_prefix
    vv = np.concatenate([v_prefix, np.zeros((pad, Hkv, d), v_prefix.dtype)]) if pad else v_prefix
    out[:, 0] = kk.reshape(m, chunk_size, Hkv, d)
    out[:, 1] = vv.reshape(m, chunk_size, Hkv, d)
    return out
