"""Matrix-product form of the oracle's scoring and attention -- TEST INFRASTRUCTURE ONLY.

The same definitions as ``ckv_oracle.c`` (token importance and Eq. 1 pooling of
Sec. 4.4; re-prefill attention of Def. 2.1 over the kept chunks plus the causal
suffix, GQA of Sec. 2.1), written with fp64 matrix products on the CPU (torch)
as the step that forms every logit and every weighted value sum, so that whole
layers at the workloads' full sizes take seconds.  Summation order inside the
products is the library's; every value is fp64, so results agree with the
sequential C oracle to ~1e-15 relative.  Pinned independently in
``tests/test_oracle_blas.py``.  Only the test suite may import this module; it
imports nothing from the product.

Inputs are numpy arrays: float32 for the fp32 dtype, uint16 bf16 bit patterns
for bf16 (widened exactly to fp64).  Outputs are float64.
"""
from __future__ import annotations

import math

import numpy as np
import torch

from . import BF16, Shape

# rows of the logit matrix formed at once (bounds memory: rows * keys * 8 bytes)
_ROW_BLOCK_ELEMS = 1 << 25


def _widen(x: np.ndarray, dtype: int) -> torch.Tensor:
    """Exact widening to fp64: bf16 bits b are the float32 with bits b << 16."""
    a = np.ascontiguousarray(x)
    if dtype == BF16:
        a = (a.astype(np.uint32) << 16).view(np.float32)
    return torch.from_numpy(np.asarray(a, np.float32)).to(torch.float64)


def _scale(s: Shape) -> float:
    return s.sm_scale if s.sm_scale > 0 else 1.0 / math.sqrt(s.head_dim)


def token_importance(s: Shape, q, k_prefix) -> np.ndarray:
    """a[i] = sum over suffix queries t and query heads h of softmax_i(scale *
    q[t,h] . k[i, h // G]) over the n prefix keys (Sec. 4.4)."""
    S, Hq, Hkv, d, n = s.n_suffix, s.n_q_heads, s.n_kv_heads, s.head_dim, s.n_prefix
    G = Hq // Hkv
    Q = _widen(q, s.dtype).reshape(S, Hq, d)
    K = _widen(k_prefix, s.dtype).reshape(n, Hkv, d)
    a = torch.zeros(n, dtype=torch.float64)
    block = max(1, _ROW_BLOCK_ELEMS // max(n, 1))
    sc = _scale(s)
    for g in range(Hkv):
        Kg = K[:, g, :].contiguous()                                # [n][d]
        Qg = Q[:, g * G:(g + 1) * G, :].reshape(S * G, d)           # rows (t, i), head g*G+i
        for r0 in range(0, S * G, block):
            logits = (Qg[r0:r0 + block] @ Kg.T) * sc                 # [rows][n]
            mx = logits.max(dim=1, keepdim=True).values
            e = torch.exp(logits - mx)
            p = e / e.sum(dim=1, keepdim=True)
            a += p.sum(dim=0)
    return a.numpy()


def chunk_scores(s: Shape, a: np.ndarray) -> np.ndarray:
    """Eq. 1: A[j] = sum of a over chunk j's tokens [j*c, min(j*c + c, n))."""
    n, c = s.n_prefix, s.chunk_size
    m = -(-n // c)
    padded = np.zeros(m * c, np.float64)
    padded[:n] = a
    return padded.reshape(m, c).sum(axis=1)


def sparse_attn(s: Shape, q, k_prefix, v_prefix, sel, k_suffix, v_suffix) -> np.ndarray:
    """Def. 2.1: for query t of head h (KV head h // G) the keys are the tokens
    of the chunks in `sel` (ascending) followed by suffix tokens 0..t; the
    output is the softmax(scale * q.k)-weighted sum of their values.
    Returns out[S][Hq][d] in fp64."""
    S, Hq, Hkv, d, n, c = (s.n_suffix, s.n_q_heads, s.n_kv_heads, s.head_dim, s.n_prefix,
                           s.chunk_size)
    G = Hq // Hkv
    sel = np.asarray(sel, np.int64)
    tok = np.concatenate([np.arange(j * c, min(j * c + c, n)) for j in sel]) if sel.size else \
        np.zeros(0, np.int64)
    T = tok.size
    Q = _widen(q, s.dtype).reshape(S, Hq, d)
    Kp = _widen(k_prefix, s.dtype).reshape(n, Hkv, d)
    Vp = _widen(v_prefix, s.dtype).reshape(n, Hkv, d)
    Ks = _widen(k_suffix, s.dtype).reshape(S, Hkv, d)
    Vs = _widen(v_suffix, s.dtype).reshape(S, Hkv, d)
    idx = torch.from_numpy(tok)
    out = torch.zeros(S, Hq, d, dtype=torch.float64)
    sc = _scale(s)
    block = max(1, _ROW_BLOCK_ELEMS // max(T + S, 1))
    t_of_row = torch.arange(S * G) // G                              # query position of row (t, i)
    for g in range(Hkv):
        Kall = torch.cat([Kp[idx, g, :], Ks[:, g, :]])               # [T + S][d]
        Vall = torch.cat([Vp[idx, g, :], Vs[:, g, :]])
        Qg = Q[:, g * G:(g + 1) * G, :].reshape(S * G, d)
        og = torch.empty(S * G, d, dtype=torch.float64)
        for r0 in range(0, S * G, block):
            r1 = min(S * G, r0 + block)
            logits = (Qg[r0:r1] @ Kall.T) * sc                        # [rows][T + S]
            # suffix key p is visible to query t iff p <= t
            hidden = torch.arange(S)[None, :] > t_of_row[r0:r1, None]
            logits[:, T:][hidden] = -math.inf
            mx = logits.max(dim=1, keepdim=True).values
            e = torch.exp(logits - mx)
            og[r0:r1] = (e @ Vall) / e.sum(dim=1, keepdim=True)
        out[:, g * G:(g + 1) * G, :] = og.reshape(S, G, d)
    return out.numpy()
