"""CPU oracle for the ContiguousKV Re-Prefill hot path -- TEST INFRASTRUCTURE ONLY.

Thin ctypes wrapper over ``libckv_oracle.so`` (plain C, fp64; see ``ckv_oracle.c``).
Only the test suite, the smoke check and the benchmark's CPU-baseline leg may
import this package.  The GPU product path never does, and this package imports
nothing from the product.

Inputs are numpy arrays: float32 for the fp32 dtype, uint16 bf16 bit patterns for
bf16.  Outputs are float64 (scores, attention) or int32 (chunk indices).
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from dataclasses import dataclass

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libckv_oracle.so")
SRC_PATH = os.path.join(_HERE, "ckv_oracle.c")

F32, BF16 = 0, 1


def build(force: bool = False) -> str:
    """Compile the oracle with gcc (no contraction, no fast-math)."""
    if force or not os.path.exists(LIB_PATH) or os.path.getmtime(LIB_PATH) < max(
        os.path.getmtime(SRC_PATH), os.path.getmtime(os.path.join(_HERE, "ckv_oracle.h"))
    ):
        tmp = LIB_PATH + ".tmp"
        cmd = [
            "gcc", "-std=c11", "-O2", "-ffp-contract=off", "-fno-fast-math", "-fPIC",
            "-shared", "-pthread", "-Wall", "-Wextra", "-o", tmp, SRC_PATH, "-lm",
        ]
        subprocess.run(cmd, check=True)
        os.replace(tmp, LIB_PATH)
    return LIB_PATH


class _Shape(ctypes.Structure):
    _fields_ = [
        ("n_prefix", ctypes.c_int64),
        ("n_suffix", ctypes.c_int32),
        ("n_q_heads", ctypes.c_int32),
        ("n_kv_heads", ctypes.c_int32),
        ("head_dim", ctypes.c_int32),
        ("chunk_size", ctypes.c_int32),
        ("dtype", ctypes.c_int32),
        ("sm_scale", ctypes.c_double),
    ]


class _Stats(ctypes.Structure):
    _fields_ = [(f, ctypes.c_int64) for f in
                ("k", "hits", "misses", "wasted", "bytes_prefetch", "bytes_demand", "bytes_used")]


class _IoCounts(ctypes.Structure):
    _fields_ = [(f, ctypes.c_int64) for f in ("tokens_selected", "runs", "blocks", "tokens_block")]


class _CacheCounts(ctypes.Structure):
    _fields_ = [(f, ctypes.c_int64) for f in ("hits_gpu", "hits_cpu", "misses", "demoted", "dropped")]


@dataclass(frozen=True)
class Shape:
    n_prefix: int
    n_suffix: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    chunk_size: int
    dtype: int = BF16
    sm_scale: float = 0.0

    def c(self) -> _Shape:
        return _Shape(self.n_prefix, self.n_suffix, self.n_q_heads, self.n_kv_heads,
                      self.head_dim, self.chunk_size, self.dtype, self.sm_scale)

    @property
    def n_chunks(self) -> int:
        return -(-self.n_prefix // self.chunk_size)


_lib = None


def load(path: str):
    """Loads an oracle shared library and declares its C signatures."""
    L = ctypes.CDLL(path)
    P = ctypes.c_void_p
    SP = ctypes.POINTER(_Shape)
    L.ckvo_num_chunks.argtypes = [ctypes.c_int64, ctypes.c_int32]
    L.ckvo_num_chunks.restype = ctypes.c_int64
    L.ckvo_num_keep.argtypes = [ctypes.c_int64, ctypes.c_double]
    L.ckvo_num_keep.restype = ctypes.c_int64
    L.ckvo_token_importance.argtypes = [SP, P, P, P, ctypes.c_int]
    L.ckvo_chunk_scores.argtypes = [SP, P, P]
    L.ckvo_select_topk.argtypes = [P, ctypes.c_int64, ctypes.c_int64, P]
    L.ckvo_sparse_attn.argtypes = [SP, P, P, P, P, ctypes.c_int64, P, P, P, ctypes.c_int64,
                                   P, ctypes.c_int]
    L.ckvo_dense_attn.argtypes = [SP, P, P, P, P, P, P, ctypes.c_int64, P, ctypes.c_int]
    L.ckvo_gather_chunks.argtypes = [SP, P, P, P, ctypes.c_int64, P, P]
    L.ckvo_layer_accounting.argtypes = [SP, P, ctypes.c_int64, P, ctypes.c_int64,
                                        ctypes.POINTER(_Stats)]
    L.ckvo_reprefill_layer.argtypes = [SP, ctypes.c_double, P, P, P, P, P, P, P,
                                       ctypes.POINTER(ctypes.c_int64), P, ctypes.c_int]
    L.ckvo_io_account.argtypes = [ctypes.c_int64, ctypes.c_int32, P, ctypes.c_int64,
                                  ctypes.c_int32, ctypes.POINTER(_IoCounts)]
    L.ckvo_cache_create.argtypes = [ctypes.c_int64, ctypes.c_int64, ctypes.c_int64, ctypes.c_int]
    L.ckvo_cache_create.restype = P
    L.ckvo_cache_destroy.argtypes = [P]
    L.ckvo_cache_destroy.restype = None
    L.ckvo_cache_access.argtypes = [P, P, P, ctypes.c_int64, P, ctypes.POINTER(_CacheCounts)]
    L.ckvo_cache_state.argtypes = [P, P, P, P]
    for f in ("ckvo_token_importance", "ckvo_chunk_scores", "ckvo_select_topk",
              "ckvo_sparse_attn", "ckvo_dense_attn", "ckvo_gather_chunks",
              "ckvo_layer_accounting", "ckvo_reprefill_layer", "ckvo_io_account",
              "ckvo_cache_access", "ckvo_cache_state"):
        getattr(L, f).restype = ctypes.c_int
    return L


def lib():
    global _lib
    if _lib is None:
        build()
        _lib = load(LIB_PATH)
    return _lib


class OracleError(RuntimeError):
    pass


def _check(rc: int, what: str) -> None:
    if rc != 0:
        raise OracleError(f"{what} failed with code {rc}")


def _elem_dtype(shape: Shape):
    return np.float32 if shape.dtype == F32 else np.uint16


def _arr(x, shape: Shape, count: int, name: str) -> np.ndarray:
    a = np.ascontiguousarray(x)
    if a.dtype != _elem_dtype(shape):
        raise TypeError(f"{name}: expected {np.dtype(_elem_dtype(shape))}, got {a.dtype}")
    if a.size != count:
        raise ValueError(f"{name}: expected {count} elements, got {a.size}")
    return a


def _ptr(a: np.ndarray):
    return ctypes.c_void_p(a.ctypes.data) if a is not None else None


def num_chunks(n: int, c: int) -> int:
    return int(lib().ckvo_num_chunks(n, c))


def num_keep(m: int, r: float) -> int:
    return int(lib().ckvo_num_keep(m, r))


def token_importance(shape: Shape, q, k_prefix, threads: int = 0) -> np.ndarray:
    s = shape
    q = _arr(q, s, s.n_suffix * s.n_q_heads * s.head_dim, "q")
    k = _arr(k_prefix, s, s.n_prefix * s.n_kv_heads * s.head_dim, "k_prefix")
    a = np.zeros(s.n_prefix, np.float64)
    _check(lib().ckvo_token_importance(ctypes.byref(s.c()), _ptr(q), _ptr(k), _ptr(a), threads),
           "token_importance")
    return a


def chunk_scores(shape: Shape, a: np.ndarray) -> np.ndarray:
    a = np.ascontiguousarray(a, np.float64)
    A = np.zeros(shape.n_chunks, np.float64)
    _check(lib().ckvo_chunk_scores(ctypes.byref(shape.c()), _ptr(a), _ptr(A)), "chunk_scores")
    return A


def select_topk(A: np.ndarray, k: int) -> np.ndarray:
    A = np.ascontiguousarray(A, np.float64)
    sel = np.zeros(k, np.int32)
    _check(lib().ckvo_select_topk(_ptr(A), A.size, k, _ptr(sel)), "select_topk")
    return sel


def _rows(row_ids):
    if row_ids is None:
        return None, 0
    r = np.ascontiguousarray(row_ids, np.int64)
    return r, r.size


def sparse_attn(shape: Shape, q, k_prefix, v_prefix, sel, k_suffix, v_suffix,
                row_ids=None, threads: int = 0) -> np.ndarray:
    s = shape
    q = _arr(q, s, s.n_suffix * s.n_q_heads * s.head_dim, "q")
    kp = _arr(k_prefix, s, s.n_prefix * s.n_kv_heads * s.head_dim, "k_prefix")
    vp = _arr(v_prefix, s, s.n_prefix * s.n_kv_heads * s.head_dim, "v_prefix")
    ks = _arr(k_suffix, s, s.n_suffix * s.n_kv_heads * s.head_dim, "k_suffix")
    vs = _arr(v_suffix, s, s.n_suffix * s.n_kv_heads * s.head_dim, "v_suffix")
    sel = np.ascontiguousarray(sel, np.int32)
    rows, nr = _rows(row_ids)
    out = np.zeros(((nr if rows is not None else s.n_suffix * s.n_q_heads), s.head_dim), np.float64)
    _check(lib().ckvo_sparse_attn(ctypes.byref(s.c()), _ptr(q), _ptr(kp), _ptr(vp), _ptr(sel),
                                  sel.size, _ptr(ks), _ptr(vs), _ptr(rows), nr, _ptr(out), threads),
           "sparse_attn")
    return out if rows is not None else out.reshape(s.n_suffix, s.n_q_heads, s.head_dim)


def dense_attn(shape: Shape, q, k_prefix, v_prefix, k_suffix, v_suffix, row_ids=None,
               threads: int = 0) -> np.ndarray:
    s = shape
    q = _arr(q, s, s.n_suffix * s.n_q_heads * s.head_dim, "q")
    kp = _arr(k_prefix, s, s.n_prefix * s.n_kv_heads * s.head_dim, "k_prefix")
    vp = _arr(v_prefix, s, s.n_prefix * s.n_kv_heads * s.head_dim, "v_prefix")
    ks = _arr(k_suffix, s, s.n_suffix * s.n_kv_heads * s.head_dim, "k_suffix")
    vs = _arr(v_suffix, s, s.n_suffix * s.n_kv_heads * s.head_dim, "v_suffix")
    rows, nr = _rows(row_ids)
    out = np.zeros(((nr if rows is not None else s.n_suffix * s.n_q_heads), s.head_dim), np.float64)
    _check(lib().ckvo_dense_attn(ctypes.byref(s.c()), _ptr(q), _ptr(kp), _ptr(vp), _ptr(ks),
                                 _ptr(vs), _ptr(rows), nr, _ptr(out), threads), "dense_attn")
    return out if rows is not None else out.reshape(s.n_suffix, s.n_q_heads, s.head_dim)


def gather_chunks(shape: Shape, k_src, v_src, sel):
    s = shape
    ks = _arr(k_src, s, s.n_prefix * s.n_kv_heads * s.head_dim, "k_src")
    vs = _arr(v_src, s, s.n_prefix * s.n_kv_heads * s.head_dim, "v_src")
    sel = np.ascontiguousarray(sel, np.int32)
    rows = sel.size * s.chunk_size
    # filled with a sentinel so that a missing zero-fill of a short chunk shows
    kd = np.full((rows, s.n_kv_heads, s.head_dim), 0xFFFF if s.dtype == BF16 else np.nan,
                 _elem_dtype(s))
    vd = kd.copy()
    _check(lib().ckvo_gather_chunks(ctypes.byref(s.c()), _ptr(ks), _ptr(vs), _ptr(sel), sel.size,
                                    _ptr(kd), _ptr(vd)), "gather_chunks")
    return kd, vd


def layer_accounting(shape: Shape, sel, pred) -> dict:
    sel = np.ascontiguousarray(sel, np.int32)
    pred = np.ascontiguousarray(pred if pred is not None else [], np.int32)
    st = _Stats()
    _check(lib().ckvo_layer_accounting(ctypes.byref(shape.c()), _ptr(sel), sel.size, _ptr(pred),
                                       pred.size, ctypes.byref(st)), "layer_accounting")
    return {f: int(getattr(st, f)) for f, _ in _Stats._fields_}


def period_first_layer(layer: int, period: int) -> int:
    """First layer of the Period that holds `layer` (Def. 4.2, Sec. 4.3): the
    layers are cut, from layer 0, into Periods of `period` consecutive layers,
    and every layer of a Period uses the important-chunk set selected at the
    Period's first layer."""
    if period < 1 or layer < 0:
        raise ValueError("period must be >= 1 and layer >= 0")
    return layer - layer % period


def period_prediction(sets: list, period: int) -> list:
    """Prefetch prediction of every layer when each layer's set follows its
    Period: P_0 = empty, P_l = the set layer l-1 used (Sec. 4.3.2), with
    layer l using sets[period_first_layer(l, period)] (only the entries of
    Period first layers are read)."""
    used = [np.asarray(sets[period_first_layer(l, period)], np.int32) for l in range(len(sets))]
    return [np.zeros(0, np.int32)] + used[:-1]


def reprefill_layer(shape: Shape, keep_ratio: float, q, k_prefix, v_prefix, k_suffix, v_suffix,
                    threads: int = 0):
    """One layer: returns (chunk scores A[m], selected chunks sel[k], out[S][Hq][d])."""
    s = shape
    q = _arr(q, s, s.n_suffix * s.n_q_heads * s.head_dim, "q")
    kp = _arr(k_prefix, s, s.n_prefix * s.n_kv_heads * s.head_dim, "k_prefix")
    vp = _arr(v_prefix, s, s.n_prefix * s.n_kv_heads * s.head_dim, "v_prefix")
    ks = _arr(k_suffix, s, s.n_suffix * s.n_kv_heads * s.head_dim, "k_suffix")
    vs = _arr(v_suffix, s, s.n_suffix * s.n_kv_heads * s.head_dim, "v_suffix")
    m = s.n_chunks
    A = np.zeros(m, np.float64)
    sel = np.zeros(m, np.int32)
    kk = ctypes.c_int64(0)
    out = np.zeros((s.n_suffix, s.n_q_heads, s.head_dim), np.float64)
    _check(lib().ckvo_reprefill_layer(ctypes.byref(s.c()), keep_ratio, _ptr(q), _ptr(kp), _ptr(vp),
                                      _ptr(ks), _ptr(vs), _ptr(A), _ptr(sel), ctypes.byref(kk),
                                      _ptr(out), threads), "reprefill_layer")
    return A, sel[: kk.value].copy(), out


def io_account(n: int, c: int, sel, block_tokens: int) -> dict:
    """Tokens a ContiguousChunk store reads for the chunk set `sel` against a
    store of fixed `block_tokens`-token blocks (Sec. 4.2; Sec. 3)."""
    sel = np.ascontiguousarray(sel, np.int32)
    out = _IoCounts()
    _check(lib().ckvo_io_account(n, c, _ptr(sel), sel.size, block_tokens, ctypes.byref(out)),
           "io_account")
    return {f: int(getattr(out, f)) for f, _ in _IoCounts._fields_}


CACHE_ATTENTION, CACHE_LFU, CACHE_LOADS = 0, 1, 2
TIER_NONE, TIER_CPU, TIER_GPU = 0, 1, 2


class Cache:
    """Attention-guided two-tier cache of Sec. 4.5 (Eq. 2); see ckv_oracle.h."""

    def __init__(self, n_keys: int, gpu_slots: int, cpu_slots: int, policy: int = CACHE_ATTENTION):
        self.n_keys = n_keys
        self._h = lib().ckvo_cache_create(n_keys, gpu_slots, cpu_slots, policy)
        if not self._h:
            raise OracleError("cache_create failed")

    def access(self, keys, scores):
        """One request's used chunks; returns (tier each key was found in, totals)."""
        keys = np.ascontiguousarray(keys, np.int64)
        scores = np.ascontiguousarray(scores, np.float64)
        if keys.size != scores.size:
            raise ValueError("keys and scores differ in length")
        where = np.zeros(keys.size, np.int8)
        cnt = _CacheCounts()
        _check(lib().ckvo_cache_access(self._h, _ptr(keys), _ptr(scores), keys.size, _ptr(where),
                                       ctypes.byref(cnt)), "cache_access")
        return where, {f: int(getattr(cnt, f)) for f, _ in _CacheCounts._fields_}

    def state(self):
        """(I, F, tier) arrays over every key."""
        I = np.zeros(self.n_keys, np.float64)
        F = np.zeros(self.n_keys, np.int64)
        tier = np.zeros(self.n_keys, np.int8)
        _check(lib().ckvo_cache_state(self._h, _ptr(I), _ptr(F), _ptr(tier)), "cache_state")
        return I, F, tier

    def close(self) -> None:
        if self._h:
            lib().ckvo_cache_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
