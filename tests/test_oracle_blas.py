"""Pins of the oracle's matrix-product form (``oracle/blas.py``).

It is held to the same outside facts as the scalar oracle -- the hand-worked
examples, the invariants of a softmax, special cases with closed forms -- and
to the scalar C oracle (itself pinned in ``oracle_pins.py``) on random GQA
shapes, bf16 and fp32, across several row blocks.  A set of plausible
mistakes planted in copies of its source must each fail a pin.
"""
import math
import os
import types

import numpy as np
import pytest

import oracle
import oracle.blas as blas
from oracle import BF16, F32, Shape
from oracle_pins import SHAPES, _inputs

E = math.e
SRC = os.path.join(os.path.dirname(oracle.__file__), "blas.py")


def _pin_h1(B):
    """q = [1], keys 0, 0, 1, 1, c = 2: weights 1, 1, e, e over 2 + 2e."""
    s = Shape(4, 1, 1, 1, 1, 2, F32, 1.0)
    a = B.token_importance(s, np.array([1.0], np.float32), np.array([0, 0, 1, 1], np.float32))
    assert np.allclose(B.chunk_scores(s, a), [1 / (1 + E), E / (1 + E)], rtol=1e-15, atol=0)
    a0 = B.token_importance(s, np.array([1.0], np.float32), np.zeros(4, np.float32))
    assert B.chunk_scores(s, a0).tolist() == [0.5, 0.5]


def _pin_h1_attention(B):
    """Keys 0, 0, 1, 1 with values 1..4, suffix key 0 with value 10: keeping
    chunk 1 gives (7e + 10)/(2e + 1); keeping both chunks (dense) gives
    (13 + 7e)/(3 + 2e)."""
    s = Shape(4, 1, 1, 1, 1, 2, F32, 1.0)
    q = np.array([1.0], np.float32)
    kp = np.array([0, 0, 1, 1], np.float32)
    vp = np.array([1, 2, 3, 4], np.float32)
    ks, vs = np.array([0.0], np.float32), np.array([10.0], np.float32)
    o1 = B.sparse_attn(s, q, kp, vp, [1], ks, vs).ravel()[0]
    assert abs(o1 - (7 * E + 10) / (2 * E + 1)) < 1e-14, o1
    o2 = B.sparse_attn(s, q, kp, vp, [0, 1], ks, vs).ravel()[0]
    assert abs(o2 - (13 + 7 * E) / (3 + 2 * E)) < 1e-14, o2


def _pin_invariants(B):
    """Every softmax row sums to 1, so sum_j A_j = S * Hq; with q = 0 every row
    is uniform, A_j = S * Hq * |chunk j| / n.  Constant V gives that constant;
    the first query with no chunk kept sees only itself."""
    for i, s in enumerate(SHAPES):
        x = _inputs(s, 300 + i)
        rows = s.n_suffix * s.n_q_heads
        A = B.chunk_scores(s, B.token_importance(s, x["q"], x["kp"]))
        assert abs(A.sum() - rows) <= 1e-12 * rows
        A0 = B.chunk_scores(s, B.token_importance(s, np.zeros_like(x["q"]), x["kp"]))
        lens = np.minimum(s.chunk_size, s.n_prefix - np.arange(s.n_chunks) * s.chunk_size)
        assert np.allclose(A0, rows * lens / s.n_prefix, rtol=1e-12, atol=0)
        const = np.full_like(x["vp"], 0x3FC0 if s.dtype == BF16 else 1.5)  # 1.5
        o = B.sparse_attn(s, x["q"], x["kp"], const, np.arange(s.n_chunks, dtype=np.int32),
                          x["ks"], np.full_like(x["vs"], const.flat[0]))
        assert np.allclose(o, 1.5, rtol=0, atol=1e-14)
        o0 = B.sparse_attn(s, x["q"], x["kp"], x["vp"], [], x["ks"], x["vs"])
        vs = oracle.blas._widen(x["vs"], s.dtype).numpy().reshape(s.n_suffix, s.n_kv_heads, -1)
        G = s.n_q_heads // s.n_kv_heads
        for h in range(s.n_q_heads):
            assert np.array_equal(o0[0, h], vs[0, h // G])


def _pin_vs_scalar_oracle(B, block_elems=None):
    """Agreement with the pinned scalar C oracle on random GQA shapes (bf16
    and fp32, ragged chunks), also with the logit matrix cut into many row
    blocks."""
    old = B._ROW_BLOCK_ELEMS
    if block_elems is not None:
        B._ROW_BLOCK_ELEMS = block_elems
    try:
        for i, s in enumerate(SHAPES + [Shape(300, 7, 6, 2, 16, 8, BF16), Shape(130, 9, 4, 4, 8, 32, F32)]):
            x = _inputs(s, 400 + i)
            a_ref = oracle.token_importance(s, x["q"], x["kp"])
            a = B.token_importance(s, x["q"], x["kp"])
            assert np.allclose(a, a_ref, rtol=1e-12, atol=1e-300), (s, np.abs(a - a_ref).max())
            A_ref = oracle.chunk_scores(s, a_ref)
            assert np.allclose(B.chunk_scores(s, a_ref), A_ref, rtol=1e-14, atol=0)
            rng = np.random.default_rng(i)
            kk = max(1, s.n_chunks // 2)
            sel = np.sort(rng.choice(s.n_chunks, size=kk, replace=False)).astype(np.int32)
            o_ref = oracle.sparse_attn(s, x["q"], x["kp"], x["vp"], sel, x["ks"], x["vs"])
            o = B.sparse_attn(s, x["q"], x["kp"], x["vp"], sel, x["ks"], x["vs"])
            assert np.allclose(o, o_ref, rtol=0, atol=1e-12), (s, np.abs(o - o_ref).max())
    finally:
        B._ROW_BLOCK_ELEMS = old


PINS = {
    "h1_scores": _pin_h1,
    "h1_attention": _pin_h1_attention,
    "invariants": _pin_invariants,
    "vs_scalar_oracle": _pin_vs_scalar_oracle,
    "vs_scalar_oracle_row_blocks": lambda B: _pin_vs_scalar_oracle(B, block_elems=64),
}


@pytest.mark.parametrize("name", list(PINS))
def test_blas_pin(name):
    PINS[name](blas)


MUTANTS = {
    "score_scale_dropped": ("logits = (Qg[r0:r0 + block] @ Kg.T) * sc", "logits = (Qg[r0:r0 + block] @ Kg.T)"),
    "score_gqa_mapping": ("Qg = Q[:, g * G:(g + 1) * G, :].reshape(S * G, d)           # rows",
                          "Qg = Q[:, g::Hkv, :].reshape(S * G, d)           # rows"),
    "score_not_normalised": ("p = e / e.sum(dim=1, keepdim=True)", "p = e"),
    "score_max_wrong_axis": ("mx = logits.max(dim=1, keepdim=True).values\n            e = torch.exp(logits - mx)\n            p",
                             "mx = logits.max(dim=0, keepdim=True).values\n            e = torch.exp(logits - mx)\n            p"),
    "pooling_drops_last_token": ("padded[:n] = a", "padded[:n - 1] = a[:-1]"),
    "attn_diagonal_hidden": ("hidden = torch.arange(S)[None, :] > t_of_row", "hidden = torch.arange(S)[None, :] >= t_of_row"),
    "attn_not_causal": ("logits[:, T:][hidden] = -math.inf", "pass"),
    "attn_scale_dropped": ("logits = (Qg[r0:r1] @ Kall.T) * sc", "logits = (Qg[r0:r1] @ Kall.T)"),
    "attn_values_are_keys": ("og[r0:r1] = (e @ Vall)", "og[r0:r1] = (e @ Kall)"),
    "attn_chunk_tail_dropped": ("np.arange(j * c, min(j * c + c, n))", "np.arange(j * c, min(j * c + c, n) - 1)"),
    "bf16_widen_shift": ("a.astype(np.uint32) << 16", "a.astype(np.uint32) << 15"),
}


def _mutant_module(old: str, new: str):
    src = open(SRC).read()
    assert src.count(old) == 1, old
    src = src.replace(old, new).replace("from . import BF16, Shape", "from oracle import BF16, Shape")
    mod = types.ModuleType("blas_mutant")
    exec(compile(src, "blas_mutant", "exec"), mod.__dict__)
    return mod


@pytest.mark.parametrize("name", list(MUTANTS))
def test_blas_mutant_caught(name):
    mod = _mutant_module(*MUTANTS[name])
    caught = []
    for pin, f in PINS.items():
        try:
            f(mod)
        except (AssertionError, IndexError, RuntimeError, ValueError):
            caught.append(pin)
    assert caught, f"mutant {name} passes every pin"
