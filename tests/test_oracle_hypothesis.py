"""The oracle on hypothesis-generated tiny shapes: partial last chunks, ties,
Hq = Hkv, head_dim not a power of two, k = 1 and k = m.

Each property is pinned to something outside the oracle: torch's fp64 softmax
and scaled_dot_product_attention, numpy's lexsort, or an exact invariant
(Eq. 1 sums to S * Hq; keeping every chunk is dense attention, bit for bit).
"""
import numpy as np
import torch
from hypothesis import given, settings, strategies as st

import oracle
from oracle import BF16, F32, Shape
from oracle_pins import _f64, _inputs, _scale, _sdpa


@st.composite
def shapes(draw):
    Hkv = draw(st.integers(1, 3))
    G = draw(st.integers(1, 3))
    return Shape(draw(st.integers(1, 48)), draw(st.integers(1, 4)), Hkv * G, Hkv,
                 draw(st.integers(1, 9)), draw(st.integers(1, 9)), draw(st.sampled_from([BF16, F32])),
                 draw(st.sampled_from([0.0, 0.3])))


@settings(max_examples=60, deadline=None)
@given(s=shapes(), seed=st.integers(0, 2**31 - 1))
def test_importance_and_chunk_scores(s, seed):
    """Token importance equals torch's fp64 softmax summed over every query row
    of every head; chunk scores pool it per chunk and sum to S * Hq (Eq. 1)."""
    x = _inputs(s, seed)
    a = oracle.token_importance(s, x["q"], x["kp"])
    q = torch.from_numpy(_f64(x["q"], s.dtype))
    k = torch.from_numpy(_f64(x["kp"], s.dtype))
    G = s.n_q_heads // s.n_kv_heads
    ref = torch.zeros(s.n_prefix, dtype=torch.float64)
    for h in range(s.n_q_heads):
        ref += torch.softmax(_scale(s) * (q[:, h, :] @ k[:, h // G, :].T), dim=-1).sum(0)
    assert np.allclose(a, ref.numpy(), rtol=1e-12, atol=1e-15)
    A = oracle.chunk_scores(s, a)
    assert A.size == -(-s.n_prefix // s.chunk_size)
    pooled = np.add.reduceat(ref.numpy(), np.arange(0, s.n_prefix, s.chunk_size))
    assert np.allclose(A, pooled, rtol=1e-12, atol=1e-15)
    assert abs(A.sum() - s.n_suffix * s.n_q_heads) <= 1e-12 * s.n_suffix * s.n_q_heads


@settings(max_examples=200, deadline=None)
@given(scores=st.lists(st.sampled_from([0.0, -0.0, 0.5, 1.0, 1.0, 2.0, 7.25, np.inf, -np.inf]),
                       min_size=1, max_size=40),
       data=st.data())
def test_select_matches_lexsort(scores, data):
    """Top-k under (score descending, index ascending), returned ascending,
    against a lexsort; heavy ties and signed zeros included."""
    A = np.array(scores, np.float64)
    k = data.draw(st.integers(1, A.size))
    order = np.lexsort((np.arange(A.size), -(A + 0.0)))  # -0.0 and 0.0 compare equal
    assert oracle.select_topk(A, k).tolist() == sorted(order[:k].tolist())


@settings(max_examples=40, deadline=None)
@given(s=shapes(), seed=st.integers(0, 2**31 - 1), data=st.data())
def test_sparse_attention_matches_sdpa(s, seed, data):
    """Sparse prefill attention (Def. 2.1) equals torch fp64 SDPA over [prefix ;
    suffix] with the kept chunks visible and the suffix causal; keeping every
    chunk is the dense path bit for bit."""
    x = _inputs(s, seed)
    m = s.n_chunks
    sel = np.array(sorted(data.draw(st.sets(st.integers(0, m - 1), min_size=1, max_size=m))),
                   np.int32)
    vis = np.zeros(s.n_prefix, bool)
    for j in sel:
        vis[j * s.chunk_size:(j + 1) * s.chunk_size] = True
    got = oracle.sparse_attn(s, x["q"], x["kp"], x["vp"], sel, x["ks"], x["vs"])
    assert np.allclose(got, _sdpa(s, x, vis), rtol=0, atol=1e-12)
    every = np.arange(m, dtype=np.int32)
    assert np.array_equal(oracle.sparse_attn(s, x["q"], x["kp"], x["vp"], every, x["ks"], x["vs"]),
                          oracle.dense_attn(s, x["q"], x["kp"], x["vp"], x["ks"], x["vs"]))
