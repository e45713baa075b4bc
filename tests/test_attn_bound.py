"""The attention check of the GPU tests (gpu_common.attn_check) on the CPU: an
emulation of the kernels' roundings (numerators rounded to bf16 for the P V
product with an unrounded denominator, the output rounded to bf16) stays
inside the bound (0.22 of it here), and the same pipeline with three bits
fewer in the numerators, the output or both fails it (1.2-1.8 times the bound):
the check sees a loss of precision of that size."""
import numpy as np
import pytest

import oracle
import synth
from gpu_common import attn_check, oshape


def _round_bits(x: np.ndarray, bits: int) -> np.ndarray:
    """x rounded to `bits` significant bits, ties to even (bits = 8: bf16)."""
    m, e = np.frexp(x)
    return np.ldexp(np.round(m * 2.0 ** bits) / 2.0 ** bits, e)


def _f64(bits: np.ndarray) -> np.ndarray:
    return (bits.astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def _emulate(w, t, sel, p_bits: int, out_bits: int) -> np.ndarray:
    q, kp, vp = _f64(t["q"]), _f64(t["k_prefix"]), _f64(t["v_prefix"])
    ks, vs = _f64(t["k_suffix"]), _f64(t["v_suffix"])
    c = w.chunk_size
    rows = np.concatenate([np.arange(j * c, min((j + 1) * c, w.n_prefix)) for j in sel])
    G = w.n_q_heads // w.n_kv_heads
    scale = w.sm_scale or 1.0 / np.sqrt(w.head_dim)
    out = np.zeros((w.n_suffix, w.n_q_heads, w.head_dim))
    for tq in range(w.n_suffix):
        for h in range(w.n_q_heads):
            g = h // G
            K = np.concatenate([kp[rows, g], ks[:tq + 1, g]])
            V = np.concatenate([vp[rows, g], vs[:tq + 1, g]])
            s = (K @ q[tq, h]) * scale
            p = np.exp(s - s.max())
            out[tq, h] = _round_bits((_round_bits(p, p_bits) @ V) / p.sum(), out_bits)
    return out


@pytest.fixture(scope="module")
def case():
    w = synth.WORKLOADS["c3_qwen7b_32k"].scaled(n_prefix=1024, n_suffix=12, n_layers=1)
    t = synth.layer_tensors(w, 0, synth.heavy_sets(w)[0])
    k = max(1, int(round(w.keep_ratio * w.n_chunks)))
    sel = np.sort(np.random.default_rng(3).choice(w.n_chunks, k, replace=False)).astype(np.int32)
    s = oshape(w)
    ref = oracle.sparse_attn(s, t["q"], t["k_prefix"], t["v_prefix"], sel, t["k_suffix"], t["v_suffix"])
    return w, t, sel, s, ref


def test_bf16_pipeline_within_bound(case):
    w, t, sel, s, ref = case
    _, ratio = attn_check(s, t, sel, _emulate(w, t, sel, 8, 8), ref)
    assert 0.01 < ratio < 0.6


@pytest.mark.parametrize("p_bits,out_bits", [(5, 8), (8, 5), (5, 5)])
def test_coarser_pipeline_fails(case, p_bits, out_bits):
    w, t, sel, s, ref = case
    with pytest.raises(AssertionError, match="exceeds its bound"):
        attn_check(s, t, sel, _emulate(w, t, sel, p_bits, out_bits), ref)
