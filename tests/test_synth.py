"""The seeded workload generator: determinism, shapes and the planted-chunk recipe."""
import numpy as np

import synth


def test_bf16_round_to_nearest_even():
    x = np.array([1.0, 1.0 + 2**-8, 1.0 + 2**-7, 1.0 + 3 * 2**-8, -2.5, 0.0], np.float32)
    b = synth.to_bf16_bits(x)
    # 1+2^-8 is a tie between 1 and 1+2^-7: even mantissa (1.0) wins; 1+3*2^-8 ties up to 1+2^-6
    assert synth.bf16_bits_to_f32(b).tolist() == [1.0, 1.0, 1.0 + 2**-7, 1.0 + 2**-6, -2.5, 0.0]


def test_workload_table():
    w = synth.WORKLOADS
    assert w["c1_f32_1k"].n_chunks == 64 and w["c2_qwen05b_8k"].n_chunks == 512
    assert w["c3_qwen7b_32k"].n_chunks == 1024 and w["c5_qwen32b_128k_host"].n_chunks == 4096
    assert [w[f"c4_qwen14b_64k_c{c}"].n_chunks for c in (8, 16, 32, 64)] == [8192, 4096, 2048, 1024]
    assert w["c3_qwen7b_32k"].group == 7 and w["c4_qwen14b_64k_c8"].group == 5


def test_deterministic_and_layer_independent():
    w = synth.WORKLOADS["c2_qwen05b_8k"].scaled(n_prefix=256, n_suffix=8, n_layers=3)
    a = synth.layer_tensors(w, 2)
    b = synth.all_layers(w, layers=[0, 2], threads=2)[1]
    for k in a:
        assert np.array_equal(a[k], b[k]), k
    assert a["q"].dtype == np.uint16 and a["q"].shape == (8, 14, 64)
    assert a["k_prefix"].shape == (256, 2, 64)


def test_heavy_sets_drift():
    w = synth.WORKLOADS["c3_qwen7b_32k"]
    hs = synth.heavy_sets(w)
    assert len(hs) == w.n_layers and all(len(h) == 51 for h in hs)
    for a, b in zip(hs, hs[1:]):
        assert len(set(a.tolist()) & set(b.tolist())) == 51 - 8  # round(0.15*51) replaced
    w4 = synth.WORKLOADS["c4_qwen14b_64k_c8"]
    h4 = synth.heavy_sets(w4)
    assert all(len(h) >= 0.05 * w4.n_chunks * 0.9 for h in h4)
    runs = np.split(h4[0], np.flatnonzero(np.diff(h4[0]) != 1) + 1)
    assert max(len(r) for r in runs) <= 8 and min(len(r) for r in runs) >= 1


def test_planted_keys_align_with_queries():
    w = synth.WORKLOADS["c1_f32_1k"]
    t = synth.layer_tensors(w, 0)
    heavy = synth.heavy_sets(w)[0]
    qbar = t["q"].mean(axis=(0, 1))
    k = t["k_prefix"][:, 0, :]
    proj = k @ qbar
    tok = np.concatenate([np.arange(j * 16, j * 16 + 16) for j in heavy])
    assert proj[tok].mean() > proj.mean() + 1.0


def test_request_queries():
    """Request 0 is the layer's own Q; other requests draw other noise around the
    same per-group directions, deterministically."""
    w = synth.WORKLOADS["c2_qwen05b_8k"].scaled(n_layers=2, n_prefix=256)
    assert np.array_equal(synth.request_queries(w, 1, 0), synth.layer_tensors(w, 1)["q"])
    a, b = synth.request_queries(w, 1, 2), synth.request_queries(w, 1, 2)
    assert np.array_equal(a, b)
    c = synth.request_queries(w, 1, 3)
    assert (a != c).mean() > 0.9
    # the planted direction is shared: group means agree far better than noise would
    fa = synth.bf16_bits_to_f32(a).mean(axis=0)
    fc = synth.bf16_bits_to_f32(c).mean(axis=0)
    assert np.abs(fa - fc).max() < 0.5 and np.abs(fa).max() > 0.05
