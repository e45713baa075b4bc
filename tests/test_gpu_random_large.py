"""Randomized parity of the layer step on long prefixes cut into many small
chunks: 2,048 to 12,000 chunks, so the per-chunk reduction takes its
many-chunk form (from 4,096 chunks), the selection its LDS-cached block form
(above 8,192) and the host path's copies and parted attention hundreds to
thousands of chunks.  Same checks as test_gpu_random."""
from dataclasses import replace

import numpy as np
import pytest

import synth
from test_gpu_random import run_layers

pytestmark = pytest.mark.gpu

N_CASES = 10
SEED0 = 6400


def _case(seed: int):
    rng = np.random.default_rng(seed)
    base = synth.WORKLOADS["c2_qwen05b_8k"]
    d = int(rng.choice([64, 128]))
    c = int(rng.choice([4, 8]))
    hkv, G = int(rng.choice([1, 2])), int(rng.choice([1, 2, 4]))
    S = int(rng.integers(1, 17))
    n = c * int(rng.integers(2048, 12001)) - int(rng.integers(0, c))  # ragged last chunk
    keep = float(rng.choice([0.01, 0.1, 0.5]))
    w = replace(base, name=f"random_large{seed}", n_layers=2, n_prefix=n, n_suffix=S,
                n_q_heads=hkv * G, n_kv_heads=hkv, head_dim=d, chunk_size=c, keep_ratio=keep,
                seed=1300 + seed % 100)
    return w, ("host" if seed % 2 else "hbm")


@pytest.mark.parametrize("seed", [SEED0 + i for i in range(N_CASES)])
def test_random_large_layer_step(seed):
    w, path = _case(seed)
    print(f"seed {seed}", end=" ")
    run_layers(w, path)
