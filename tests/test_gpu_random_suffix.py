"""Randomized parity of the layer step with long suffixes: 49 to 400 new
tokens with 1 to 7 query heads per KV head, so a KV head's rows span up to
22 row blocks of the attention and the causal mask over the suffix crosses
row-block and split boundaries at random offsets.  Same checks as
test_gpu_random."""
from dataclasses import replace

import numpy as np
import pytest

import synth
from test_gpu_random import run_layers

pytestmark = pytest.mark.gpu

N_CASES = 8
SEED0 = 7500


def _case(seed: int):
    rng = np.random.default_rng(seed)
    base = synth.WORKLOADS["c2_qwen05b_8k"]
    d = int(rng.choice([64, 128]))
    c = int(rng.choice([4, 8, 16, 32, 64] + ([96] if d == 128 else [])))
    hkv, G = int(rng.choice([1, 2, 4])), int(rng.choice([1, 2, 5, 7]))
    S = int(rng.integers(49, 401))
    n = int(rng.integers(c, 2001))
    m = -(-n // c)
    keep = float(rng.choice([0.5 / m, 0.1, 0.37, 1.0]))
    w = replace(base, name=f"random_suffix{seed}", n_layers=2, n_prefix=n, n_suffix=S,
                n_q_heads=hkv * G, n_kv_heads=hkv, head_dim=d, chunk_size=c, keep_ratio=keep,
                seed=1700 + seed % 100)
    return w, ("host" if seed % 2 else "hbm")


@pytest.mark.parametrize("seed", [SEED0 + i for i in range(N_CASES)])
def test_random_suffix_layer_step(seed):
    w, path = _case(seed)
    print(f"seed {seed}", end=" ")
    run_layers(w, path)
