"""Randomized parity of the caller-given prediction (ckv_layer_io.pred_idx,
Sec. 4.3.2) on the host-resident layer step: seeded shapes, three layers per
case, each given a prediction of random size that mixes chunks of the
oracle's set with chunks outside it (from none to all of either).  Every
layer's set must be the oracle's selection from the GPU's own scores, its
output within its bound, and its hits, misses, wasted chunks and prefetched
and demand bytes equal to the oracle's set algebra for that prediction."""
from dataclasses import replace

import numpy as np
import pytest
import torch

import oracle
import synth
from gpu_common import (DEV, SCORE_RTOL_BOUND, attn_check, check_set, dev, dims_of, oshape,
                        rel_err, to_f64)

pytestmark = pytest.mark.gpu

N_CASES = 12
SEED0 = 8800


def _case(seed: int):
    rng = np.random.default_rng(seed)
    base = synth.WORKLOADS["c2_qwen05b_8k"]
    d = int(rng.choice([64, 128]))
    c = int(rng.choice([4, 8, 16, 32, 64] + ([96] if d == 128 else [])))
    hkv, G = int(rng.choice([1, 2, 4])), int(rng.choice([1, 2, 5, 7]))
    S = int(rng.integers(1, 33))
    n = int(rng.integers(c, 3001))
    m = -(-n // c)
    keep = float(rng.choice([0.5 / m, 0.1, 0.37, 1.0]))
    w = replace(base, name=f"random_pred{seed}", n_layers=3, n_prefix=n, n_suffix=S,
                n_q_heads=hkv * G, n_kv_heads=hkv, head_dim=d, chunk_size=c, keep_ratio=keep,
                seed=1900 + seed % 100)
    return w, rng


def _pinned(w, t):
    cm = synth.chunk_major(t["k_prefix"], t["v_prefix"], w.chunk_size)
    h = torch.from_numpy(cm.reshape(-1))
    if cm.dtype == np.uint16:
        h = h.view(torch.bfloat16)
    return h.pin_memory()


@pytest.mark.parametrize("seed", [SEED0 + i for i in range(N_CASES)])
def test_random_prediction(seed):
    import paper_2601_13631_amd as ckv
    w, rng = _case(seed)
    m = w.n_chunks
    print(f"seed {seed}: n {w.n_prefix} S {w.n_suffix} Hq {w.n_q_heads} Hkv {w.n_kv_heads} "
          f"d {w.head_dim} c {w.chunk_size} keep {w.keep_ratio:.4f}", flush=True)
    s = oshape(w)
    hs = synth.heavy_sets(w)
    layers = [synth.layer_tensors(w, l, hs[l]) for l in range(w.n_layers)]
    ctx = ckv.Context(dims_of(w), w.n_layers, w.keep_ratio, ckv.CTX_HOST_PREFIX)
    k = ctx.k
    for l, t in enumerate(layers):
        A_ref = oracle.chunk_scores(s, oracle.token_importance(s, t["q"], t["k_prefix"]))
        inside = oracle.select_topk(A_ref, k)
        outside = np.setdiff1d(np.arange(m, dtype=np.int32), inside)
        q = int(rng.integers(0, k + 1))
        r = int(rng.integers(0, min(k - q, outside.size) + 1))
        pred = np.sort(np.concatenate([rng.choice(inside, q, replace=False),
                                       rng.choice(outside, r, replace=False)])).astype(np.int32)
        tt = {kk: dev(v) for kk, v in t.items()}
        store = _pinned(w, t)  # held until the layer's copies have run
        A = torch.empty(m, dtype=torch.float64, device=DEV)
        sel = torch.empty(k, dtype=torch.int32, device=DEV)
        out = torch.empty_like(tt["q"])
        st = ctx.reprefill_layer(l, tt["q"], tt["k_suffix"], tt["v_suffix"], tt["k_prefix"], out,
                                 kv_host=store, chunk_scores=A, sel_idx=sel, pred_idx=pred)
        torch.cuda.synchronize()
        A, sel = A.cpu().numpy(), sel.cpu().numpy()
        err = rel_err(A, A_ref)
        assert err <= SCORE_RTOL_BOUND, (l, err)  # see test_gpu_random
        check_set(A_ref, sel, k, err, require=False)
        assert np.array_equal(oracle.select_topk(A, k), sel)
        ref = oracle.sparse_attn(s, t["q"], t["k_prefix"], t["v_prefix"], sel, t["k_suffix"],
                                 t["v_suffix"])
        aerr, ratio = attn_check(s, t, sel, to_f64(out).reshape(ref.shape), ref)
        acc = oracle.layer_accounting(s, sel, pred)
        for f in ("hits", "misses", "wasted", "bytes_prefetch", "bytes_demand"):
            assert st[f] == acc[f], (l, f, st[f], acc[f])
        print(f"  layer {l}: k {k} prediction {pred.size} ({q} of the set) hits {st['hits']} "
              f"misses {st['misses']} attn max abs {aerr:.2e} ({ratio:.2f} of its bound)", flush=True)
    ctx.close()
