"""Randomized parity of the host-resident layer step with Periods and the
attention-guided cache: seeded shapes (as in test_gpu_random), a Period of 1
to 3 layers, with or without a cache of random tier sizes, two requests of 4
layers each.  Every layer's set must be the Period's (selected at its first
layer, certified against the oracle or inside the near-tie band) and its
output within its bound of the oracle's attention over that set; the cache
changes only where the chunk bytes come from."""
from dataclasses import replace

import numpy as np
import pytest
import torch

import oracle
import synth
from gpu_common import (DEV, SCORE_RTOL_BOUND, attn_check, check_set, dev, dims_of, oshape,
                        rel_err, to_f64)

pytestmark = pytest.mark.gpu

N_CASES = 24
SEED0 = 3100


def _case(i: int):
    rng = np.random.default_rng(SEED0 + i)
    base = synth.WORKLOADS["c2_qwen05b_8k"]
    d = int(rng.choice([64, 128]))
    c = int(rng.choice([4, 8, 16, 32, 64] + ([96] if d == 128 else [])))
    hkv, G = int(rng.choice([1, 2, 4])), int(rng.choice([1, 2, 5, 7]))
    S = int(rng.integers(1, 33))
    n = int(rng.integers(c, 3001))
    m = -(-n // c)
    keep = float(rng.choice([0.5 / m, 0.1, 0.37, 1.0]))
    period = int(rng.integers(1, 4))
    cache = bool(rng.integers(0, 2))
    w = replace(base, name=f"random_host{i}", n_layers=4, n_prefix=n, n_suffix=S,
                n_q_heads=hkv * G, n_kv_heads=hkv, head_dim=d, chunk_size=c, keep_ratio=keep,
                seed=500 + i)
    gpu_frac, cpu_frac = float(rng.choice([0.1, 0.5, 1.0])), float(rng.choice([0.5, 1.0, 2.0]))
    return w, period, cache, gpu_frac, cpu_frac


def _store(w, t):
    cm = synth.chunk_major(t["k_prefix"], t["v_prefix"], w.chunk_size)
    h = torch.from_numpy(cm.reshape(-1))
    if cm.dtype == np.uint16:
        h = h.view(torch.bfloat16)
    return h.pin_memory()


@pytest.mark.parametrize("i", range(N_CASES))
def test_random_host_layer_step(i):
    import paper_2601_13631_amd as ckv
    w, period, with_cache, gpu_frac, cpu_frac = _case(i)
    L, m = w.n_layers, w.n_chunks
    print(f"case {i}: n {w.n_prefix} S {w.n_suffix} Hq {w.n_q_heads} Hkv {w.n_kv_heads} "
          f"d {w.head_dim} c {w.chunk_size} keep {w.keep_ratio:.4f} period {period} "
          f"cache {with_cache} ({gpu_frac}, {cpu_frac})", flush=True)
    s = oshape(w)
    hs = synth.heavy_sets(w)
    layers = [synth.layer_tensors(w, l, hs[l]) for l in range(L)]
    stores = [_store(w, t) for t in layers]
    base = [{kk: dev(v) for kk, v in t.items()} for t in layers]
    ctx = ckv.Context(dims_of(w), L, w.keep_ratio, ckv.CTX_HOST_PREFIX)
    ctx.set_period(period)
    k = ctx.k
    cache = None
    if with_cache:
        cache = ckv.Cache(L * m, max(1, int(gpu_frac * L * k)), max(1, int(cpu_frac * L * k)))
        ctx.attach_cache(cache)
    for r in range(2):
        ctx.reset()
        sets = {}
        for l in range(L):
            first = l - l % period
            t = dict(layers[l], q=synth.request_queries(w, l, r))
            q = dev(t["q"])
            A = torch.full((m,), float("nan"), dtype=torch.float64, device=DEV)
            sel = torch.empty(k, dtype=torch.int32, device=DEV)
            out = torch.empty_like(q)
            ctx.reprefill_layer(l, q, base[l]["k_suffix"], base[l]["v_suffix"], base[l]["k_prefix"],
                                out, kv_host=stores[l], kv_host_next=stores[l + 1] if l + 1 < L else None,
                                chunk_scores=A, sel_idx=sel)
            torch.cuda.synchronize()
            A, sel = A.cpu().numpy(), sel.cpu().numpy()
            if l == first:
                A_ref = oracle.chunk_scores(s, oracle.token_importance(s, t["q"], t["k_prefix"]))
                err = rel_err(A, A_ref)
                assert err <= SCORE_RTOL_BOUND, (r, l, err)  # see test_gpu_random
                check_set(A_ref, sel, k, err, require=False)
                assert np.array_equal(oracle.select_topk(A, k), sel)
                sets[first] = sel
            else:
                assert np.isnan(A).all()  # no scoring inside a Period
                assert np.array_equal(sel, sets[first]), (r, l)
            ref = oracle.sparse_attn(s, t["q"], t["k_prefix"], t["v_prefix"], sets[first],
                                     t["k_suffix"], t["v_suffix"])
            aerr, ratio = attn_check(s, t, sets[first], to_f64(out).reshape(ref.shape), ref)
            print(f"  request {r} layer {l}: attn max abs {aerr:.2e} ({ratio:.2f} of its bound)",
                  flush=True)
    ctx.reset()
    if cache is not None:
        ctx.attach_cache(None)
        cache.close()
    ctx.close()
