"""Randomized parity of the layer step run without any host synchronisation
between layers: seeded shapes, a Period of 1 to 4 layers, the chunks coming
from per-call pinned stores, from stores registered for every layer (the
Period's copies queued at its first layer, a SubPeriod of 1 to 3), from a
file through the storage tier (each with or without the attention-guided
cache) or from HBM (read in place or through the materialised copy), two
requests.  Layers inside a Period never wait on the host, so the host runs
ahead of the GPU and rewrites staging lists and pool slots while earlier
layers' copies and attention may still be in flight; every layer's
scores, set and output are read only after the whole request and compared
with the oracle: scores within the derived bound at a Period's first layer,
untouched elsewhere, every set the Period's, every output within its bound."""
from dataclasses import replace

import numpy as np
import pytest
import torch

import oracle
import synth
from gpu_common import (DEV, SCORE_RTOL_BOUND, attn_check, check_set, dev, dims_of, oshape,
                        rel_err, to_f64)

pytestmark = pytest.mark.gpu

N_CASES = 20
SEED0 = 5300


SOURCES = ("pinned", "registered", "store", "hbm", "hbm-copy")


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
    period = int(rng.integers(1, 5))
    source = SOURCES[seed % len(SOURCES)]
    sub = int(rng.integers(1, 4)) if source in ("registered", "store") else 1
    cache = bool(rng.integers(0, 2)) and not source.startswith("hbm")
    L = int(rng.integers(4, 8))
    w = replace(base, name=f"random_async{seed}", n_layers=L, n_prefix=n, n_suffix=S,
                n_q_heads=hkv * G, n_kv_heads=hkv, head_dim=d, chunk_size=c, keep_ratio=keep,
                seed=900 + seed % 100)
    return w, period, source, sub, cache


def _pinned(w, t):
    cm = synth.chunk_major(t["k_prefix"], t["v_prefix"], w.chunk_size)
    h = torch.from_numpy(cm.reshape(-1))
    if cm.dtype == np.uint16:
        h = h.view(torch.bfloat16)
    return h.pin_memory()


@pytest.mark.parametrize("seed", [SEED0 + i for i in range(N_CASES)])
def test_random_async_layer_step(seed, tmp_path):
    import paper_2601_13631_amd as ckv
    w, period, source, sub, with_cache = _case(seed)
    L, m = w.n_layers, w.n_chunks
    print(f"seed {seed}: L {L} n {w.n_prefix} S {w.n_suffix} Hq {w.n_q_heads} Hkv {w.n_kv_heads} "
          f"d {w.head_dim} c {w.chunk_size} keep {w.keep_ratio:.4f} period {period} {source} "
          f"sub {sub} cache {with_cache}", flush=True)
    s = oshape(w)
    hs = synth.heavy_sets(w)
    layers = [synth.layer_tensors(w, l, hs[l]) for l in range(L)]
    flags = {"hbm": 0, "hbm-copy": ckv.CTX_MATERIALIZE}.get(source, ckv.CTX_HOST_PREFIX)
    ctx = ckv.Context(dims_of(w), L, w.keep_ratio, flags)
    ctx.set_period(period)
    k = ctx.k
    stores, store, cache = None, None, None
    if with_cache:
        cache = ckv.Cache(L * m, max(1, k // 2), max(1, L * k // 2))
        ctx.attach_cache(cache)
    if source == "store":
        path = str(tmp_path / "kv.bin")
        with open(path, "wb") as f:
            for t in layers:
                synth.chunk_major(t["k_prefix"], t["v_prefix"], w.chunk_size).tofile(f)
        store = ckv.Store(path, L * m, 2 * w.chunk_size * w.n_kv_heads * w.head_dim * w.elem_bytes, 4, 0)
        ctx.set_subperiod(sub)
        ctx.attach_store(store)
    elif not source.startswith("hbm"):
        stores = [_pinned(w, t) for t in layers]
        if source == "registered":
            ctx.set_host_layers(stores)
            ctx.set_subperiod(sub)
    base = [{kk: dev(v) for kk, v in t.items() if kk != "q"} for t in layers]
    for r in range(2):
        # every upload first: a copy from pageable memory would synchronise
        qs = [synth.request_queries(w, l, r) for l in range(L)]
        qd = [dev(q) for q in qs]
        res = [(torch.full((m,), float("nan"), dtype=torch.float64, device=DEV),
                torch.empty(k, dtype=torch.int32, device=DEV), torch.empty_like(q)) for q in qd]
        torch.cuda.synchronize()
        ctx.reset()
        for l in range(L):
            A, sel, out = res[l]
            kw = {}
            if source == "pinned":
                kw = dict(kv_host=stores[l], kv_host_next=stores[l + 1] if l + 1 < L else None)
            elif source.startswith("hbm"):
                kw = dict(k_prefix=base[l]["k_prefix"], v_prefix=base[l]["v_prefix"])
            ctx.reprefill_layer(l, qd[l], base[l]["k_suffix"], base[l]["v_suffix"],
                                base[l]["k_prefix"], out, chunk_scores=A, sel_idx=sel, **kw)
        torch.cuda.synchronize()
        sets = {}
        for l in range(L):
            first = l - l % period
            t = dict(layers[l], q=qs[l])
            A, sel, out = (x.cpu() for x in res[l])
            A, sel = A.numpy(), sel.numpy()
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
    if store is not None:
        ctx.attach_store(None)
        store.close()
    if source == "registered":
        ctx.set_host_layers(None)
    if cache is not None:
        ctx.attach_cache(None)
        cache.close()
    ctx.close()
