"""GPU parity of the whole layer step (ckv_reprefill_layer) against the oracle."""
import numpy as np
import pytest
import torch

import oracle
import synth
from gpu_common import (DEV, SCORE_RTOL_UNIT as SCORE_RTOL, attn_check, check_set, dev, dims_of, oshape,
                        rel_err, to_f64)

pytestmark = pytest.mark.gpu



def small(name, **kw):
    return synth.WORKLOADS[name].scaled(**kw)


HBM_CASES = [
    (synth.WORKLOADS["c1_f32_1k"], 0),
    (small("c2_qwen05b_8k", n_prefix=2000, n_suffix=24, n_layers=3), 0),
    (small("c3_qwen7b_32k", n_prefix=4096, n_suffix=40, n_layers=2), 0),
    (small("c3_qwen7b_32k", n_prefix=4096, n_suffix=40, n_layers=2), 2),  # materialised gather
    (small("c4_qwen14b_64k_c8", n_prefix=3000, n_suffix=20, n_layers=2), 0),
    (small("c3_qwen7b_32k", n_prefix=45, n_suffix=1, n_layers=2), 0),  # m = 2, one query
]


def _oracle_layer(w, t, sel_gpu):
    s = oshape(w)
    A = oracle.chunk_scores(s, oracle.token_importance(s, t["q"], t["k_prefix"]))
    out = oracle.sparse_attn(s, t["q"], t["k_prefix"], t["v_prefix"], sel_gpu, t["k_suffix"],
                             t["v_suffix"])
    return A, out


@pytest.mark.parametrize("w,flags", HBM_CASES, ids=lambda x: getattr(x, "name", str(x)))
def test_layer_hbm_resident(w, flags):
    import paper_2601_13631_amd as ckv
    ctx = ckv.Context(dims_of(w), w.n_layers, w.keep_ratio, flags)
    k = ctx.k
    hs = synth.heavy_sets(w)
    for layer in range(w.n_layers):
        print(f"case {w.name} flags={flags} layer {layer}", flush=True)
        t = synth.layer_tensors(w, layer, hs[layer])
        tt = {kk: dev(v) for kk, v in t.items()}
        A = torch.empty(w.n_chunks, dtype=torch.float64, device=DEV)
        sel = torch.empty(k, dtype=torch.int32, device=DEV)
        out = torch.empty_like(tt["q"])
        st = ctx.reprefill_layer(layer, tt["q"], tt["k_suffix"], tt["v_suffix"], tt["k_prefix"], out,
                                 k_prefix=tt["k_prefix"], v_prefix=tt["v_prefix"], chunk_scores=A,
                                 sel_idx=sel)
        torch.cuda.synchronize()
        assert st["k"] == k
        A, sel = A.cpu().numpy(), sel.cpu().numpy()
        A_ref, out_ref = _oracle_layer(w, t, sel)
        err = rel_err(A, A_ref)
        assert err <= SCORE_RTOL, err
        check_set(A_ref, sel, k, err)
        assert np.all(np.diff(sel) > 0)
        aerr, ratio = attn_check(oshape(w), t, sel, to_f64(out).reshape(out_ref.shape), out_ref)
        print(f"  score rel err {err:.2e}  attn max abs {aerr:.2e} ({ratio:.2f} of its bound)",
              flush=True)
    ctx.close()


def _host_store(w, tensors):
    """Pinned chunk-major store of every layer plus an HBM copy of K for scoring."""
    stores = []
    for t in tensors:
        cm = synth.chunk_major(t["k_prefix"], t["v_prefix"], w.chunk_size)
        h = torch.from_numpy(cm.reshape(-1))
        if cm.dtype == np.uint16:
            h = h.view(torch.bfloat16)
        stores.append(h.pin_memory())
    return stores


@pytest.mark.parametrize("scenario", ["drift", "repeat", "disjoint", "tiny", "d64", "f32"])
def test_layer_host_resident_prefetch(scenario):
    """Host-resident prefix: outputs equal the HBM path's oracle, and the
    hit/miss/byte counts equal the oracle's set algebra with the previous
    layer's selection as the prediction.  "tiny": two chunks (the last one
    partial, kept), one query; "d64": head_dim 64, 7 query heads per KV head,
    16-token chunks; "f32": the fp32 path (one attention launch after the
    demand copy)."""
    import paper_2601_13631_amd as ckv
    if scenario == "tiny":
        w = small("c5_qwen32b_128k_host", n_prefix=45, n_suffix=1, n_layers=3)
    elif scenario == "d64":
        w = small("c2_qwen05b_8k", n_prefix=3000, n_suffix=20, n_layers=4)
    elif scenario == "f32":
        w = small("c1_f32_1k", n_prefix=1000, n_suffix=12, n_layers=3)
    else:
        w = small("c5_qwen32b_128k_host", n_prefix=4096, n_suffix=24, n_layers=4)
    hs = synth.heavy_sets(w)
    if scenario == "repeat":      # identical layers: perfect prediction after layer 0
        layers = [synth.layer_tensors(w, 0, hs[0])] * w.n_layers
    elif scenario == "disjoint":  # heavy sets change completely between layers
        m = w.n_chunks
        blocks = [np.arange(i * 7, m, 4 * 7)[: len(hs[0])] for i in range(w.n_layers)]
        layers = [synth.layer_tensors(w, l, np.sort(blocks[l % 4])) for l in range(w.n_layers)]
    else:
        layers = [synth.layer_tensors(w, l, hs[l]) for l in range(w.n_layers)]
    stores = _host_store(w, layers)
    s = oshape(w)
    ctx = ckv.Context(dims_of(w), w.n_layers, w.keep_ratio, ckv.CTX_HOST_PREFIX)
    k = ctx.k
    prev = np.zeros(0, np.int32)
    for layer, t in enumerate(layers):
        print(f"scenario {scenario} layer {layer}", flush=True)
        tt = {kk: dev(v) for kk, v in t.items()}
        A = torch.empty(w.n_chunks, dtype=torch.float64, device=DEV)
        sel = torch.empty(k, dtype=torch.int32, device=DEV)
        out = torch.empty_like(tt["q"])
        nxt = stores[layer + 1] if layer + 1 < len(stores) else None
        st = ctx.reprefill_layer(layer, tt["q"], tt["k_suffix"], tt["v_suffix"], tt["k_prefix"], out,
                                 kv_host=stores[layer], kv_host_next=nxt, chunk_scores=A, sel_idx=sel)
        torch.cuda.synchronize()
        A, sel = A.cpu().numpy(), sel.cpu().numpy()
        A_ref, out_ref = _oracle_layer(w, t, sel)
        err = rel_err(A, A_ref)
        assert err <= SCORE_RTOL
        check_set(A_ref, sel, k, err)
        aerr, _ = attn_check(s, t, sel, to_f64(out).reshape(out_ref.shape), out_ref)
        acc = oracle.layer_accounting(s, sel, prev)
        assert st["hits"] == acc["hits"] and st["misses"] == acc["misses"]
        assert st["wasted"] == acc["wasted"] and st["bytes_demand"] == acc["bytes_demand"]
        assert st["bytes_gathered"] == acc["bytes_used"]
        if nxt is not None:
            assert st["bytes_prefetch"] == oracle.layer_accounting(s, sel, sel)["bytes_prefetch"]
        if scenario == "repeat" and layer > 0:
            assert st["misses"] == 0 and st["hits"] == k
        if layer == 0:
            assert st["hits"] == 0 and st["misses"] == k
        print(f"  hits {st['hits']} misses {st['misses']} attn err {aerr:.2e}", flush=True)
        prev = sel if nxt is not None else np.zeros(0, np.int32)
    # out-of-order layers are refused; reset starts a request over
    with pytest.raises(ckv.CkvError):
        ctx.reprefill_layer(0, tt["q"], tt["k_suffix"], tt["v_suffix"], tt["k_prefix"], out,
                            kv_host=stores[0])
    ctx.reset()
    st = ctx.reprefill_layer(0, tt["q"], tt["k_suffix"], tt["v_suffix"], tt["k_prefix"], out,
                             kv_host=stores[-1])
    assert st["hits"] == 0 and st["misses"] == k
    ctx.close()


@pytest.mark.parametrize("host", [False, True], ids=["hbm", "host"])
def test_layer_periods(host):
    """Periods of 2 layers (Def. 4.2): layers 0, 2, 4 score and select; layers
    1 and 3 attend over their Period's set without scoring (chunk scores left
    untouched) and, from host memory, with every chunk prefetched."""
    import paper_2601_13631_amd as ckv
    p = 2
    if host:
        w = small("c5_qwen32b_128k_host", n_prefix=4096, n_suffix=24, n_layers=5)
    else:
        w = small("c3_qwen7b_32k", n_prefix=4096, n_suffix=40, n_layers=5)
    hs = synth.heavy_sets(w)
    layers = [synth.layer_tensors(w, l, hs[l]) for l in range(w.n_layers)]
    stores = _host_store(w, layers) if host else None
    s = oshape(w)
    ctx = ckv.Context(dims_of(w), w.n_layers, w.keep_ratio, ckv.CTX_HOST_PREFIX if host else 0)
    ctx.set_period(p)
    k = ctx.k
    sets = [None] * w.n_layers
    prev = np.zeros(0, np.int32)
    for layer, t in enumerate(layers):
        first = oracle.period_first_layer(layer, p)
        print(f"host={host} layer {layer} (Period of layer {first})", flush=True)
        tt = {kk: dev(v) for kk, v in t.items()}
        A = torch.full((w.n_chunks,), float("nan"), dtype=torch.float64, device=DEV)
        sel = torch.full((k,), -7, dtype=torch.int32, device=DEV)
        out = torch.empty_like(tt["q"])
        if host:
            nxt = stores[layer + 1] if layer + 1 < len(stores) else None
            st = ctx.reprefill_layer(layer, tt["q"], tt["k_suffix"], tt["v_suffix"], tt["k_prefix"],
                                     out, kv_host=stores[layer], kv_host_next=nxt, chunk_scores=A,
                                     sel_idx=sel)
        else:
            st = ctx.reprefill_layer(layer, tt["q"], tt["k_suffix"], tt["v_suffix"], tt["k_prefix"],
                                     out, k_prefix=tt["k_prefix"], v_prefix=tt["v_prefix"],
                                     chunk_scores=A, sel_idx=sel)
        torch.cuda.synchronize()
        A, sel = A.cpu().numpy(), sel.cpu().numpy()
        if first == layer:
            A_ref = oracle.chunk_scores(s, oracle.token_importance(s, t["q"], t["k_prefix"]))
            err = rel_err(A, A_ref)
            assert err <= SCORE_RTOL, err
            check_set(A_ref, sel, k, err)
            sets[layer] = sel
        else:
            assert np.isnan(A).all()  # no scoring on this layer
            assert np.array_equal(sel, sets[first])
        out_ref = oracle.sparse_attn(s, t["q"], t["k_prefix"], t["v_prefix"], sets[first],
                                     t["k_suffix"], t["v_suffix"])
        aerr, ratio = attn_check(s, t, sets[first], to_f64(out).reshape(out_ref.shape), out_ref)
        print(f"  attn max abs {aerr:.2e} ({ratio:.2f} of its bound)", flush=True)
        if host:
            acc = oracle.layer_accounting(s, sel, prev)
            assert st["hits"] == acc["hits"] and st["misses"] == acc["misses"]
            assert st["bytes_demand"] == acc["bytes_demand"]
            if first != layer:
                assert st["hits"] == k and st["misses"] == 0
            prev = sel if layer + 1 < w.n_layers else np.zeros(0, np.int32)
    # the oracle's prediction chain for these sets is the one the context used
    pred = oracle.period_prediction(sets, p)
    assert all(np.array_equal(pred[l + 1], sets[oracle.period_first_layer(l, p)])
               for l in range(w.n_layers - 1))
    # a layer past the first of its Period needs that first layer's set
    ctx.reset()
    t = layers[0]
    tt = {kk: dev(v) for kk, v in t.items()}
    out = torch.empty_like(tt["q"])
    if host:  # in order, but set_period forgets the set layer 0 selected
        ctx.reprefill_layer(0, tt["q"], tt["k_suffix"], tt["v_suffix"], tt["k_prefix"], out,
                            kv_host=stores[0])
        ctx.set_period(p)
    with pytest.raises(ckv.CkvError) as e:
        if host:
            ctx.reprefill_layer(1, tt["q"], tt["k_suffix"], tt["v_suffix"], tt["k_prefix"], out,
                                kv_host=stores[1])
        else:
            ctx.reprefill_layer(3, tt["q"], tt["k_suffix"], tt["v_suffix"], tt["k_prefix"], out,
                                k_prefix=tt["k_prefix"], v_prefix=tt["v_prefix"])
    assert e.value.status == ckv.ESTATE
    torch.cuda.synchronize()
    with pytest.raises(ckv.CkvError) as e:
        ctx.set_period(0)
    assert e.value.status == ckv.EINVAL
    ctx.close()


def _host_layers(w, n_layers=None):
    L = w.n_layers if n_layers is None else n_layers
    hs = synth.heavy_sets(w)
    layers = [synth.layer_tensors(w, l, hs[l]) for l in range(L)]
    return layers, _host_store(w, layers)


def _run_host(ctx, w, t, store, layer, pred=None, nxt=None):
    k = ctx.k
    tt = {kk: dev(v) for kk, v in t.items()}
    A = torch.empty(w.n_chunks, dtype=torch.float64, device=DEV)
    sel = torch.empty(k, dtype=torch.int32, device=DEV)
    out = torch.empty_like(tt["q"])
    st = ctx.reprefill_layer(layer, tt["q"], tt["k_suffix"], tt["v_suffix"], tt["k_prefix"], out,
                             kv_host=store, kv_host_next=nxt, chunk_scores=A, sel_idx=sel,
                             pred_idx=pred)
    return A, sel, out, st


@pytest.mark.parametrize("how", ["empty", "perfect", "complement", "partial", "four_misses",
                                 "five_misses"])
def test_layer_caller_prediction(how):
    """A caller-given prediction (ckv_layer_io.pred_idx, Sec. 4.3.2's set from a
    previous Period or layer) replaces the context's own: its chunks are copied
    beside the layer's scoring, the rest fetched on demand.  Outputs lie within
    their bound of the oracle's (and equal the first run's bit for bit when the
    prediction is empty again); hits, misses, wasted
    and the prefetched and demand bytes equal the oracle's set algebra for that
    prediction."""
    import paper_2601_13631_amd as ckv
    w = small("c5_qwen32b_128k_host", n_prefix=4096, n_suffix=24, n_layers=3)
    layers, stores = _host_layers(w)
    s = oshape(w)
    ctx = ckv.Context(dims_of(w), w.n_layers, w.keep_ratio, ckv.CTX_HOST_PREFIX)
    k, m = ctx.k, w.n_chunks
    layer = 2  # the first layer of a request may be any layer
    t = layers[layer]
    # the layer's own set, with an empty prediction
    A0, sel0, out0, st0 = _run_host(ctx, w, t, stores[layer], layer, pred=[])
    torch.cuda.synchronize()
    sel0 = sel0.cpu().numpy()
    assert st0["hits"] == 0 and st0["misses"] == k and st0["bytes_prefetch"] == 0
    rest = np.setdiff1d(np.arange(m, dtype=np.int32), sel0)
    rng = np.random.default_rng(3)
    pred = {"empty": np.zeros(0, np.int32), "perfect": sel0,
            "complement": rest[:k],
            "partial": np.sort(np.concatenate([sel0[: k // 2], rng.choice(rest, k - k // 2, replace=False)])),
            # few misses: as many shares of the demand copy as misses, or fewer
            "four_misses": np.delete(sel0, [0, 3, 6, 9]),
            "five_misses": np.delete(sel0, [1, 2, 5, 8, 11]),
            }[how].astype(np.int32)
    ctx.reset()
    print(f"prediction {how}: {pred.size} chunks", flush=True)
    A, sel, out, st = _run_host(ctx, w, t, stores[layer], layer, pred=pred)
    torch.cuda.synchronize()
    A, sel = A.cpu().numpy(), sel.cpu().numpy()
    assert np.array_equal(sel, sel0)
    if how == "empty":  # the same chunks in HBM when the layer attends: the same roundings
        assert torch.equal(out.view(torch.int16), out0.view(torch.int16))
    A_ref, out_ref = _oracle_layer(w, t, sel)
    err = rel_err(A, A_ref)
    assert err <= SCORE_RTOL, err
    check_set(A_ref, sel, k, err)
    attn_check(s, t, sel, to_f64(out).reshape(out_ref.shape), out_ref)
    acc = oracle.layer_accounting(s, sel, pred)
    for f in ("hits", "misses", "wasted", "bytes_prefetch", "bytes_demand"):
        assert st[f] == acc[f], (f, st[f], acc[f])
    assert st["bytes_gathered"] == acc["bytes_used"]
    if how == "perfect":
        assert st["misses"] == 0 and st["hits"] == k
    if how == "complement":
        assert st["hits"] == 0 and st["wasted"] == k
    if how.endswith("_misses"):
        assert st["misses"] == (4 if how == "four_misses" else 5)
    print(f"  hits {st['hits']} misses {st['misses']} wasted {st['wasted']}", flush=True)
    # refusals: not ascending, out of range, more than k
    ctx.reset()
    for bad in (np.array([3, 2], np.int32), np.array([m], np.int32), np.arange(k + 1, dtype=np.int32)):
        with pytest.raises(ckv.CkvError) as e:
            _run_host(ctx, w, t, stores[layer], layer, pred=bad)
        assert e.value.status == ckv.EINVAL
    ctx.close()


def test_layer_copy_error_injection():
    """A host-to-HBM copy that fails (injected at its enqueue) returns CKV_EHIP;
    the context refuses further layers until a reset, after which it runs the
    request again with outputs bit-equal to a context that never failed."""
    import paper_2601_13631_amd as ckv
    w = small("c5_qwen32b_128k_host", n_prefix=4096, n_suffix=24, n_layers=3)
    layers, stores = _host_layers(w)
    ctx = ckv.Context(dims_of(w), w.n_layers, w.keep_ratio, ckv.CTX_HOST_PREFIX)
    clean = ckv.Context(dims_of(w), w.n_layers, w.keep_ratio, ckv.CTX_HOST_PREFIX)
    nxt = lambda l: stores[l + 1] if l + 1 < w.n_layers else None
    ref = [_run_host(clean, w, layers[l], stores[l], l, nxt=nxt(l)) for l in range(w.n_layers)]
    torch.cuda.synchronize()
    ctx.inject_copy_error(1)
    _run_host(ctx, w, layers[0], stores[0], 0, nxt=nxt(0))
    with pytest.raises(ckv.CkvError) as e:
        _run_host(ctx, w, layers[1], stores[1], 1, nxt=nxt(1))
    assert e.value.status == ckv.EHIP and "injected" in str(e.value)
    with pytest.raises(ckv.CkvError) as e:
        _run_host(ctx, w, layers[2], stores[2], 2, nxt=nxt(2))
    assert e.value.status == ckv.ESTATE
    ctx.reset()
    got = [_run_host(ctx, w, layers[l], stores[l], l, nxt=nxt(l)) for l in range(w.n_layers)]
    torch.cuda.synchronize()
    for l, (a, b) in enumerate(zip(ref, got)):
        assert torch.equal(a[1], b[1]), l
        assert torch.equal(a[2].view(torch.int16), b[2].view(torch.int16)), l
        assert a[3] == b[3], l
    with pytest.raises(ckv.CkvError) as e:  # HBM-resident contexts move no host chunks
        hbm = ckv.Context(dims_of(w), w.n_layers, w.keep_ratio, 0)
        try:
            hbm.inject_copy_error(0)
        finally:
            hbm.close()
    assert e.value.status == ckv.EINVAL
    ctx.close()
    clean.close()


@pytest.mark.parametrize("registered,subperiod", [(False, 1), (True, 1), (True, 2), (True, 4)],
                         ids=["one-ahead", "period-sp1", "period-sp2", "period-sp4"])
def test_layer_periods_host_unsynchronised(registered, subperiod):
    """Periods of 4 layers on the host-resident path with no host
    synchronisation between layers (layers inside a Period never wait on the
    host, so the host runs ahead of the GPU and rewrites pinned staging the
    GPU may not have read yet).  With the per-layer stores registered, a
    Period's first layer queues the copies of the whole Period and, with a
    SubPeriod of sp, its attention waits for the first sp layers.  Every
    layer's output is compared with the oracle after the whole request; sets
    follow the oracle's Period rule and the hit/miss/byte counts its set
    algebra (every later layer of a Period fully predicted)."""
    import paper_2601_13631_amd as ckv
    p = 4
    w = small("c5_qwen32b_128k_host", n_prefix=4096, n_suffix=24, n_layers=10)
    layers, stores = _host_layers(w)
    s = oshape(w)
    ctx = ckv.Context(dims_of(w), w.n_layers, w.keep_ratio, ckv.CTX_HOST_PREFIX)
    if registered:
        ctx.set_host_layers(stores)
    ctx.set_period(p)
    ctx.set_subperiod(subperiod)
    k = ctx.k
    # inputs uploaded first: an upload from pageable memory would synchronise
    base = [{kk: dev(v) for kk, v in t.items()} for t in layers]
    torch.cuda.synchronize()
    res = []
    for r in range(2):  # twice: the second request reuses buffers of the first
        ctx.reset()
        res = []
        for l, tt in enumerate(base):
            kw = {} if registered else dict(kv_host=stores[l],
                                            kv_host_next=stores[l + 1] if l + 1 < w.n_layers else None)
            sel = torch.empty(k, dtype=torch.int32, device=DEV)
            out = torch.empty_like(tt["q"])
            st = ctx.reprefill_layer(l, tt["q"], tt["k_suffix"], tt["v_suffix"], tt["k_prefix"], out,
                                     sel_idx=sel, **kw)
            res.append((sel, out, st, tt))
    torch.cuda.synchronize()
    sets = [None] * w.n_layers
    total_pref = 0
    for l, (sel, out, st, _) in enumerate(res):
        first = oracle.period_first_layer(l, p)
        sel = sel.cpu().numpy()
        if first == l:
            sets[l] = sel
        assert np.array_equal(sel, sets[first]), l
    preds = oracle.period_prediction(sets, p)
    for l, (sel, out, st, _) in enumerate(res):
        print(f"layer {l}: hits {st['hits']} misses {st['misses']} prefetch {st['bytes_prefetch']}",
              flush=True)
        t = layers[l]
        out_ref = oracle.sparse_attn(s, t["q"], t["k_prefix"], t["v_prefix"], sets[l - l % p],
                                     t["k_suffix"], t["v_suffix"])
        attn_check(s, t, sets[l - l % p], to_f64(out).reshape(out_ref.shape), out_ref)
        acc = oracle.layer_accounting(s, sets[l - l % p], preds[l])
        for f in ("hits", "misses", "wasted", "bytes_demand"):
            assert st[f] == acc[f], (l, f, st[f], acc[f])
        if l % p:
            assert st["hits"] == k and st["misses"] == 0
        total_pref += st["bytes_prefetch"]
    # the prefetch bytes over the request are those of every layer's prediction
    # (issued a layer ahead, or a whole Period ahead by its first layer)
    assert total_pref == sum(oracle.layer_accounting(s, preds[l], preds[l])["bytes_prefetch"]
                             for l in range(w.n_layers))
    ctx.close()


@pytest.mark.parametrize("host", [False, True], ids=["hbm", "host"])
def test_layer_step_deterministic(host):
    """The whole layer step run twice on the same inputs gives bitwise equal
    scores, sets and outputs."""
    import paper_2601_13631_amd as ckv
    w = small("c3_qwen7b_32k", n_prefix=8192, n_suffix=64, n_layers=2)
    layers, stores = _host_layers(w)
    outs = []
    for rep in range(2):
        ctx = ckv.Context(dims_of(w), w.n_layers, w.keep_ratio, ckv.CTX_HOST_PREFIX if host else 0)
        got = []
        for l, t in enumerate(layers):
            tt = {kk: dev(v) for kk, v in t.items()}
            A = torch.empty(w.n_chunks, dtype=torch.float64, device=DEV)
            sel = torch.empty(ctx.k, dtype=torch.int32, device=DEV)
            out = torch.empty_like(tt["q"])
            kw = dict(kv_host=stores[l], kv_host_next=stores[l + 1] if l + 1 < len(stores) else None) \
                if host else dict(k_prefix=tt["k_prefix"], v_prefix=tt["v_prefix"])
            ctx.reprefill_layer(l, tt["q"], tt["k_suffix"], tt["v_suffix"], tt["k_prefix"], out,
                                chunk_scores=A, sel_idx=sel, **kw)
            got.append((A, sel, out))
        torch.cuda.synchronize()
        ctx.close()
        outs.append(got)
    for (a1, s1, o1), (a2, s2, o2) in zip(*outs):
        assert torch.equal(a1.view(torch.int64), a2.view(torch.int64))
        assert torch.equal(s1, s2)
        assert torch.equal(o1.view(torch.int16), o2.view(torch.int16))
