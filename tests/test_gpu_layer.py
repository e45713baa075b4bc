"""GPU parity of the whole layer step (ckv_reprefill_layer) against the oracle."""
import numpy as np
import pytest
import torch

import oracle
import synth
from gpu_common import DEV, check_set, dev, dims_of, oshape, rel_err, to_f64

pytestmark = pytest.mark.gpu

SCORE_RTOL = 2e-6


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
    ctx = ckv.Context(dims_of(w), w.keep_ratio, flags)
    k = ctx.k
    hs = synth.heavy_sets(w)
    tol = 1e-5 if w.dtype == "f32" else 2e-2
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
        aerr = float(np.abs(to_f64(out) - out_ref).max())
        print(f"  score rel err {err:.2e}  attn max abs {aerr:.2e}", flush=True)
        assert aerr <= tol
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


@pytest.mark.parametrize("scenario", ["drift", "repeat", "disjoint", "tiny"])
def test_layer_host_resident_prefetch(scenario):
    """Host-resident prefix: outputs equal the HBM path's oracle, and the
    hit/miss/byte counts equal the oracle's set algebra with the previous
    layer's selection as the prediction.  "tiny": two chunks (the last one
    partial, kept), one query."""
    import paper_2601_13631_amd as ckv
    if scenario == "tiny":
        w = small("c5_qwen32b_128k_host", n_prefix=45, n_suffix=1, n_layers=3)
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
    ctx = ckv.Context(dims_of(w), w.keep_ratio, ckv.CTX_HOST_PREFIX)
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
        aerr = float(np.abs(to_f64(out) - out_ref).max())
        assert aerr <= 2e-2, aerr
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
    ctx = ckv.Context(dims_of(w), w.keep_ratio, ckv.CTX_HOST_PREFIX if host else 0)
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
        aerr = float(np.abs(to_f64(out) - out_ref).max())
        print(f"  attn max abs {aerr:.2e}", flush=True)
        assert aerr <= 2e-2
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
