"""The attention-guided cache (Sec. 4.5) on the host-resident layer step.

Three requests on one prefix run layer by layer through a context with a
cache attached and through one without.  Kept sets and chunk scores must
agree bit for bit (the cache only changes where the chunk bytes come from),
and both outputs must lie within their bound of the oracle's attention: a
host-resident layer attends first over the chunks already in HBM (cache slots
and prefetched chunks) and then over the chunks copied on demand, so the
cache changes how the keys are grouped and with it the roundings.  The
chunks read from HBM cache slots, the host-link counts and the cache fills
must equal what the oracle cache, fed the same chunk scores, predicts; the
final tiers and scores must equal the oracle cache's.
"""
import numpy as np
import pytest
import torch

import oracle
import synth
from gpu_common import DEV, attn_check, dev, dims_of, oshape, to_f64

pytestmark = pytest.mark.gpu


def _store(w, t):
    cm = synth.chunk_major(t["k_prefix"], t["v_prefix"], w.chunk_size)
    h = torch.from_numpy(cm.reshape(-1))
    if cm.dtype == np.uint16:
        h = h.view(torch.bfloat16)
    return h.pin_memory()


@pytest.mark.parametrize("period,n_prefix", [(1, 4096), (2, 4096), (1, 45)])  # 45: two chunks
def test_layer_cache_requests(period, n_prefix):
    import paper_2601_13631_amd as ckv
    w = synth.WORKLOADS["c5_qwen32b_128k_host"].scaled(n_prefix=n_prefix, n_suffix=24, n_layers=4)
    L, m = w.n_layers, w.n_chunks
    layers = [synth.layer_tensors(w, l) for l in range(L)]
    stores = [_store(w, t) for t in layers]
    base = [{kk: dev(v) for kk, v in t.items()} for t in layers]
    s = oshape(w)
    ctx = ckv.Context(dims_of(w), w.n_layers, w.keep_ratio, ckv.CTX_HOST_PREFIX)
    plain = ckv.Context(dims_of(w), w.n_layers, w.keep_ratio, ckv.CTX_HOST_PREFIX)
    ctx.set_period(period)
    plain.set_period(period)
    k = ctx.k
    gpu_slots, cpu_slots = (L * k) // 2, L * k
    cache = ckv.Cache(L * m, gpu_slots, cpu_slots)
    ctx.attach_cache(cache)
    ref = oracle.Cache(L * m, gpu_slots, cpu_slots)
    per_tok = 2 * w.n_kv_heads * w.head_dim * w.elem_bytes
    lens = np.minimum(w.chunk_size, w.n_prefix - np.arange(m) * w.chunk_size)
    slot_bytes = w.chunk_size * per_tok
    total_cache_hits = 0
    for r in range(3):
        ctx.reset()
        plain.reset()
        prev = np.zeros(0, np.int64)
        A_first = None
        for l in range(L):
            first = l - l % period
            print(f"period {period} request {r} layer {l}", flush=True)
            q = dev(synth.request_queries(w, l, r))
            outs, sels, As, stats = [], [], [], []
            for c in (ctx, plain):
                A = torch.full((m,), float("nan"), dtype=torch.float64, device=DEV)
                sel = torch.empty(k, dtype=torch.int32, device=DEV)
                out = torch.empty_like(q)
                st = c.reprefill_layer(l, q, base[l]["k_suffix"], base[l]["v_suffix"],
                                       base[l]["k_prefix"], out, kv_host=stores[l],
                                       kv_host_next=stores[l + 1] if l + 1 < L else None,
                                       chunk_scores=A, sel_idx=sel)
                outs.append(out)
                sels.append(sel)
                As.append(A)
                stats.append(st)
            torch.cuda.synchronize()
            sel = sels[0].cpu().numpy().astype(np.int64)
            assert np.array_equal(sel, sels[1].cpu().numpy())
            if first == l:
                A_first = As[0].cpu().numpy()
                assert np.array_equal(A_first.view(np.int64), As[1].cpu().numpy().view(np.int64))
            st = stats[0]
            # expected counts from the oracle cache before and after this layer's access
            tier = ref.state()[2]
            resident = set(int(j) for j in sel if tier[l * m + j] == oracle.TIER_GPU)
            S = set(int(j) for j in sel)
            P = set(int(j) for j in prev) - resident
            hits = (S - resident) & P
            miss = S - resident - P
            assert st["cache_hits"] == len(resident)
            assert st["hits"] == len(hits) and st["misses"] == len(miss)
            assert st["wasted"] == len(P) - len(hits)
            assert st["bytes_demand"] == int(sum(lens[j] for j in miss)) * per_tok
            assert st["bytes_gathered"] == int(sum(lens[j] for j in S)) * per_tok
            before = tier[l * m + sel]
            ref.access(l * m + sel, A_first[sel])
            after = ref.state()[2]
            fills = int(np.sum((after[l * m + sel] == oracle.TIER_GPU) &
                               (before != oracle.TIER_GPU)))
            assert st["bytes_cache_fill"] == fills * slot_bytes
            if l + 1 < L:
                nxt = [j for j in S if after[(l + 1) * m + j] != oracle.TIER_GPU]
                assert st["bytes_prefetch"] == int(sum(lens[j] for j in nxt)) * per_tok
            # every layer's output against the oracle's attention over the same set
            t = dict(layers[l], q=synth.request_queries(w, l, r))
            out_ref = oracle.sparse_attn(s, t["q"], t["k_prefix"], t["v_prefix"],
                                         sel.astype(np.int32), t["k_suffix"], t["v_suffix"])
            for o in outs:
                attn_check(s, t, sel.astype(np.int32), to_f64(o).reshape(out_ref.shape), out_ref)
            total_cache_hits += st["cache_hits"]
            print(f"  cache hits {st['cache_hits']} prefetch hits {st['hits']} "
                  f"misses {st['misses']} fills {fills}", flush=True)
            prev = sel if l + 1 < L else np.zeros(0, np.int64)
    assert total_cache_hits > 0  # later requests do find chunks in HBM
    I1, F1, T1 = cache.state()
    I2, F2, T2 = ref.state()
    assert np.array_equal(I1.view(np.int64), I2.view(np.int64))
    assert np.array_equal(F1, F2) and np.array_equal(T1, T2)
    ctx.reset()
    ctx.attach_cache(None)
    ctx.close()
    plain.close()
    cache.close()


def test_attach_cache_refusals():
    import paper_2601_13631_amd as ckv
    w = synth.WORKLOADS["c5_qwen32b_128k_host"].scaled(n_prefix=4096, n_suffix=24, n_layers=2)
    m = w.n_chunks
    t = synth.layer_tensors(w, 0)
    tt = {kk: dev(v) for kk, v in t.items()}
    store = _store(w, t)
    hbm = ckv.Context(dims_of(w), w.n_layers, w.keep_ratio, 0)
    cache = ckv.Cache(2 * m, 8, 8)
    with pytest.raises(ckv.CkvError) as e:  # needs a host-resident prefix
        hbm.attach_cache(cache)
    assert e.value.status == ckv.EINVAL
    hbm.close()
    ctx = ckv.Context(dims_of(w), w.n_layers, w.keep_ratio, ckv.CTX_HOST_PREFIX)
    odd = ckv.Cache(2 * m + 1, 8, 8)
    with pytest.raises(ckv.CkvError) as e:  # keys not a whole number of layers
        ctx.attach_cache(odd)
    assert e.value.status == ckv.EINVAL
    used = ckv.Cache(2 * m, 8, 8)
    used.access([3], [1.0])
    with pytest.raises(ckv.CkvError) as e:  # GPU tier not empty
        ctx.attach_cache(used)
    assert e.value.status == ckv.ESTATE
    one_layer = ckv.Cache(m, 8, 8)
    ctx.attach_cache(one_layer)
    out = torch.empty_like(tt["q"])
    ctx.reprefill_layer(0, tt["q"], tt["k_suffix"], tt["v_suffix"], tt["k_prefix"], out,
                        kv_host=store, kv_host_next=store)
    with pytest.raises(ckv.CkvError) as e:  # mid-request
        ctx.attach_cache(cache)
    assert e.value.status == ckv.ESTATE
    with pytest.raises(ckv.CkvError) as e:  # layer 1 has no keys in a one-layer cache
        ctx.reprefill_layer(1, tt["q"], tt["k_suffix"], tt["v_suffix"], tt["k_prefix"], out,
                            kv_host=store)
    assert e.value.status == ckv.EINVAL
    torch.cuda.synchronize()
    ctx.reset()
    ctx.attach_cache(None)
    ctx.close()
    for c in (cache, odd, used, one_layer):
        c.close()


@pytest.mark.parametrize("period,with_cache,direct,n_prefix", [
    (1, False, False, 4096), (1, True, True, 4096), (2, True, False, 4096),
    (1, True, False, 45),     # two chunks per layer, the last one partial; one kept
    (1, True, True, 32768)])  # the last: 1,024 chunks of 128 KiB per layer, a 512 MiB file
def test_layer_store(tmp_path, period, with_cache, direct, n_prefix):
    """Chunks read from a file by the storage tier's I/O threads into the pinned
    chunk pool: every layer's output, set and host-link counts equal those of
    the same layers reading the pinned host store (with or without the cache,
    across three requests), and the bytes read from the file are exactly the
    chunks that were neither in HBM slots nor in the pool, which holds the
    chunks of the cache's two tiers (the oracle cache, fed the same scores,
    says which)."""
    import paper_2601_13631_amd as ckv
    w = synth.WORKLOADS["c5_qwen32b_128k_host"].scaled(n_prefix=n_prefix, n_suffix=24, n_layers=4)
    L, m = w.n_layers, w.n_chunks
    layers = [synth.layer_tensors(w, l) for l in range(L)]
    stores = [_store(w, t) for t in layers]
    path = str(tmp_path / "kv.bin")
    with open(path, "wb") as f:
        for t in layers:
            synth.chunk_major(t["k_prefix"], t["v_prefix"], w.chunk_size).tofile(f)
    span = 2 * w.chunk_size * w.n_kv_heads * w.head_dim * w.elem_bytes
    try:
        store = ckv.Store(path, L * m, span, 4, ckv.STORE_DIRECT if direct else 0)
    except ckv.CkvError:
        pytest.skip("this filesystem refuses O_DIRECT")
    base = [{kk: dev(v) for kk, v in t.items()} for t in layers]
    ctxs = [ckv.Context(dims_of(w), w.n_layers, w.keep_ratio, ckv.CTX_HOST_PREFIX) for _ in range(2)]
    k = ctxs[0].k
    gpu_slots, cpu_slots = (L * k) // 2, L * k
    caches = []
    for c in ctxs:
        c.set_period(period)
        if with_cache:
            caches.append(ckv.Cache(L * m, gpu_slots, cpu_slots))
            c.attach_cache(caches[-1])
    ctxs[1].attach_store(store)
    ref = oracle.Cache(L * m, gpu_slots, cpu_slots) if with_cache else None
    storage_total = 0
    for r in range(3):
        for c in ctxs:
            c.reset()
        prev = []
        A_first = None
        for l in range(L):
            first = l - l % period
            print(f"store n {n_prefix} period {period} cache {with_cache} direct {direct} "
                  f"request {r} layer {l}", flush=True)
            q = dev(synth.request_queries(w, l, r))
            outs, sels, sts = [], [], []
            A = torch.full((m,), float("nan"), dtype=torch.float64, device=DEV)
            for i, c in enumerate(ctxs):
                sel = torch.empty(k, dtype=torch.int32, device=DEV)
                out = torch.empty_like(q)
                kv = dict(kv_host=stores[l], kv_host_next=stores[l + 1] if l + 1 < L else None) \
                    if i == 0 else {}
                sts.append(c.reprefill_layer(l, q, base[l]["k_suffix"], base[l]["v_suffix"],
                                             base[l]["k_prefix"], out, sel_idx=sel,
                                             chunk_scores=A if i == 1 else None, **kv))
                outs.append(out)
                sels.append(sel)
            torch.cuda.synchronize()
            assert torch.equal(sels[0], sels[1])
            assert torch.equal(outs[0].view(torch.int16), outs[1].view(torch.int16))
            if n_prefix <= 4096:  # and against the oracle over the same set
                t = dict(layers[l], q=synth.request_queries(w, l, r))
                sel1 = sels[1].cpu().numpy()
                out_ref = oracle.sparse_attn(oshape(w), t["q"], t["k_prefix"], t["v_prefix"],
                                             sel1, t["k_suffix"], t["v_suffix"])
                attn_check(oshape(w), t, sel1, to_f64(outs[1]).reshape(out_ref.shape), out_ref)
            got = dict(sts[1])
            storage = got.pop("bytes_storage")
            assert sts[0].pop("bytes_storage") == 0
            assert got == sts[0], (got, sts[0])
            sel = sels[1].cpu().numpy().astype(np.int64)
            if first == l:
                A_first = A.cpu().numpy()
            # expected file reads from the oracle cache's tiers
            if ref is None:
                tier = np.zeros(L * m, np.int8)
            else:
                tier = ref.state()[2]
            hbm = {int(j) for j in sel if tier[l * m + j] == oracle.TIER_GPU}
            P = [j for j in prev if j not in hbm]
            miss = [int(j) for j in sel if int(j) not in hbm and int(j) not in P]
            reads = sum(1 for j in miss if tier[l * m + j] == oracle.TIER_NONE)
            if ref is not None:
                ref.access(l * m + sel, A_first[sel])
                tier = ref.state()[2]
            if l + 1 < L:
                nxt = [int(j) for j in sel if tier[(l + 1) * m + j] != oracle.TIER_GPU]
                reads += sum(1 for j in nxt if tier[(l + 1) * m + j] == oracle.TIER_NONE)
                prev = nxt
            else:
                prev = []
            assert storage == reads * span, (storage // span, reads)
            storage_total += storage
            print(f"  file reads {storage // span} chunks", flush=True)
    if with_cache:  # later requests find chunks in the pool
        assert storage_total < 3 * L * k * span
    for c in ctxs:
        c.reset()
    ctxs[1].attach_store(None)
    for c in ctxs:
        if with_cache:
            c.attach_cache(None)
        c.close()
    for cache in caches:
        cache.close()
    store.close()


def test_attach_store_refusals(tmp_path):
    import paper_2601_13631_amd as ckv
    w = synth.WORKLOADS["c5_qwen32b_128k_host"].scaled(n_prefix=4096, n_suffix=24, n_layers=1)
    m = w.n_chunks
    span = 2 * w.chunk_size * w.n_kv_heads * w.head_dim * w.elem_bytes
    t = synth.layer_tensors(w, 0)
    path = str(tmp_path / "kv.bin")
    cm = synth.chunk_major(t["k_prefix"], t["v_prefix"], w.chunk_size)
    with open(path, "wb") as f:
        cm.tofile(f)
        cm.tofile(f)  # two layers' worth of spans
    tt = {kk: dev(v) for kk, v in t.items()}
    out = torch.empty_like(tt["q"])
    hbm = ckv.Context(dims_of(w), w.n_layers, w.keep_ratio, 0)
    good = ckv.Store(path, 2 * m, span, 2)
    with pytest.raises(ckv.CkvError) as e:  # needs a host-resident prefix
        hbm.attach_store(good)
    assert e.value.status == ckv.EINVAL
    hbm.close()
    ctx = ckv.Context(dims_of(w), 4, w.keep_ratio, ckv.CTX_HOST_PREFIX)  # layers past the store's
    for bad in (ckv.Store(path, 2 * m, span // 2, 2),      # spans are not chunks
                ckv.Store(path, 2 * m - 1, span, 2)):     # not a whole number of layers
        with pytest.raises(ckv.CkvError) as e:
            ctx.attach_store(bad)
        assert e.value.status == ckv.EINVAL
        bad.close()
    cache = ckv.Cache(2 * m, 8, 8)
    ctx.attach_store(good)
    with pytest.raises(ckv.CkvError) as e:  # the cache goes first
        ctx.attach_cache(cache)
    assert e.value.status == ckv.ESTATE
    ctx.reprefill_layer(0, tt["q"], tt["k_suffix"], tt["v_suffix"], tt["k_prefix"], out)
    ctx.reprefill_layer(1, tt["q"], tt["k_suffix"], tt["v_suffix"], tt["k_prefix"], out)
    with pytest.raises(ckv.CkvError) as e:  # mid-request
        ctx.attach_store(None)
    assert e.value.status == ckv.ESTATE
    with pytest.raises(ckv.CkvError) as e:  # the store holds two layers
        ctx.reprefill_layer(2, tt["q"], tt["k_suffix"], tt["v_suffix"], tt["k_prefix"], out)
    assert e.value.status == ckv.EINVAL
    torch.cuda.synchronize()
    ctx.reset()
    ctx.attach_store(None)
    ctx.close()
    cache.close()
    good.close()


@pytest.mark.parametrize("with_cache", [False, True, "small"])
def test_layer_store_subperiod(tmp_path, with_cache):
    """Periods of 4 layers with a SubPeriod of 3: a Period's layers queue the
    storage reads of the next two layers of the Period.  Sets equal the
    pinned-store path's; without a cache so do the outputs, bit for bit (the
    same chunks are in HBM when each layer attends), the hit/miss counts and,
    over a request, the prefetched and file-read bytes of one layer ahead.
    With a cache the read-ahead is listed against an earlier cache state, so
    which chunks a layer finds in HBM may differ: every output is checked
    against the oracle's attention instead."""
    import paper_2601_13631_amd as ckv
    w = synth.WORKLOADS["c5_qwen32b_128k_host"].scaled(n_prefix=4096, n_suffix=24, n_layers=8)
    L, m = w.n_layers, w.n_chunks
    layers = [synth.layer_tensors(w, l) for l in range(L)]
    stores = [_store(w, t) for t in layers]
    path = str(tmp_path / "kv.bin")
    with open(path, "wb") as f:
        for t in layers:
            synth.chunk_major(t["k_prefix"], t["v_prefix"], w.chunk_size).tofile(f)
    span = 2 * w.chunk_size * w.n_kv_heads * w.head_dim * w.elem_bytes
    store = ckv.Store(path, L * m, span, 4)
    base = [{kk: dev(v) for kk, v in t.items()} for t in layers]
    ctxs = [ckv.Context(dims_of(w), w.n_layers, w.keep_ratio, ckv.CTX_HOST_PREFIX) for _ in range(3)]
    k = ctxs[0].k
    caches = []
    for i, c in enumerate(ctxs):
        c.set_period(4)
        if with_cache == "small":
            # tiers of about one layer's chunks: the cascade sends chunks of
            # later layers, listed by read-ahead entries while in the CPU
            # tier, out of memory before their layer runs
            caches.append(ckv.Cache(L * m, k // 2, k))
            c.attach_cache(caches[-1])
        elif with_cache:
            caches.append(ckv.Cache(L * m, (L * k) // 2, L * k))
            c.attach_cache(caches[-1])
        if i > 0:
            c.set_subperiod(3 if i == 2 else 1)
            c.attach_store(store)
    with pytest.raises(ckv.CkvError) as e:  # the SubPeriod sizes the pool: set it first
        ctxs[2].set_subperiod(2)
    assert e.value.status == ckv.ESTATE
    for r in range(2):
        for c in ctxs:
            c.reset()
        tot = [dict(bytes_prefetch=0, bytes_storage=0) for _ in ctxs]
        for l in range(L):
            print(f"subperiod cache {with_cache} request {r} layer {l}", flush=True)
            q = dev(synth.request_queries(w, l, r))
            outs, sels, sts = [], [], []
            for i, c in enumerate(ctxs):
                sel = torch.empty(k, dtype=torch.int32, device=DEV)
                out = torch.empty_like(q)
                kv = dict(kv_host=stores[l], kv_host_next=stores[l + 1] if l + 1 < L else None) \
                    if i == 0 else {}
                sts.append(c.reprefill_layer(l, q, base[l]["k_suffix"], base[l]["v_suffix"],
                                             base[l]["k_prefix"], out, sel_idx=sel, **kv))
                outs.append(out)
                sels.append(sel)
            torch.cuda.synchronize()
            for i in (1, 2):
                assert torch.equal(sels[0], sels[i])
                if not with_cache:
                    assert torch.equal(outs[0].view(torch.int16), outs[i].view(torch.int16))
            if with_cache:
                t = dict(layers[l], q=synth.request_queries(w, l, r))
                sel0 = sels[0].cpu().numpy()
                out_ref = oracle.sparse_attn(oshape(w), t["q"], t["k_prefix"], t["v_prefix"],
                                             sel0, t["k_suffix"], t["v_suffix"])
                for o in outs:
                    attn_check(oshape(w), t, sel0, to_f64(o).reshape(out_ref.shape), out_ref)
            for i, st in enumerate(sts):
                for f in tot[i]:
                    tot[i][f] += st[f]
            if not with_cache:
                for f in ("hits", "misses", "wasted", "bytes_demand", "bytes_gathered"):
                    assert sts[2][f] == sts[1][f] == sts[0][f], (f, sts)
        if not with_cache:
            assert tot[2] == tot[1], tot
            assert tot[1]["bytes_prefetch"] == tot[0]["bytes_prefetch"]
    for c in ctxs:
        c.reset()
    for c in ctxs[1:]:
        c.attach_store(None)
    for c in ctxs:
        if with_cache:
            c.attach_cache(None)
        c.close()
    for cache in caches:
        cache.close()
    store.close()
