"""Host-side parts of the library against the oracle, element by element.

Read accounting against a block store (Sec. 4.2; Sec. 3) and the
attention-guided two-tier cache (Sec. 4.5, Eq. 2) are host code in libckv;
these tests call them through the C ABI on the CPU and require the oracle's
results exactly (integers, tiers, and the cumulative importance bit for bit).
"""
import numpy as np
import pytest

import oracle
import paper_2601_13631_amd as ckv


def _random_selection(rng, m):
    k = int(rng.integers(0, m + 1))
    return np.sort(rng.choice(m, size=k, replace=False)).astype(np.int32)


@pytest.mark.parametrize("seed", range(6))
def test_io_account_matches_oracle(seed):
    rng = np.random.default_rng(100 + seed)
    for _ in range(60):
        n = int(rng.integers(1, 20000))
        c = int(rng.choice([1, 2, 4, 8, 16, 32, 64, 100]))
        b = int(rng.choice([1, 16, 50, 64, 128, 4096]))
        sel = _random_selection(rng, -(-n // c))
        assert ckv.io_account(n, c, sel, b) == oracle.io_account(n, c, sel, b), (n, c, b, sel.size)


def test_io_account_workload_shapes():
    """Kept sets of the prefix shapes used elsewhere (8K..128K tokens, c 8..64, 64-token blocks)."""
    rng = np.random.default_rng(7)
    for n, c, r in ((8192, 16, 0.2), (32768, 32, 0.1), (65536, 8, 0.15), (65536, 64, 0.15),
                    (131072, 32, 0.1), (1000, 16, 1.0)):
        m = -(-n // c)
        k = ckv.num_keep(m, r)
        sel = np.sort(rng.choice(m, size=k, replace=False)).astype(np.int32)
        got = ckv.io_account(n, c, sel, 64)
        assert got == oracle.io_account(n, c, sel, 64)
        assert got["tokens_block"] >= got["tokens_selected"] == min(k * c, n) or \
            got["tokens_selected"] < k * c  # a short last chunk


def test_io_account_rejects_bad_arguments():
    for args in ((0, 4, [0], 64), (10, 0, [0], 64), (10, 4, [0], 0), (10, 4, [3], 64),
                 (10, 4, [-1], 64), (10, 4, [1, 0], 64), (10, 4, [1, 1], 64),
                 (10, 4, [0, 1, 2, 2], 64)):
        with pytest.raises(ckv.CkvError) as e:
            ckv.io_account(*args)
        assert e.value.status == ckv.EINVAL


def _stream(rng, n_keys, n_req, max_len, zipf=1.3):
    pop = rng.zipf(zipf, size=n_keys).astype(np.float64)
    pop /= pop.sum()
    for _ in range(n_req):
        cnt = int(rng.integers(0, min(max_len, n_keys) + 1))
        keys = rng.choice(n_keys, size=cnt, replace=False, p=pop)
        # attention scores: many exact ties (dyadic) and some arbitrary doubles
        A = np.where(rng.random(cnt) < 0.5, rng.choice([0.0, 0.25, 0.5, 2.0], size=cnt),
                     rng.exponential(1.0, size=cnt))
        yield keys, A


@pytest.mark.parametrize("policy", [ckv.CACHE_ATTENTION, ckv.CACHE_LFU, ckv.CACHE_LOADS])
@pytest.mark.parametrize("n_keys,gpu,cpu", [(50, 4, 6), (300, 32, 64), (120, 0, 20), (80, 12, 0),
                                            (40, 100, 100), (1, 1, 0), (2000, 64, 256)])
def test_cache_matches_oracle(policy, n_keys, gpu, cpu):
    rng = np.random.default_rng(n_keys * 7 + gpu + policy)
    lib = ckv.Cache(n_keys, gpu, cpu, policy)
    ref = oracle.Cache(n_keys, gpu, cpu, policy)
    for keys, A in _stream(rng, n_keys, 150, 40):
        w1, t1 = lib.access(keys, A)
        w2, t2 = ref.access(keys, A)
        assert np.array_equal(w1, w2) and t1 == t2
        assert np.array_equal(lib.lookup(np.arange(n_keys)), ref.state()[2])
    I1, F1, T1 = lib.state()
    I2, F2, T2 = ref.state()
    assert np.array_equal(I1.view(np.int64), I2.view(np.int64))  # bit for bit
    assert np.array_equal(F1, F2) and np.array_equal(T1, T2)
    for t in (ckv.TIER_GPU, ckv.TIER_CPU):
        assert np.array_equal(lib.resident(t), np.flatnonzero(T2 == t))
    assert len(lib.resident(ckv.TIER_GPU)) <= gpu and len(lib.resident(ckv.TIER_CPU)) <= cpu
    lib.close()
    ref.close()


def test_cache_layer_chunk_stream():
    """Keys layer * m + chunk over a 28-layer, 1024-chunk prefix: eight requests
    keep 103 chunks per layer, a shared hot core plus request-specific chunks."""
    rng = np.random.default_rng(42)
    L, m, k = 28, 1024, 103
    hot = [np.sort(rng.choice(m, size=51, replace=False)) for _ in range(L)]
    caches = [(ckv.Cache(L * m, 2048, 4096, p), oracle.Cache(L * m, 2048, 4096, p))
              for p in (ckv.CACHE_ATTENTION, ckv.CACHE_LFU, ckv.CACHE_LOADS)]
    for r in range(8):
        for layer in range(L):
            rest = rng.choice(np.setdiff1d(np.arange(m), hot[layer]), size=k - 51, replace=False)
            chunks = np.sort(np.concatenate([hot[layer], rest]))
            A = np.where(np.isin(chunks, hot[layer]), rng.uniform(20, 40, k), rng.uniform(0, 4, k))
            for lib, ref in caches:
                w1, t1 = lib.access(layer * m + chunks, A)
                w2, t2 = ref.access(layer * m + chunks, A)
                assert np.array_equal(w1, w2) and t1 == t2
    for lib, ref in caches:
        assert np.array_equal(lib.state()[2], ref.state()[2])


def test_cache_rejects_bad_requests_without_change():
    lib = ckv.Cache(10, 2, 2)
    lib.access([1, 2, 3], [0.5, 0.25, 0.125])
    before = [a.copy() for a in lib.state()]
    for keys, A in (([1, 1], [0.1, 0.2]), ([4, 10], [0.1, 0.2]), ([4, -1], [0.1, 0.2]),
                    ([4, 5], [0.1, -0.5]), ([4, 5], [0.1, np.nan]), ([4, 5], [np.inf, 0.0])):
        with pytest.raises(ckv.CkvError) as e:
            lib.access(keys, A)
        assert e.value.status == ckv.EINVAL
        after = lib.state()
        assert all(np.array_equal(a, b) for a, b in zip(before, after))
    for args in ((0, 1, 1, 0), (5, -1, 1, 0), (5, 1, -1, 0), (5, 1, 1, 7)):
        with pytest.raises(ckv.CkvError):
            ckv.Cache(*args)
    lib.close()
