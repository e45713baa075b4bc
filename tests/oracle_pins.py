"""Pins of the CPU oracle to facts outside itself.

Each ``pin_*`` raises AssertionError when the oracle disagrees with a closed form,
a hand-worked example, a library routine (torch softmax / SDPA in fp64), an
invariant, or brute force.  ``test_oracle.py`` runs them against the oracle;
``test_oracle_mutants.py`` runs them against deliberately broken copies of the
oracle and requires every copy to fail at least one pin.
"""
from __future__ import annotations

import itertools
import json
import math
import os

import numpy as np
import torch

import oracle
from oracle import BF16, F32, Shape
from synth import bf16_bits_to_f32, to_bf16_bits

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")
E = math.e


def _rand(shape, rng, dtype):
    x = rng.standard_normal(shape).astype(np.float32)
    return to_bf16_bits(x) if dtype == BF16 else x


def _f64(x, dtype):
    return (bf16_bits_to_f32(x) if dtype == BF16 else np.asarray(x, np.float32)).astype(np.float64)


def _inputs(s: Shape, seed: int):
    rng = np.random.default_rng(seed)
    return {
        "q": _rand((s.n_suffix, s.n_q_heads, s.head_dim), rng, s.dtype),
        "kp": _rand((s.n_prefix, s.n_kv_heads, s.head_dim), rng, s.dtype),
        "vp": _rand((s.n_prefix, s.n_kv_heads, s.head_dim), rng, s.dtype),
        "ks": _rand((s.n_suffix, s.n_kv_heads, s.head_dim), rng, s.dtype),
        "vs": _rand((s.n_suffix, s.n_kv_heads, s.head_dim), rng, s.dtype),
    }


# tiny shapes: GQA groups 1..4, partial last chunks, d not a power of two
SHAPES = [
    Shape(37, 3, 6, 2, 8, 5, BF16),
    Shape(64, 4, 4, 1, 16, 16, F32),
    Shape(50, 5, 8, 2, 12, 7, BF16, 0.37),
    Shape(9, 2, 3, 3, 4, 4, F32),
]


def _scale(s: Shape) -> float:
    return s.sm_scale if s.sm_scale > 0 else 1.0 / math.sqrt(s.head_dim)


def pin_partition():
    """Def. 4.1: m = ceil(n/c); the last chunk holds the remainder."""
    for n, c, m in [(5, 2, 3), (1024, 16, 64), (8192, 16, 512), (32768, 32, 1024),
                    (65536, 8, 8192), (131072, 32, 4096), (1, 1, 1), (0, 4, 0), (17, 32, 1)]:
        assert oracle.num_chunks(n, c) == m, (n, c)
    assert oracle.num_chunks(5, 0) == -1
    s = Shape(5, 1, 1, 1, 1, 2, F32)
    k = np.arange(5, dtype=np.float32)
    kd, vd = oracle.gather_chunks(s, k, k + 10, np.array([2], np.int32))
    assert kd.ravel().tolist() == [4.0, 0.0] and vd.ravel().tolist() == [14.0, 0.0]
    kd, _ = oracle.gather_chunks(s, k, k, np.array([0, 1], np.int32))
    assert kd.ravel().tolist() == [0.0, 1.0, 2.0, 3.0]


def pin_num_keep():
    """Budget: the 1024-token fp32 case states 25% of 64 chunks = 16 chunks."""
    assert oracle.num_keep(64, 0.25) == 16
    assert oracle.num_keep(10, 0.1) == 1 and oracle.num_keep(10, 1.0) == 10
    assert oracle.num_keep(3, 1e-6) == 1 and oracle.num_keep(0, 0.5) == 0
    assert oracle.num_keep(7, 0.5) == 4 and oracle.num_keep(7, 0.0) == -1


def pin_h1_scores():
    """Hand example: q=[1], keys [0,0,1,1], c=2: weights 1,1,e,e over 2+2e."""
    s = Shape(4, 1, 1, 1, 1, 2, F32, 1.0)
    a = oracle.token_importance(s, np.array([1.0], np.float32), np.array([0, 0, 1, 1], np.float32))
    ref = [1 / (2 + 2 * E), 1 / (2 + 2 * E), E / (2 + 2 * E), E / (2 + 2 * E)]
    assert np.allclose(a, ref, rtol=1e-15, atol=0), a
    A = oracle.chunk_scores(s, a)
    assert np.allclose(A, [1 / (1 + E), E / (1 + E)], rtol=1e-15, atol=0), A
    assert oracle.select_topk(A, 1).tolist() == [1]


def pin_h2_tie():
    """All keys equal: every chunk scores 1/2; the lower index wins the tie."""
    s = Shape(4, 1, 1, 1, 1, 2, F32, 1.0)
    a = oracle.token_importance(s, np.array([1.0], np.float32), np.zeros(4, np.float32))
    A = oracle.chunk_scores(s, a)
    assert A.tolist() == [0.5, 0.5], A
    assert oracle.select_topk(A, 1).tolist() == [0]
    assert oracle.select_topk(A, 2).tolist() == [0, 1]


def pin_importance_invariants():
    """Each softmax row sums to 1, so sum_j A_j = S*Hq; with q = 0 every row is
    uniform and A_j = S*Hq*|chunk j|/n."""
    for i, s in enumerate(SHAPES):
        x = _inputs(s, 100 + i)
        A = oracle.chunk_scores(s, oracle.token_importance(s, x["q"], x["kp"]))
        rows = s.n_suffix * s.n_q_heads
        assert abs(A.sum() - rows) <= 1e-12 * rows, (s, A.sum())
        zq = np.zeros_like(x["q"])
        A0 = oracle.chunk_scores(s, oracle.token_importance(s, zq, x["kp"]))
        lens = np.minimum(s.chunk_size, s.n_prefix - np.arange(s.n_chunks) * s.chunk_size)
        assert np.allclose(A0, rows * lens / s.n_prefix, rtol=1e-12, atol=0), (s, A0)


def pin_importance_vs_torch():
    """Token importance equals torch's fp64 softmax over prefix keys, summed over
    every query row of every head (GQA: head h reads KV head h // G)."""
    for i, s in enumerate(SHAPES):
        x = _inputs(s, 200 + i)
        a = oracle.token_importance(s, x["q"], x["kp"], threads=3)
        q = torch.from_numpy(_f64(x["q"], s.dtype))  # [S][Hq][d]
        k = torch.from_numpy(_f64(x["kp"], s.dtype))  # [n][Hkv][d]
        G = s.n_q_heads // s.n_kv_heads
        ref = torch.zeros(s.n_prefix, dtype=torch.float64)
        for h in range(s.n_q_heads):
            logits = _scale(s) * (q[:, h, :] @ k[:, h // G, :].T)
            ref += torch.softmax(logits, dim=-1).sum(0)
        assert np.allclose(a, ref.numpy(), rtol=1e-12, atol=1e-15), (s, np.abs(a - ref.numpy()).max())
        A = oracle.chunk_scores(s, a)
        pooled = [ref[j * s.chunk_size:(j + 1) * s.chunk_size].sum().item() for j in range(s.n_chunks)]
        assert np.allclose(A, pooled, rtol=1e-12, atol=1e-15)


def _brute_topk(A, k):
    """Exhaustive: among the k-subsets of maximal score sum, the lexicographically
    smallest ascending tuple (scores are small integers, so sums are exact)."""
    best = None
    for sub in itertools.combinations(range(len(A)), k):
        key = (-sum(A[j] for j in sub), sub)
        if best is None or key < best:
            best = key
    return list(best[1])


def pin_select_bruteforce():
    """Top-k with lowest-index tie-break against exhaustive subset search."""
    rng = np.random.default_rng(7)
    for m in range(1, 11):
        for trial in range(3):
            A = rng.integers(0, 4, size=m).astype(np.float64)
            for k in range(1, m + 1):
                assert oracle.select_topk(A, k).tolist() == _brute_topk(A.tolist(), k), (A, k)


def pin_select_special_values():
    """NaN ranks below -inf, -0.0 ties with +0.0 (lower index wins)."""
    A = np.array([np.nan, -0.0, 0.0, -np.inf, np.inf, 1.0, np.nan, -1.0])
    order = [4, 5, 1, 2, 7, 3, 0, 6]
    for k in range(1, len(A) + 1):
        assert oracle.select_topk(A, k).tolist() == sorted(order[:k]), k


def pin_attention_h1():
    """Hand example extended: V=[1,2,3,4], suffix key 0 / value 10.
    keep chunk {1}: weights e,e,1 over values 3,4,10 -> (7e+10)/(2e+1).
    dense: weights 1,1,e,e,1 over 1,2,3,4,10 -> (13+7e)/(3+2e)."""
    s = Shape(4, 1, 1, 1, 1, 2, F32, 1.0)
    args = dict(q=np.array([1.0], np.float32), k_prefix=np.array([0, 0, 1, 1], np.float32),
                v_prefix=np.array([1, 2, 3, 4], np.float32), k_suffix=np.array([0.0], np.float32),
                v_suffix=np.array([10.0], np.float32))
    o = oracle.sparse_attn(s, sel=np.array([1], np.int32), **args)
    assert abs(o.item() - (7 * E + 10) / (2 * E + 1)) <= 1e-14, o
    o = oracle.dense_attn(s, **args)
    assert abs(o.item() - (13 + 7 * E) / (3 + 2 * E)) <= 1e-14, o
    o = oracle.sparse_attn(s, sel=np.array([0], np.int32), **args)
    assert abs(o.item() - 13.0 / 3.0) <= 1e-14, o


def _sdpa(s: Shape, x, visible_prefix):
    """torch fp64 SDPA over [prefix ; suffix] keys with an explicit boolean mask."""
    q = torch.from_numpy(_f64(x["q"], s.dtype)).permute(1, 0, 2)  # [Hq][S][d]
    G = s.n_q_heads // s.n_kv_heads
    k = torch.cat([torch.from_numpy(_f64(x["kp"], s.dtype)), torch.from_numpy(_f64(x["ks"], s.dtype))])
    v = torch.cat([torch.from_numpy(_f64(x["vp"], s.dtype)), torch.from_numpy(_f64(x["vs"], s.dtype))])
    k = k.permute(1, 0, 2).repeat_interleave(G, dim=0).contiguous()
    v = v.permute(1, 0, 2).repeat_interleave(G, dim=0).contiguous()
    n, S = s.n_prefix, s.n_suffix
    mask = torch.zeros(S, n + S, dtype=torch.bool)
    mask[:, :n] = torch.from_numpy(visible_prefix)[None, :]
    mask[:, n:] = torch.tril(torch.ones(S, S, dtype=torch.bool))
    o = torch.nn.functional.scaled_dot_product_attention(q, k, v, attn_mask=mask, scale=_scale(s))
    return o.permute(1, 0, 2).numpy()


def pin_attention_vs_sdpa():
    """Dense and sparse attention equal torch fp64 SDPA with the matching mask."""
    for i, s in enumerate(SHAPES):
        x = _inputs(s, 300 + i)
        dense = oracle.dense_attn(s, x["q"], x["kp"], x["vp"], x["ks"], x["vs"])
        ref = _sdpa(s, x, np.ones(s.n_prefix, bool))
        assert np.allclose(dense, ref, rtol=0, atol=1e-12), (s, np.abs(dense - ref).max())
        rng = np.random.default_rng(400 + i)
        k = max(1, s.n_chunks // 2)
        sel = np.sort(rng.choice(s.n_chunks, size=k, replace=False)).astype(np.int32)
        if s.n_chunks - 1 not in sel:  # include the partial last chunk
            sel[-1] = s.n_chunks - 1
            sel = np.unique(sel).astype(np.int32)
        vis = np.zeros(s.n_prefix, bool)
        for j in sel:
            vis[j * s.chunk_size:(j + 1) * s.chunk_size] = True
        sparse = oracle.sparse_attn(s, x["q"], x["kp"], x["vp"], sel, x["ks"], x["vs"])
        ref = _sdpa(s, x, vis)
        assert np.allclose(sparse, ref, rtol=0, atol=1e-12), (s, np.abs(sparse - ref).max())
        rows = np.array([0, s.n_suffix * s.n_q_heads - 1, 1], np.int64)
        part = oracle.sparse_attn(s, x["q"], x["kp"], x["vp"], sel, x["ks"], x["vs"], row_ids=rows)
        full = sparse.reshape(-1, s.head_dim)
        assert np.array_equal(part, full[rows])


def pin_keep_all_is_dense():
    """With every chunk kept the sparse path visits the dense key sequence: equal bit for bit."""
    for i, s in enumerate(SHAPES):
        x = _inputs(s, 500 + i)
        sel = np.arange(s.n_chunks, dtype=np.int32)
        a = oracle.sparse_attn(s, x["q"], x["kp"], x["vp"], sel, x["ks"], x["vs"])
        b = oracle.dense_attn(s, x["q"], x["kp"], x["vp"], x["ks"], x["vs"])
        assert np.array_equal(a, b), s


def pin_attention_constant_v():
    """Softmax weights sum to 1: constant values come back unchanged."""
    for i, s in enumerate(SHAPES):
        x = _inputs(s, 600 + i)
        const = np.full_like(x["vp"], to_bf16_bits(np.float32(1.5)) if s.dtype == BF16 else 1.5)
        consts = np.full_like(x["vs"], to_bf16_bits(np.float32(1.5)) if s.dtype == BF16 else 1.5)
        sel = np.arange(0, s.n_chunks, 2, dtype=np.int32)
        o = oracle.sparse_attn(s, x["q"], x["kp"], const, sel, x["ks"], consts)
        assert np.allclose(o, 1.5, rtol=1e-14, atol=0), s


def pin_gather():
    """Gather is a byte copy of whole chunk spans, zero past n."""
    s = Shape(37, 1, 2, 2, 8, 5, BF16)
    x = _inputs(s, 700)
    sel = np.array([0, 3, 7], np.int32)  # chunk 7 is the partial one (35, 36)
    kd, vd = oracle.gather_chunks(s, x["kp"], x["vp"], sel)
    for u, j in enumerate(sel):
        lo, hi = j * 5, min(j * 5 + 5, 37)
        assert np.array_equal(kd[u * 5:u * 5 + hi - lo], x["kp"][lo:hi])
        assert np.array_equal(vd[u * 5:u * 5 + hi - lo], x["vp"][lo:hi])
        assert not kd[u * 5 + hi - lo:(u + 1) * 5].any() and not vd[u * 5 + hi - lo:(u + 1) * 5].any()


def pin_accounting():
    """Prefetch accounting is set algebra over chunk spans (Sec. 4.3.2)."""
    s = Shape(37, 1, 2, 2, 8, 5, BF16)
    per_tok = 2 * 2 * 8 * 2
    lens = {j: min(5, 37 - 5 * j) for j in range(8)}
    rng = np.random.default_rng(9)
    cases = [(np.array([1, 2, 7]), np.array([], int)),      # first layer: no prediction
             (np.array([1, 2, 7]), np.array([1, 2, 7])),    # perfect prediction
             (np.array([1, 2, 7]), np.array([0, 3, 4, 5, 6]))]  # complement
    for _ in range(20):
        cases.append((np.sort(rng.choice(8, 3, replace=False)), np.sort(rng.choice(8, 4, replace=False))))
    for sel, pred in cases:
        st = oracle.layer_accounting(s, sel, pred)
        S, P = set(sel.tolist()), set(pred.tolist())
        assert st["k"] == len(S) and st["hits"] == len(S & P)
        assert st["misses"] == len(S - P) and st["wasted"] == len(P - S)
        assert st["bytes_prefetch"] == sum(lens[j] for j in P) * per_tok
        assert st["bytes_demand"] == sum(lens[j] for j in S - P) * per_tok
        assert st["bytes_used"] == sum(lens[j] for j in S) * per_tok


def pin_paper_byte_accounting():
    """Byte figures the paper prints for Qwen2.5-7B (Sec. 4.2, Sec. 3)."""
    g = json.load(open(os.path.join(GOLDEN, "paper_byte_accounting.json")))
    m = g["qwen25_7b"]
    c = 16
    s = Shape(c, 1, 28, m["kv_heads"], m["head_dim"], c, BF16)
    st = oracle.layer_accounting(s, np.array([0]), np.array([], int))
    # K and V of one chunk in one layer; the paper's per-token figure is one of K or V over all layers
    per_token_one_tensor_all_layers = st["bytes_used"] // 2 // c * m["layers"]
    assert round(per_token_one_tensor_all_layers / 1024) == g["per_token_kb_approx"]
    block = per_token_one_tensor_all_layers * g["block_tokens"]
    assert abs(block / 1000 - g["block_kb_approx"]) / g["block_kb_approx"] < 0.02
    assert g["block_tokens"] // g["useful_tokens_per_block"] == g["read_amplification_block"]
    amp = g["example_blocks"] * g["block_tokens"] / g["example_needed_tokens"]
    assert int(amp) == g["example_read_amplification"]


def pin_planted_chunks_found():
    """The 1024-token fp32 workload plants 3 chunks along the query direction;
    the full layer keeps all of them among its 16 chunks."""
    import synth
    w = synth.WORKLOADS["c1_f32_1k"]
    t = synth.layer_tensors(w, 0)
    s = Shape(w.n_prefix, w.n_suffix, w.n_q_heads, w.n_kv_heads, w.head_dim, w.chunk_size, F32)
    A, sel, out = oracle.reprefill_layer(s, w.keep_ratio, t["q"], t["k_prefix"], t["v_prefix"],
                                         t["k_suffix"], t["v_suffix"])
    assert len(sel) == 16
    assert set(synth.heavy_sets(w)[0].tolist()) <= set(sel.tolist())
    assert abs(A.sum() - w.n_suffix * w.n_q_heads) < 1e-9


def pin_period_rule():
    """Periods (Def. 4.2): layers cut from layer 0 into runs of p share the set
    of the run's first layer; the prefetch prediction is the previous layer's
    set (Sec. 4.3.2), so every layer but a Period's first is predicted exactly."""
    # brute force: enumerate the Periods
    for p in range(1, 10):
        for start in range(0, 60, p):
            for layer in range(start, start + p):
                assert oracle.period_first_layer(layer, p) == start
    assert [oracle.period_first_layer(l, 8) for l in (0, 7, 8, 13, 16)] == [0, 0, 8, 8, 16]
    for bad in ((3, 0), (-1, 2)):
        try:
            oracle.period_first_layer(*bad)
        except ValueError:
            continue
        raise AssertionError("accepted an invalid period or layer")
    sets = [np.array([1, 2]), None, np.array([3, 5]), None, np.array([0, 7])]
    pred = oracle.period_prediction(sets, 2)
    assert [list(x) for x in pred] == [[], [1, 2], [1, 2], [3, 5], [3, 5]]
    s = Shape(40, 1, 2, 2, 8, 5, BF16)
    for l in (1, 3):  # layers past a Period's first: all hits, nothing on demand
        used = sets[oracle.period_first_layer(l, 2)]
        st = oracle.layer_accounting(s, used, pred[l])
        assert st["hits"] == 2 and st["misses"] == 0 and st["bytes_demand"] == 0
    # period 1 is per-layer selection: every prediction is the previous set
    per_layer = [np.array([i, i + 1]) for i in range(4)]
    assert [list(x) for x in oracle.period_prediction(per_layer, 1)] == [[], [0, 1], [1, 2], [2, 3]]


def pin_io_paper_examples():
    """Read amplification figures the paper prints (Sec. 4.2; Sec. 3, Motivation 1)."""
    g = json.load(open(os.path.join(GOLDEN, "paper_byte_accounting.json")))
    b = g["block_tokens"]
    useful = g["useful_tokens_per_block"]
    # one 16-token ContiguousChunk inside a 64-token block: the block store reads 4x
    r = oracle.io_account(b, useful, [1], b)
    assert r["tokens_selected"] == useful and r["blocks"] == 1 and r["tokens_block"] == b
    assert r["tokens_block"] // r["tokens_selected"] == g["read_amplification_block"]
    # a store whose blocks are the ContiguousChunks reads only what is needed
    r = oracle.io_account(b, useful, [1], useful)
    assert r["tokens_block"] == r["tokens_selected"] == useful
    # 11 needed tokens over 9 blocks (token-level selection, c = 1): 52x
    nb, need = g["example_blocks"], g["example_needed_tokens"]
    toks = list(range(need - nb + 1)) + [b * i + 7 for i in range(1, nb)]
    r = oracle.io_account(nb * b, 1, toks, b)
    assert r["tokens_selected"] == need and r["blocks"] == nb
    assert int(r["tokens_block"] / r["tokens_selected"]) == g["example_read_amplification"]


def pin_io_closed_forms():
    """Closed forms of block read accounting."""
    # everything selected: both stores read the whole prefix once, in one run
    for n, c, b in ((1000, 16, 64), (1001, 32, 64), (77, 5, 9)):
        m = -(-n // c)
        r = oracle.io_account(n, c, np.arange(m), b)
        assert r == {"tokens_selected": n, "runs": 1, "blocks": -(-n // b), "tokens_block": n}
    # nothing selected
    assert oracle.io_account(100, 8, [], 64) == dict(tokens_selected=0, runs=0, blocks=0,
                                                     tokens_block=0)
    # blocks of one token, or chunks that are whole aligned blocks: no amplification
    rng = np.random.default_rng(5)
    for n, c, b in ((4096, 16, 1), (4096, 64, 64), (4096, 128, 64), (5000, 64, 32)):
        sel = np.sort(rng.choice(-(-n // c), size=20, replace=False))
        r = oracle.io_account(n, c, sel, b)
        assert r["tokens_block"] == r["tokens_selected"]
    # a short last chunk and a short last block: n=5, c=2 (chunk 2 = token 4), b=4
    assert oracle.io_account(5, 2, [2], 4) == dict(tokens_selected=1, runs=1, blocks=1,
                                                   tokens_block=1)
    assert oracle.io_account(5, 2, [1], 4) == dict(tokens_selected=2, runs=1, blocks=1,
                                                   tokens_block=4)
    # chunk 1 = tokens 2,3 and chunk 2 = token 4 straddle blocks 0 and 1
    assert oracle.io_account(5, 2, [1, 2], 4) == dict(tokens_selected=3, runs=1, blocks=2,
                                                      tokens_block=5)


def pin_io_vs_set_algebra():
    """Random selections against a set formulation: the distinct block ids of the
    selected tokens, with run starts taken from index gaps."""
    rng = np.random.default_rng(11)
    for trial in range(40):
        n = int(rng.integers(1, 3000))
        c = int(rng.choice([1, 3, 4, 8, 16, 32, 64]))
        b = int(rng.choice([1, 7, 16, 64, 100]))
        m = -(-n // c)
        k = int(rng.integers(0, m + 1))
        sel = np.sort(rng.choice(m, size=k, replace=False))
        tokens = np.concatenate([np.arange(j * c, min((j + 1) * c, n)) for j in sel]) \
            if k else np.zeros(0, np.int64)
        blk = np.unique(tokens // b)
        expect = {"tokens_selected": int(tokens.size),
                  "runs": int(k and 1 + np.count_nonzero(np.diff(sel) != 1)),
                  "blocks": int(blk.size),
                  "tokens_block": int(np.minimum(b, n - blk * b).sum())}
        assert oracle.io_account(n, c, rng.permutation(sel), b) == expect, (trial, n, c, b)


def pin_cache_hand_trace():
    """Sec. 4.5 rules traced by hand on a 2-slot GPU tier and a 1-slot CPU tier,
    with dyadic scores so every product is exact."""
    T0, T1, T2 = oracle.TIER_NONE, oracle.TIER_CPU, oracle.TIER_GPU
    c = oracle.Cache(6, 2, 1, oracle.CACHE_ATTENTION)
    # keys 1, 2 fill the GPU tier; key 3 (S=.25) displaces key 2 (S=.125) to the CPU tier
    w, n = c.access([1, 2, 3], [0.5, 0.125, 0.25])
    assert list(w) == [T0, T0, T0] and n["misses"] == 3 and n["demoted"] == 1
    assert list(c.state()[2]) == [T0, T2, T1, T2, T0, T0]
    # key 2 found in the CPU tier: I=.25, F=2, S=.5 outranks key 3 (.25), which goes down;
    # key 4 (S=.375) loses to the GPU tier's weakest (key 1: S=.5, older than key 2's .5),
    # then displaces key 3 (.25) from the CPU tier, which leaves memory
    w, n = c.access([2, 4], [0.125, 0.375])
    assert list(w) == [T1, T0] and n == dict(hits_gpu=0, hits_cpu=1, misses=4, demoted=2,
                                             dropped=1)
    assert list(c.state()[2]) == [T0, T2, T2, T0, T1, T0]
    # key 3 returns with I=.75, F=2, S=1.5: key 1 goes down, key 4 leaves memory
    w, n = c.access([3], [0.5])
    assert list(w) == [T0] and n == dict(hits_gpu=0, hits_cpu=1, misses=5, demoted=3, dropped=2)
    I, F, tier = c.state()
    assert list(tier) == [T0, T1, T2, T2, T0, T0]
    assert list(I) == [0, 0.5, 0.25, 0.75, 0.375, 0] and list(F) == [0, 1, 2, 2, 1, 0]
    c.close()
    # the same stream ranked by frequency alone: ties go to the more recent access
    c = oracle.Cache(6, 2, 1, oracle.CACHE_LFU)
    c.access([1, 2, 3], [0.5, 0.125, 0.25])  # key 3 displaces key 1 (equal F, older)
    assert list(c.state()[2]) == [T0, T1, T2, T2, T0, T0]
    w, n = c.access([2, 4], [0.125, 0.375])  # key 4 displaces key 3, which displaces key 1
    assert list(w) == [T2, T0] and n["hits_gpu"] == 1 and n["dropped"] == 1
    assert list(c.state()[2]) == [T0, T0, T2, T1, T2, T0]
    w, n = c.access([3], [0.5])  # key 3 (F=2) displaces key 4 (F=1) to the CPU tier
    assert list(w) == [T1] and list(c.state()[2]) == [T0, T0, T2, T2, T1, T0]
    c.close()
    # F read as loads into GPU or CPU memory: the same three requests place
    # every key as with F counting uses (each use loaded its chunk); then key 2,
    # used from the GPU tier, gains I but no F (S = .5 * 2 = 1 against 1.5 when
    # uses count), so when key 1 (CPU tier, S = 1 * 2 = 2) returns, it is key 2
    # that goes down -- with F counting uses, key 3 (S 1.5, older) goes down
    for policy, F_end, tier_end in (
            (oracle.CACHE_LOADS, [0, 2, 2, 2, 1, 0], [T0, T2, T1, T2, T0, T0]),
            (oracle.CACHE_ATTENTION, [0, 2, 3, 2, 1, 0], [T0, T2, T2, T1, T0, T0])):
        c = oracle.Cache(6, 2, 1, policy)
        c.access([1, 2, 3], [0.5, 0.125, 0.25])
        c.access([2, 4], [0.125, 0.375])
        w, n = c.access([3], [0.5])
        assert list(c.state()[2]) == [T0, T1, T2, T2, T0, T0]
        w, n = c.access([2], [0.25])
        assert list(w) == [T2]
        w, n = c.access([1], [0.5])
        I, F, tier = c.state()
        assert list(w) == [T1] and list(F) == F_end and list(tier) == tier_end
        assert list(I) == [0, 1.0, 0.5, 0.75, 0.375, 0]
        assert n == dict(hits_gpu=1, hits_cpu=2, misses=5, demoted=4, dropped=2)
        c.close()


def pin_cache_tiers_are_top_ranks():
    """With scores that only grow (A >= 0), the cascade keeps the GPU tier equal to
    the gpu_slots highest-ranked accessed keys under (S, latest access) and the
    CPU tier equal to the next cpu_slots; checked after every request of random
    streams by sorting every accessed key."""
    rng = np.random.default_rng(3)
    for policy in (oracle.CACHE_ATTENTION, oracle.CACHE_LFU, oracle.CACHE_LOADS):
        for n_keys, g, cpu in ((40, 5, 7), (200, 16, 0), (64, 0, 10), (30, 40, 40)):
            c = oracle.Cache(n_keys, g, cpu, policy)
            one = oracle.Cache(n_keys, g, cpu, policy)  # fed one key per call
            I = np.zeros(n_keys)
            F = np.zeros(n_keys, np.int64)
            last = np.zeros(n_keys, np.int64)
            clock = 0
            pop = rng.zipf(1.5, size=n_keys).astype(np.float64)
            pop /= pop.sum()
            for _ in range(60):
                cnt = int(rng.integers(1, min(12, n_keys) + 1))
                keys = rng.choice(n_keys, size=cnt, replace=False, p=pop)
                A = rng.choice([0.0, 0.25, 0.5, 1.0, 3.0], size=cnt)
                w, tot = c.access(keys, A)
                for u in range(cnt):  # a request is its keys taken in order
                    before = one.state()[2][keys[u]]
                    w1, tot1 = one.access(keys[u:u + 1], A[u:u + 1])
                    assert w1[0] == before == w[u]
                assert tot1 == tot
                for x, a, where in zip(keys, A, w):
                    I[x] += a
                    if policy != oracle.CACHE_LOADS or where != oracle.TIER_GPU:
                        F[x] += 1
                    clock += 1
                    last[x] = clock
                S = F.astype(np.float64) if policy == oracle.CACHE_LFU else I * F
                seen = np.flatnonzero(F > 0)
                order = seen[np.lexsort((-last[seen], -S[seen]))]
                tier = c.state()[2]
                assert set(np.flatnonzero(tier == oracle.TIER_GPU)) == set(order[:g])
                assert set(np.flatnonzero(tier == oracle.TIER_CPU)) == set(order[g:g + cpu])
            Io, Fo, _ = c.state()
            assert np.array_equal(Fo, F) and np.array_equal(Io, I)
            c.close()
            one.close()


ALL_PINS = [v for k, v in sorted(globals().items()) if k.startswith("pin_")]
