"""GPU parity of each kernel against the oracle, called through the C ABI.

Bars: chunk indices bit-exact (certified sets; select itself on identical
scores always exact); gather byte-exact; chunk scores within rtol 4e-7 on these
small seeded shapes (1e-7 at the workloads' full sizes, where a chunk's score
sums thousands of terms; 2e-6, the bound derived from fp32 logits/exp2 with
fp64 cross-row sums, only for inputs built at the edge of fp32's range); attention
within the per-element bound of gpu_common.attn_check (bf16; derived from the
roundings the kernels make) or 1e-5 absolute (fp32) against the oracle run with
the GPU's own set.
"""
import numpy as np
import pytest
import torch

import oracle
import synth
from gpu_common import (DEV, SCORE_RTOL_UNIT as SCORE_RTOL, SCORE_RTOL_BOUND, attn_check, check_set, dev,
                        dims_of, gpu_scores, gpu_select, host_bits, oshape, rel_err, to_f64, workspace)

pytestmark = pytest.mark.gpu



def W(n, S, Hq, Hkv, d, c, keep=0.2, dtype="bf16", seed=1, alpha=1.5, sm_scale=0.0):
    return synth.Workload(f"t{n}_{S}_{Hq}_{Hkv}_{d}_{c}", 90, 1, n, S, Hq, Hkv, d, c, keep, dtype,
                          seed, alpha, "uniform", 0.05, 0.0, sm_scale=sm_scale)


SCORE_CASES = [
    W(1000, 9, 6, 2, 64, 16),            # ragged n, ragged rows, several key ranges
    W(777, 5, 4, 4, 128, 4),             # c=4, G=1
    W(1500, 11, 8, 2, 64, 8),            # c=8
    W(2048, 70, 4, 1, 128, 32),          # 280 rows: two row blocks
    W(3000, 3, 14, 2, 64, 64),           # c=64: chunks span two subtiles
    W(4100, 4, 5, 1, 128, 96),           # c=96, ragged last chunk
    W(20000, 2, 8, 8, 128, 32, seed=3),  # long prefix, large key ranges
    W(1024, 32, 4, 1, 64, 16, dtype="f32", seed=0, alpha=2.0),  # fp32 path
    W(600, 7, 3, 3, 64, 16, dtype="f32", sm_scale=0.31),
    W(5, 1, 2, 1, 64, 4),                # one query, prefix shorter than one subtile
    W(31, 1, 4, 2, 128, 32),             # a single partial chunk (m = 1)
    W(64, 1, 1, 1, 128, 64),             # exactly one stage and one chunk, G = 1
    # 4,096 chunks or more: the reduction's many-chunk kernel, with a ragged
    # row count (6 and 15 rows), a chunk count that is not a multiple of its
    # chunks per workgroup, and (c = 32) workgroups across segment boundaries
    W(131099, 3, 2, 1, 64, 32, seed=5),
    W(16411, 5, 3, 1, 128, 4, seed=6),
]


@pytest.mark.parametrize("w", SCORE_CASES, ids=lambda w: f"{w.name}_{w.dtype}")
def test_scores_match_oracle(w):
    t = synth.layer_tensors(w, 0)
    print(f"case {w.name} {w.dtype}", flush=True)
    A = gpu_scores(w, {k: dev(v) for k, v in t.items()})
    torch.cuda.synchronize()
    A = A.cpu().numpy()
    s = oshape(w)
    A_ref = oracle.chunk_scores(s, oracle.token_importance(s, t["q"], t["k_prefix"]))
    err = rel_err(A, A_ref)
    print(f"  max rel err {err:.3e}", flush=True)
    assert err <= SCORE_RTOL
    assert abs(A.sum() - w.n_suffix * w.n_q_heads) <= 1e-9 * w.n_suffix * w.n_q_heads
    k = oracle.num_keep(w.n_chunks, w.keep_ratio)
    sel = gpu_select(torch.from_numpy(A).to(DEV), k).cpu().numpy()
    check_set(A_ref, sel, k, err)


def test_scores_deterministic():
    w = SCORE_CASES[3]
    t = {k: dev(v) for k, v in synth.layer_tensors(w, 0).items()}
    a = gpu_scores(w, t).cpu().numpy()
    b = gpu_scores(w, t).cpu().numpy()
    assert np.array_equal(a.view(np.uint64), b.view(np.uint64))


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_scores_exact_fallback_on_overflow(dtype):
    """A key far above the first keys of its range overflows exp2 against the
    first-subtile reference; the workgroup must redo the range exactly."""
    n, d, c = 256, 64, 16
    q = np.zeros((1, 1, d), np.float32)
    q[0, 0, 0] = 8.0
    k = np.zeros((n, 1, d), np.float32)
    k[100, 0, 0] = 127.0          # logit 1016/8 = 127 -> exp2 arg ~183 against reference 0
    k[200:210, 0, 0] = -3.0
    w = W(n, 1, 1, 1, d, c, dtype=dtype)
    t = {"q": q, "k_prefix": k}
    if dtype == "bf16":
        t = {kk: synth.to_bf16_bits(v) for kk, v in t.items()}
    A = gpu_scores(w, {kk: dev(v) for kk, v in t.items()}).cpu().numpy()
    s = oshape(w)
    A_ref = oracle.chunk_scores(s, oracle.token_importance(s, t["q"], t["k_prefix"]))
    assert np.isfinite(A).all()
    assert rel_err(A, A_ref) <= SCORE_RTOL_BOUND
    assert int(np.argmax(A)) == 100 // c


SELECT_CASES = [1, 2, 7, 64, 512, 1000, 1024, 1025, 2048, 3000, 4096, 4097, 8192, 16384, 20000,
                70000]


@pytest.mark.parametrize("m", SELECT_CASES)
def test_select_exchange_exact(m):
    rng = np.random.default_rng(m)
    arrays = [rng.random(m) * 10,                              # distinct
              rng.integers(0, 5, m).astype(np.float64),        # heavy ties
              np.full(m, 0.25),                                 # all equal
              np.exp(rng.normal(0, 20, m))]                     # wide exponent range
    for A in arrays:
        for k in sorted({1, max(1, m // 10), max(1, m // 2), m}):
            sel = gpu_select(torch.from_numpy(A).to(DEV), k).cpu().numpy()
            ref = oracle.select_topk(A, k)
            assert np.array_equal(sel, ref), (m, k)


SPECIAL = np.array([np.nan, -0.0, 0.0, -np.inf, np.inf, 1.0, np.nan, -1.0, 5e-324, -5e-324])


def test_select_special_values():
    A = SPECIAL
    for k in range(1, len(A) + 1):
        sel = gpu_select(torch.from_numpy(A).to(DEV), k).cpu().numpy()
        assert np.array_equal(sel, oracle.select_topk(A, k)), k


# every selection path: 256 threads with 4 and with 8 keys each, 512 and 1024
# threads with 8, and the LDS-histogram kernel
@pytest.mark.parametrize("m", [1000, 1500, 4000, 6000, 9000, 20000])
def test_select_special_values_large(m):
    rng = np.random.default_rng(m + 1)
    A = rng.normal(0, 1, m) * np.exp(rng.normal(0, 30, m))  # both signs, wide exponents
    pos = rng.choice(m, 40 * len(SPECIAL), replace=False)
    A[pos] = np.tile(SPECIAL, 40)
    for k in sorted({1, 45, 80, 81, m // 3, m - 50, m}):
        sel = gpu_select(torch.from_numpy(A).to(DEV), k).cpu().numpy()
        assert np.array_equal(sel, oracle.select_topk(A, k)), (m, k)


@pytest.mark.parametrize("c,d,n", [(4, 128, 37), (16, 64, 1000), (32, 128, 1000), (64, 128, 3000)])
def test_gather_bytes(c, d, n):
    import paper_2601_13631_amd as ckv
    w = W(n, 2, 4, 2, d, c)
    t = synth.layer_tensors(w, 0)
    m = w.n_chunks
    rng = np.random.default_rng(c)
    sel = np.sort(rng.choice(m, size=max(1, m // 3), replace=False)).astype(np.int32)
    sel[-1] = m - 1  # the short last chunk
    sel = np.unique(sel).astype(np.int32)
    k = sel.size
    kd_ref, vd_ref = oracle.gather_chunks(oshape(w), t["k_prefix"], t["v_prefix"], sel)
    kp, vp = dev(t["k_prefix"]), dev(t["v_prefix"])
    kd = torch.full((k * c, w.n_kv_heads, d), 7.0, dtype=torch.bfloat16, device=DEV)
    vd = torch.full_like(kd, 7.0)
    ckv.gather_chunks(dims_of(w), kp, vp, torch.from_numpy(sel).to(DEV), k, kd, vd)
    assert np.array_equal(host_bits(kd), kd_ref) and np.array_equal(host_bits(vd), vd_ref)
    # same copy from pinned host memory
    kh = torch.from_numpy(t["k_prefix"]).view(torch.bfloat16).pin_memory()
    vh = torch.from_numpy(t["v_prefix"]).view(torch.bfloat16).pin_memory()
    kd.fill_(3.0)
    vd.fill_(3.0)
    ckv.gather_chunks(dims_of(w), kh, vh, torch.from_numpy(sel).to(DEV), k, kd, vd)
    assert np.array_equal(host_bits(kd), kd_ref) and np.array_equal(host_bits(vd), vd_ref)


def W2(n, S, Hq, Hkv, d, c, dtype="bf16", seed=5, sm_scale=0.0):
    return W(n, S, Hq, Hkv, d, c, dtype=dtype, seed=seed, sm_scale=sm_scale)


ATTN_CASES = [
    (W2(1000, 9, 6, 2, 64, 16), "third"),      # ragged rows, partial last chunk kept
    (W2(2048, 40, 28, 4, 128, 32), "tenth"),   # G=7, several row blocks, splits
    (W2(777, 5, 4, 4, 128, 4), "half"),        # c=4, G=1
    (W2(3000, 13, 10, 2, 64, 64), "tenth"),    # c=64
    (W2(512, 17, 8, 1, 128, 8), "none"),       # k=0: suffix only
    (W2(300, 33, 4, 2, 128, 16), "all"),       # every chunk (dense)
    (W2(4096, 256, 28, 4, 128, 32), "tenth"),  # suffix 256: long causal part
    (W2(1024, 32, 4, 1, 64, 16, dtype="f32"), "quarter"),
    (W2(500, 6, 3, 1, 64, 4, dtype="f32", sm_scale=0.2), "half"),
    (W2(5, 1, 2, 1, 64, 4), "all"),            # one query, both chunks, the last one partial
    (W2(31, 1, 4, 2, 128, 32), "all"),         # a single partial chunk
    (W2(33, 2, 2, 2, 64, 32), "half"),         # keeps only the one-row last chunk
]


def _sel_for(w, how, rng):
    m = w.n_chunks
    if how == "none":
        return np.zeros(0, np.int32)
    if how == "all":
        return np.arange(m, dtype=np.int32)
    frac = {"tenth": 0.1, "third": 1 / 3, "half": 0.5, "quarter": 0.25}[how]
    k = max(1, int(round(frac * m)))
    sel = np.sort(rng.choice(m, size=k, replace=False)).astype(np.int32)
    if m - 1 not in sel:
        sel[-1] = m - 1
    return np.unique(sel).astype(np.int32)


@pytest.mark.parametrize("w,how", ATTN_CASES, ids=lambda x: x.name if hasattr(x, "name") else x)
def test_attention_matches_oracle(w, how):
    import paper_2601_13631_amd as ckv
    print(f"case {w.name} {w.dtype} {how}", flush=True)
    t = synth.layer_tensors(w, 0)
    rng = np.random.default_rng(11)
    sel = _sel_for(w, how, rng)
    k = sel.size
    s = oshape(w)
    ref = oracle.sparse_attn(s, t["q"], t["k_prefix"], t["v_prefix"], sel, t["k_suffix"], t["v_suffix"])
    d = dims_of(w)
    kd_np, vd_np = oracle.gather_chunks(s, t["k_prefix"], t["v_prefix"], sel) if k else (None, None)
    # compact operands made by the GPU gather (checked byte-exact elsewhere)
    tt = {kk: dev(v) for kk, v in t.items()}
    sel_d = torch.from_numpy(sel).to(DEV) if k else torch.zeros(1, dtype=torch.int32, device=DEV)
    if k:
        kd = torch.empty((k * w.chunk_size, w.n_kv_heads, w.head_dim), dtype=tt["k_prefix"].dtype, device=DEV)
        vd = torch.empty_like(kd)
        ckv.gather_chunks(d, tt["k_prefix"], tt["v_prefix"], sel_d, k, kd, vd)
    else:
        kd = vd = None
    out = torch.empty_like(tt["q"])
    ws = workspace(ckv.attn_workspace_bytes(d, k))
    ckv.sparse_prefill_attn(d, tt["q"], kd, vd, sel_d if k else None, k, tt["k_suffix"], tt["v_suffix"],
                            out, ws)
    got = to_f64(out).reshape(ref.shape)
    err = float(np.abs(got - ref).max())
    print(f"  max abs err {err:.3e}", flush=True)
    _, ratio = attn_check(s, t, sel, got, ref)
    print(f"  {ratio:.2f} of its bound", flush=True)


def test_attention_deterministic():
    """Attention run twice (with split-K and its combine) is bitwise equal."""
    import paper_2601_13631_amd as ckv
    w = W2(4096, 256, 28, 4, 128, 32)
    t = synth.layer_tensors(w, 0)
    sel = _sel_for(w, "tenth", np.random.default_rng(5))
    k = sel.size
    d = dims_of(w)
    tt = {kk: dev(v) for kk, v in t.items()}
    sel_d = torch.from_numpy(sel).to(DEV)
    kd = torch.empty((k * w.chunk_size, w.n_kv_heads, w.head_dim), dtype=torch.bfloat16, device=DEV)
    vd = torch.empty_like(kd)
    ckv.gather_chunks(d, tt["k_prefix"], tt["v_prefix"], sel_d, k, kd, vd)
    ws = workspace(ckv.attn_workspace_bytes(d, k))
    outs = []
    for _ in range(2):
        out = torch.empty_like(tt["q"])
        ckv.sparse_prefill_attn(d, tt["q"], kd, vd, sel_d, k, tt["k_suffix"], tt["v_suffix"], out, ws)
        outs.append(out)
    torch.cuda.synchronize()
    assert torch.equal(outs[0].view(torch.int16), outs[1].view(torch.int16))


@pytest.mark.parametrize("w,how", [(W2(2048, 40, 28, 4, 128, 32), "tenth"), (W2(1000, 9, 6, 2, 64, 16), "third"),
                                   (W2(512, 17, 8, 1, 128, 8), "none")],
                         ids=lambda x: x.name if hasattr(x, "name") else x)
def test_attention_wide_addressing(w, how):
    """The 64-bit row addressing that sources past 4 GiB take, forced on small
    inputs: the standalone attention over the compact copy and the layer step
    reading the kept spans in place give bit-identical outputs either way."""
    import paper_2601_13631_amd as ckv
    print(f"case {w.name} {how}", flush=True)
    t = synth.layer_tensors(w, 0)
    sel = _sel_for(w, how, np.random.default_rng(13))
    k = sel.size
    d = dims_of(w)
    tt = {kk: dev(v) for kk, v in t.items()}
    sel_d = torch.from_numpy(sel).to(DEV) if k else torch.zeros(1, dtype=torch.int32, device=DEV)
    if k:
        kd = torch.empty((k * w.chunk_size, w.n_kv_heads, w.head_dim), dtype=torch.bfloat16, device=DEV)
        vd = torch.empty_like(kd)
        ckv.gather_chunks(d, tt["k_prefix"], tt["v_prefix"], sel_d, k, kd, vd)
    else:
        kd = vd = None
    ws = workspace(ckv.attn_workspace_bytes(d, k))

    def run_both():
        out = torch.empty_like(tt["q"])
        ckv.sparse_prefill_attn(d, tt["q"], kd, vd, sel_d if k else None, k, tt["k_suffix"],
                                tt["v_suffix"], out, ws)
        ctx = ckv.Context(d, 1, w.keep_ratio)
        A = torch.empty(w.n_chunks, dtype=torch.float64, device=DEV)
        lsel = torch.empty(ctx.k, dtype=torch.int32, device=DEV)
        lout = torch.empty_like(tt["q"])
        ctx.reprefill_layer(0, tt["q"], tt["k_suffix"], tt["v_suffix"], tt["k_prefix"], lout,
                            k_prefix=tt["k_prefix"], v_prefix=tt["v_prefix"], chunk_scores=A,
                            sel_idx=lsel)
        torch.cuda.synchronize()
        ctx.close()
        return out, lout

    narrow = run_both()
    ckv.debug_attn_wide_addressing(True)
    try:
        wide = run_both()
    finally:
        ckv.debug_attn_wide_addressing(False)
    for a, b in zip(narrow, wide):
        assert torch.equal(a.view(torch.int16), b.view(torch.int16))
    ref = oracle.sparse_attn(oshape(w), t["q"], t["k_prefix"], t["v_prefix"], sel, t["k_suffix"],
                             t["v_suffix"])
    attn_check(oshape(w), t, sel, to_f64(wide[0]).reshape(ref.shape), ref)
