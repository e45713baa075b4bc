"""Helpers of the GPU parity tests: device copies of the seeded inputs, calls
through the C ABI, and the comparison rules against the oracle."""
from __future__ import annotations

import numpy as np
import torch

import oracle
import synth

DEV = "cuda"


def dev(a: np.ndarray) -> torch.Tensor:
    """numpy (float32 or uint16 bf16 bits) -> device tensor (float32 or bfloat16)."""
    a = np.ascontiguousarray(a)
    t = torch.from_numpy(a)
    if a.dtype == np.uint16:
        t = t.view(torch.bfloat16)
    return t.to(DEV)


def host_bits(t: torch.Tensor) -> np.ndarray:
    t = t.detach().cpu().contiguous()
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).numpy().view(np.uint16)
    return t.numpy()


def to_f64(t: torch.Tensor) -> np.ndarray:
    return t.detach().float().cpu().numpy().astype(np.float64)


def dims_of(w: synth.Workload):
    import paper_2601_13631_amd as ckv
    return ckv.make_dims(w.n_prefix, w.n_suffix, w.n_q_heads, w.n_kv_heads, w.head_dim,
                         w.chunk_size, ckv.DTYPE_F32 if w.dtype == "f32" else ckv.DTYPE_BF16,
                         w.sm_scale)


def oshape(w: synth.Workload) -> oracle.Shape:
    return oracle.Shape(w.n_prefix, w.n_suffix, w.n_q_heads, w.n_kv_heads, w.head_dim,
                        w.chunk_size, oracle.F32 if w.dtype == "f32" else oracle.BF16, w.sm_scale)


def workspace(nbytes: int) -> torch.Tensor:
    return torch.empty(max(nbytes, 256), dtype=torch.uint8, device=DEV)


def gpu_scores(w, t) -> torch.Tensor:
    import paper_2601_13631_amd as ckv
    d = dims_of(w)
    A = torch.empty(w.n_chunks, dtype=torch.float64, device=DEV)
    ws = workspace(ckv.score_workspace_bytes(d))
    ckv.score_chunks(d, t["q"], t["k_prefix"], A, ws)
    return A


def gpu_select(A: torch.Tensor, k: int) -> torch.Tensor:
    import paper_2601_13631_amd as ckv
    sel = torch.empty(k, dtype=torch.int32, device=DEV)
    ckv.select_topk_chunks(A, A.numel(), k, sel)
    return sel


def rel_err(a: np.ndarray, ref: np.ndarray) -> float:
    """Largest relative error; scores below 1e-30 of the total mass (under fp32's
    range relative to a row's maximum: their terms underflow to zero on the GPU)
    are compared against that floor instead of their own size."""
    floor = 1e-30 * float(np.abs(ref).sum())
    return float(np.max(np.abs(a - ref) / np.maximum(np.abs(ref), max(floor, 1e-300))))


# Relative score error allowed on the seeded workloads.  The arithmetic bounds
# a chunk score's error by ~2e-6 (fp32 logits, exp2 and per-chunk partials
# over at most one chunk, every cross-row sum in fp64); what the seeded
# workloads achieve is 2e-9 .. 6e-9, so they are held to 1e-7 and a loss of
# accuracy shows.  The worst-case bound is kept for inputs built to sit at
# the edge of fp32's range (the forced exact-recompute cases).
# The small shapes of the unit tests sum a chunk's score over few rows and
# tokens (20 rows of 4-token chunks in the smallest), so per-term rounding
# (fp32 exp2 within ~2 ulp, fp32 logits) does not average out: they are held
# to 4e-7, about three fp32 ulps of one term.
SCORE_RTOL = 1e-7
SCORE_RTOL_UNIT = 4e-7
SCORE_RTOL_BOUND = 2e-6


# Attention: a per-element bound from the arithmetic, not a blanket
# tolerance.  With u = 2^-8 (bf16's unit roundoff, round to nearest even) and
# a the same row's attention over |V| (the same softmax weights, so a >= |o|),
# the GPU's bf16 output differs from the fp64 oracle by at most
#   u |o|   the output's rounding to bf16;
#   u a     the numerators rounded to bf16 for the P V product (the
#           denominator sums them unrounded);
#   u a     each split's normalised partial stored in bf16 (the combine
#           weights sum to one);
# plus the fp32 effects -- logits accumulated over head_dim, O over a split's
# keys, the denominators and combine weights -- which stay below 2^-11 a.
# Each element is held to the smaller of that bound and the stated max-abs
# tolerance of 2e-2; the fp32 path is held to 1e-5 absolute.
BF16_U = 2.0 ** -8
ATTN_ATOL_BF16 = 2e-2
ATTN_ATOL_F32 = 1e-5


def _abs_vals(a: np.ndarray) -> np.ndarray:
    """|x| elementwise: bf16 bit patterns lose their sign bit, fp32 takes abs."""
    return a & np.uint16(0x7FFF) if a.dtype == np.uint16 else np.abs(a)


def attn_check(s: oracle.Shape, t: dict, sel: np.ndarray, got: np.ndarray, ref: np.ndarray,
               attn=None) -> tuple:
    """Checks the GPU's attention `got` against the oracle's `ref` (computed with
    attention function `attn`, default oracle.sparse_attn, over the kept set
    `sel` and the inputs `t`) element by element.  Returns (largest absolute
    error, largest error / bound)."""
    err = np.abs(got - ref)
    if s.dtype == oracle.F32:
        bound = ATTN_ATOL_F32
    else:
        attn = attn or oracle.sparse_attn
        a = attn(s, t["q"], t["k_prefix"], _abs_vals(t["v_prefix"]), sel, t["k_suffix"],
                 _abs_vals(t["v_suffix"]))
        bound = np.minimum(BF16_U * np.abs(ref) + (2 * BF16_U + 2.0 ** -11) * a + 1e-6,
                           ATTN_ATOL_BF16)
    ratio = float(np.max(err / bound))
    assert ratio <= 1.0, f"attention error {float(err.max()):.3e} exceeds its bound ({ratio:.3g} x)"
    return float(err.max()), ratio


def check_set(A_ref: np.ndarray, sel_gpu: np.ndarray, k: int, err: float, require: bool = True) -> dict:
    """Certified comparison of a top-k set.

    With e the measured relative score error: if A_ref(k) (1-e) > A_ref(k+1) (1+e)
    the set is certified and must equal the oracle's exactly; otherwise every
    chunk in the symmetric difference must have its oracle score inside the
    uncertainty band [A_ref(k+1)(1-e), A_ref(k)(1+e)].  With require=True an
    uncertified set fails the test (with its gap/error ratio).  Returns
    {"certified", "gap_over_err", "equal"}."""
    sel_ref = oracle.select_topk(A_ref, k)
    order = np.lexsort((np.arange(A_ref.size), -A_ref))
    kth = A_ref[order[k - 1]]
    nxt = A_ref[order[k]] if k < A_ref.size else -np.inf
    e = max(err, 1e-15)
    certified = bool(kth * (1 - e) > nxt * (1 + e))
    gap = float((kth - nxt) / kth) if np.isfinite(nxt) and kth > 0 else float("inf")
    ratio = gap / e
    equal = bool(np.array_equal(np.sort(sel_gpu), sel_ref))
    if certified:
        assert equal, "certified set differs"
    else:
        diff = set(sel_gpu.tolist()) ^ set(sel_ref.tolist())
        lo, hi = nxt * (1 - e) * (1 - 1e-12), kth * (1 + e) * (1 + 1e-12)
        for j in diff:
            assert lo <= A_ref[j] <= hi, f"chunk {j} outside the near-tie band"
        print(f"  uncertified set: boundary gap / score error = {ratio:.3g} (sets equal: {equal})",
              flush=True)
        assert not require, f"uncertified set (gap/error ratio {ratio:.3g}, sets equal: {equal})"
    return {"certified": certified, "gap_over_err": ratio, "equal": equal}
