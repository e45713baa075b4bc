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


def check_set(A_ref: np.ndarray, sel_gpu: np.ndarray, k: int, err: float) -> bool:
    """Certified comparison of a top-k set (returns True when certified).

    With e the measured relative score error: if A_ref(k) (1-e) > A_ref(k+1) (1+e)
    the set is certified and must equal the oracle's exactly; otherwise every
    chunk in the symmetric difference must have its oracle score inside the
    uncertainty band [A_ref(k+1)(1-e), A_ref(k)(1+e)]."""
    sel_ref = oracle.select_topk(A_ref, k)
    order = np.lexsort((np.arange(A_ref.size), -A_ref))
    kth = A_ref[order[k - 1]]
    nxt = A_ref[order[k]] if k < A_ref.size else -np.inf
    e = max(err, 1e-15)
    certified = kth * (1 - e) > nxt * (1 + e)
    if certified:
        assert np.array_equal(np.sort(sel_gpu), sel_ref), "certified set differs"
        return True
    diff = set(sel_gpu.tolist()) ^ set(sel_ref.tolist())
    lo, hi = nxt * (1 - e) * (1 - 1e-12), kth * (1 + e) * (1 + 1e-12)
    for j in diff:
        assert lo <= A_ref[j] <= hi, f"chunk {j} outside the near-tie band"
    return False
