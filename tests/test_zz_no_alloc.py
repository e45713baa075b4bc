"""The allocation-free layer step (ckv_reprefill_layer_noalloc) against the
layer step of an HBM-resident context (ckv_reprefill_layer), through the C ABI.

Three calls in a row on the fixed scratch array -- the 32K-token 7B-shaped
layer at full size, then a smaller ragged bf16 layer, then the 1K fp32 layer --
each compared bit for bit (chunk scores, kept set, output) with a context's
layer step on the same inputs; then the same with the scores and set kept in
the scratch (no output pointers); then a shape above the scratch maximum,
refused before anything is enqueued.
"""
import numpy as np
import pytest
import torch

import synth
from gpu_common import DEV, dev, dims_of

pytestmark = pytest.mark.gpu


def _inputs(w, layer):
    return {kk: dev(v) for kk, v in synth.layer_tensors(w, layer).items()}


def _outputs(w, k, tt):
    return (torch.full((w.n_chunks,), float("nan"), dtype=torch.float64, device=DEV),
            torch.full((k,), -1, dtype=torch.int32, device=DEV), torch.zeros_like(tt["q"]))


def test_noalloc_matches_layer_step():
    import paper_2601_13631_amd as ckv
    big = synth.WORKLOADS["c3_qwen7b_32k"]
    cases = [(big, 1), (big.scaled(n_prefix=3000, n_suffix=40, n_layers=1), 0),
             (synth.WORKLOADS["c1_f32_1k"], 0)]
    inputs = [_inputs(w, l) for w, l in cases]
    got = []
    for (w, _), tt in zip(cases, inputs):  # the calls in a row, each smaller than the last
        k = ckv.num_keep(w.n_chunks, w.keep_ratio)
        print(f"no-alloc call: {w.name} n={w.n_prefix} S={w.n_suffix} {w.dtype}", flush=True)
        A, sel, out = _outputs(w, k, tt)
        ckv.reprefill_layer_noalloc(dims_of(w), w.keep_ratio, tt["q"], tt["k_prefix"], tt["v_prefix"],
                                    tt["k_suffix"], tt["v_suffix"], out, chunk_scores=A, sel_idx=sel)
        got.append((A, sel, out))
    torch.cuda.synchronize()
    for (w, l), tt, (A, sel, out) in zip(cases, inputs, got):
        ctx = ckv.Context(dims_of(w), w.n_layers, w.keep_ratio, 0)
        A0, sel0, out0 = _outputs(w, ctx.k, tt)
        ctx.reprefill_layer(l, tt["q"], tt["k_suffix"], tt["v_suffix"], tt["k_prefix"], out0,
                            k_prefix=tt["k_prefix"], v_prefix=tt["v_prefix"], chunk_scores=A0,
                            sel_idx=sel0)
        torch.cuda.synchronize()
        ctx.close()
        assert torch.equal(A.view(torch.int64), A0.view(torch.int64)), w.name
        assert torch.equal(sel, sel0), w.name
        assert torch.equal(out.view(torch.int16 if out.dtype == torch.bfloat16 else torch.int32),
                           out0.view(torch.int16 if out0.dtype == torch.bfloat16 else torch.int32)), w.name
        # scores and set kept in the scratch: the same output
        out2 = torch.zeros_like(out)
        ckv.reprefill_layer_noalloc(dims_of(w), w.keep_ratio, tt["q"], tt["k_prefix"], tt["v_prefix"],
                                    tt["k_suffix"], tt["v_suffix"], out2)
        torch.cuda.synchronize()
        assert torch.equal(out2, out0), w.name
        print(f"  {w.name}: bitwise equal to the context's layer step", flush=True)


def test_noalloc_refuses_shapes_above_its_scratch():
    import paper_2601_13631_amd as ckv
    w = synth.WORKLOADS["c4_qwen14b_64k_c8"]  # ~0.7 GB of scoring partials
    tt = {kk: torch.empty(8, dtype=torch.bfloat16, device=DEV) for kk in
          ("q", "k_prefix", "v_prefix", "k_suffix", "v_suffix", "out")}
    with pytest.raises(ckv.CkvError) as e:
        ckv.reprefill_layer_noalloc(dims_of(w), w.keep_ratio, tt["q"], tt["k_prefix"], tt["v_prefix"],
                                    tt["k_suffix"], tt["v_suffix"], tt["out"])
    assert e.value.status == ckv.EINVAL and "maximum" in str(e.value)
