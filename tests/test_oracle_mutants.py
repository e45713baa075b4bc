"""Every plausible mistake planted in a copy of the oracle fails at least one pin.

Each mutant is a textual edit of ``oracle/ckv_oracle.c`` compiled into a
temporary library (CPU only).  The pins of ``oracle_pins.py`` are then run
against it; a mutant that passes every pin would mean the pins cannot see that
kind of mistake.
"""
import os
import subprocess

import pytest

import oracle
import oracle_pins

MUTANTS = {
    "logit_scale_dropped": ("logit[x] = c->scale * dot;", "logit[x] = dot;"),
    "max_not_tracked": ("if (logit[x] > mx) mx = logit[x];", ";"),
    "softmax_not_normalised": ("acc[x] += logit[x] / z;", "acc[x] += logit[x];"),
    "gqa_head_mapping": ("int64_t h = g * G + i;", "int64_t h = i * Hkv + g;"),
    "query_layout_transposed": ("const double* qr = c->q + (t * Hq + h) * d;\n    double mx",
                                "const double* qr = c->q + (h * S + t) * d;\n    double mx"),
    "pooling_drops_a_token": ("for (int64_t x = first; x < first + len; ++x) sum += a[x];",
                              "for (int64_t x = first; x < first + len - 1; ++x) sum += a[x];"),
    "select_ascending": ("if (x > y) return -1; /* higher", "if (x < y) return -1; /* higher"),
    "tie_break_highest_index": ("return (ia > ib) - (ia < ib);", "return (ia < ib) - (ia > ib);"),
    "nan_ranks_first": ("if (xn != yn) return xn ? 1 : -1;", "if (xn != yn) return xn ? -1 : 1;"),
    "suffix_diagonal_dropped": ("for (int64_t x = 0; x <= t; ++x) {\n    krow",
                                "for (int64_t x = 0; x < t; ++x) {\n    krow"),
    "suffix_not_causal": ("for (int64_t x = 0; x <= t; ++x) {\n    krow",
                          "for (int64_t x = 0; x < s->n_suffix; ++x) {\n    krow"),
    "attn_weights_unnormalised": ("double p = w[x] / z;", "double p = w[x];"),
    "attn_scale_dropped": ("w[x] = c->scale * dot;", "w[x] = dot;"),
    "attn_kv_head_mapping": ("int64_t t = id / Hq, h = id % Hq, g = h / G;",
                             "int64_t t = id / Hq, h = id % Hq, g = h % Hkv;"),
    "bf16_widen_shift": ("(uint32_t)((const uint16_t*)p)[i] << 16", "(uint32_t)((const uint16_t*)p)[i] << 15"),
    "gather_no_zero_fill": ("memset((char*)k_dst + u * slot + len, 0, slot - len);", ";"),
    "accounting_wasted_bytes": ("      st->wasted++;\n      st->bytes_prefetch += chunk_len(s, pred[b]) * per_token;",
                                "      st->wasted++;"),
    "keep_floor": ("double x = ceil(r * (double)m - 1e-9);", "double x = floor(r * (double)m);"),
    "chunk_count_floor": ("return (n + c - 1) / c;", "return n / c;"),
    "io_runs_count_chunks": ("if (chunk_marked[j] && (j == 0 || !chunk_marked[j - 1])) out->runs++;",
                             "if (chunk_marked[j]) out->runs++;"),
    "io_last_block_full": ("out->tokens_block += last - first;", "out->tokens_block += b;"),
    "io_block_decided_by_last_token": ("any |= token_marked[t];", "any = token_marked[t];"),
    "io_chunk_one_token_short": ("for (int64_t t = j * c; t < (j + 1) * c && t < n; ++t)",
                                 "for (int64_t t = j * c; t < (j + 1) * c - 1 && t < n; ++t)"),
    "cache_lfu_uses_importance": ("if (c->policy == CKVO_CACHE_LFU) return (double)c->F[x];",
                                  "if (c->policy == CKVO_CACHE_LFU) return c->I[x];"),
    "cache_score_is_importance": ("return c->I[x] * (double)c->F[x];", "return c->I[x];"),
    "cache_newer_leaves_first": ("return c->last[x] < c->last[y];", "return c->last[x] > c->last[y];"),
    "cache_gpu_evictions_dropped": ("    c->counts.demoted += admit_cpu(c, y);",
                                    "    c->counts.dropped++;"),
    "cache_cpu_never_evicts": ("  if (y >= 0 && leaves_before(c, y, x)) {\n    c->tier[y] = CKVO_TIER_NONE;\n    c->counts.dropped++;",
                               "  if (0) {\n    c->tier[y] = CKVO_TIER_NONE;\n    c->counts.dropped++;"),
    "cache_frequency_not_counted": ("c->F[x] += 1;", ";"),
    "cache_loads_counts_gpu_uses": ("if (c->policy != CKVO_CACHE_LOADS || was != CKVO_TIER_GPU) c->F[x] += 1;",
                                    "c->F[x] += 1;"),
    "cache_loads_skips_cpu_loads": ("if (c->policy != CKVO_CACHE_LOADS || was != CKVO_TIER_GPU) c->F[x] += 1;",
                                    "if (c->policy != CKVO_CACHE_LOADS || was == CKVO_TIER_NONE) c->F[x] += 1;"),
}


@pytest.fixture(scope="module")
def source():
    return open(oracle.SRC_PATH).read()


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutant_is_caught(name, source, tmp_path, monkeypatch):
    old, new = MUTANTS[name]
    assert source.count(old) == 1, f"mutation anchor for {name} not unique/present"
    src = tmp_path / "ckv_oracle.c"
    src.write_text(source.replace(old, new))
    hdr = os.path.join(os.path.dirname(oracle.SRC_PATH), "ckv_oracle.h")
    so = tmp_path / "libmutant.so"
    subprocess.run(["gcc", "-std=c11", "-O2", "-ffp-contract=off", "-fno-fast-math", "-fPIC",
                    "-shared", "-pthread", "-I", os.path.dirname(hdr), "-o", str(so), str(src),
                    "-lm"], check=True)
    monkeypatch.setattr(oracle, "_lib", oracle.load(str(so)))
    failed = []
    for pin in oracle_pins.ALL_PINS:
        try:
            pin()
        except Exception as e:  # AssertionError or an oracle error code
            failed.append(pin.__name__)
    assert failed, f"mutant {name} passed every pin"
