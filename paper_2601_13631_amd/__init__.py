"""Python binding of libckv, the MI355X (gfx950) Re-Prefill hot path of ContiguousKV.

Argument marshalling only: every function forwards to the C ABI declared in
``include/ckv.h`` (same names without the ``ckv_`` prefix).  Every step of the
path runs in the library's HIP kernels; torch supplies device memory and
streams.  There is no fallback: if ``libckv.so`` is missing or fails to load,
importing this package raises.

Tensor arguments are torch tensors on the current HIP device (or, where the C
ABI allows host memory, pinned host tensors); they are passed by data pointer.
``stream`` defaults to torch's current stream.
"""
from __future__ import annotations

import ctypes
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libckv.so")

OK, EINVAL, EUNSUPPORTED, EHIP, ENOMEM, ESTATE = range(6)
DTYPE_F32, DTYPE_BF16 = 0, 1
CTX_HOST_PREFIX, CTX_MATERIALIZE, CTX_STAGE_TIMING, CTX_SCORE_TIMING = 0x1, 0x2, 0x4, 0x8
CACHE_ATTENTION, CACHE_LFU, CACHE_LOADS = 0, 1, 2
STORE_DIRECT = 0x1
TIER_NONE, TIER_CPU, TIER_GPU = 0, 1, 2
STAGES = ("score", "finalize", "select", "move", "attn")

if not os.path.exists(LIB_PATH):
    raise ImportError(f"libckv.so not built at {LIB_PATH}; run `python paper_2601_13631_amd/build.py`")
_lib = ctypes.CDLL(LIB_PATH)


class Dims(ctypes.Structure):
    """``ckv_dims``: the problem shape."""
    _fields_ = [
        ("n_prefix", ctypes.c_int64),
        ("n_suffix", ctypes.c_int32),
        ("n_q_heads", ctypes.c_int32),
        ("n_kv_heads", ctypes.c_int32),
        ("head_dim", ctypes.c_int32),
        ("chunk_size", ctypes.c_int32),
        ("dtype", ctypes.c_int32),
        ("sm_scale", ctypes.c_float),
    ]

    @property
    def n_chunks(self) -> int:
        return num_chunks(self.n_prefix, self.chunk_size)


class LayerIO(ctypes.Structure):
    """``ckv_layer_io``."""
    _fields_ = [(f, ctypes.c_void_p) for f in (
        "q", "k_suffix", "v_suffix", "k_probe", "k_prefix", "v_prefix", "kv_host", "kv_host_next",
        "out", "chunk_scores", "sel_idx", "stream", "pred_idx")] + [("n_pred", ctypes.c_int64)]


class LayerStats(ctypes.Structure):
    """``ckv_layer_stats``."""
    _fields_ = [(f, ctypes.c_int64) for f in (
        "k", "hits", "misses", "wasted", "bytes_prefetch", "bytes_demand", "bytes_gathered",
        "cache_hits", "bytes_cache_fill", "bytes_storage")]

    def as_dict(self) -> dict:
        return {f: int(getattr(self, f)) for f, _ in self._fields_}


class IoCounts(ctypes.Structure):
    """``ckv_io_counts``."""
    _fields_ = [(f, ctypes.c_int64) for f in ("tokens_selected", "runs", "blocks", "tokens_block")]


class CacheCounts(ctypes.Structure):
    """``ckv_cache_counts``."""
    _fields_ = [(f, ctypes.c_int64) for f in ("hits_gpu", "hits_cpu", "misses", "demoted", "dropped")]


_P = ctypes.c_void_p
_DP = ctypes.POINTER(Dims)
_SIG = {
    "ckv_last_error": ([], ctypes.c_char_p),
    "ckv_version": ([], ctypes.c_char_p),
    "ckv_num_chunks": ([ctypes.c_int64, ctypes.c_int32], ctypes.c_int64),
    "ckv_num_keep": ([ctypes.c_int64, ctypes.c_double], ctypes.c_int64),
    "ckv_score_workspace_bytes": ([_DP], ctypes.c_size_t),
    "ckv_score_chunks": ([_DP, _P, _P, _P, _P, ctypes.c_size_t, _P], ctypes.c_int32),
    "ckv_select_workspace_bytes": ([ctypes.c_int64], ctypes.c_size_t),
    "ckv_select_topk_chunks": ([_P, ctypes.c_int64, ctypes.c_int64, _P, _P, ctypes.c_size_t, _P],
                               ctypes.c_int32),
    "ckv_gather_chunks": ([_DP, _P, _P, _P, ctypes.c_int64, _P, _P, _P], ctypes.c_int32),
    "ckv_attn_workspace_bytes": ([_DP, ctypes.c_int64], ctypes.c_size_t),
    "ckv_debug_attn_wide_addressing": ([ctypes.c_int32], ctypes.c_int32),
    "ckv_sparse_prefill_attn": ([_DP, _P, _P, _P, _P, ctypes.c_int64, _P, _P, _P, _P,
                                 ctypes.c_size_t, _P], ctypes.c_int32),
    "ckv_ctx_create": ([_DP, ctypes.c_int32, ctypes.c_double, ctypes.c_int32, ctypes.POINTER(_P)],
                       ctypes.c_int32),
    "ckv_ctx_set_host_layers": ([_P, ctypes.POINTER(_P), ctypes.c_int32], ctypes.c_int32),
    "ckv_ctx_inject_copy_error": ([_P, ctypes.c_int32], ctypes.c_int32),
    "ckv_ctx_destroy": ([_P], ctypes.c_int32),
    "ckv_ctx_reset": ([_P], ctypes.c_int32),
    "ckv_ctx_set_period": ([_P, ctypes.c_int32], ctypes.c_int32),
    "ckv_ctx_attach_cache": ([_P, _P], ctypes.c_int32),
    "ckv_ctx_attach_store": ([_P, _P], ctypes.c_int32),
    "ckv_ctx_set_subperiod": ([_P, ctypes.c_int32], ctypes.c_int32),
    "ckv_store_open": ([ctypes.c_char_p, ctypes.c_int64, ctypes.c_int64, ctypes.c_int32, ctypes.c_int32,
                        ctypes.POINTER(_P)], ctypes.c_int32),
    "ckv_store_close": ([_P], ctypes.c_int32),
    "ckv_store_read": ([_P, _P, ctypes.c_int64, _P], ctypes.c_int32),
    "ckv_ctx_stage_times": ([_P, ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_int64)],
                            ctypes.c_int32),
    "ckv_reprefill_layer": ([_P, ctypes.c_int32, ctypes.POINTER(LayerIO),
                             ctypes.POINTER(LayerStats)], ctypes.c_int32),
    "ckv_reprefill_layer_noalloc": ([_DP, ctypes.c_double, _P, _P, _P, _P, _P, _P, _P, _P, _P],
                                    ctypes.c_int32),
    "ckv_io_account": ([ctypes.c_int64, ctypes.c_int32, _P, ctypes.c_int64, ctypes.c_int32,
                        ctypes.POINTER(IoCounts)], ctypes.c_int32),
    "ckv_cache_create": ([ctypes.c_int64, ctypes.c_int64, ctypes.c_int64, ctypes.c_int32,
                          ctypes.POINTER(_P)], ctypes.c_int32),
    "ckv_cache_destroy": ([_P], ctypes.c_int32),
    "ckv_cache_access": ([_P, _P, _P, ctypes.c_int64, _P, ctypes.POINTER(CacheCounts)],
                         ctypes.c_int32),
    "ckv_cache_lookup": ([_P, _P, ctypes.c_int64, _P], ctypes.c_int32),
    "ckv_cache_state": ([_P, _P, _P, _P], ctypes.c_int32),
    "ckv_cache_resident": ([_P, ctypes.c_int32, _P, ctypes.c_int64, ctypes.POINTER(ctypes.c_int64)],
                           ctypes.c_int32),
}
for _name, (_args, _res) in _SIG.items():
    _f = getattr(_lib, _name)
    _f.argtypes = _args
    _f.restype = _res

EXPORTED = tuple(_SIG)

# a valid host address for an empty caller prediction (n_pred = 0 with a
# non-NULL pred_idx); nothing is read from it
_EMPTY_PRED = (ctypes.c_int32 * 1)()
_EMPTY_PRED_ADDR = ctypes.addressof(_EMPTY_PRED)


class CkvError(RuntimeError):
    def __init__(self, status: int, what: str):
        msg = _lib.ckv_last_error().decode(errors="replace")
        super().__init__(f"{what} returned {status}: {msg}")
        self.status = status


def _check(status: int, what: str) -> None:
    if status != OK:
        raise CkvError(status, what)


def _ptr(t) -> int | None:
    if t is None:
        return None
    if isinstance(t, int):
        return t
    return t.data_ptr()


def _stream(stream) -> int | None:
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def version() -> str:
    return _lib.ckv_version().decode()


def last_error() -> str:
    return _lib.ckv_last_error().decode(errors="replace")


def num_chunks(n: int, c: int) -> int:
    return int(_lib.ckv_num_chunks(n, c))


def num_keep(m: int, r: float) -> int:
    return int(_lib.ckv_num_keep(m, r))


def make_dims(n_prefix, n_suffix, n_q_heads, n_kv_heads, head_dim, chunk_size, dtype=DTYPE_BF16,
              sm_scale=0.0) -> Dims:
    return Dims(n_prefix, n_suffix, n_q_heads, n_kv_heads, head_dim, chunk_size, dtype, sm_scale)


def score_workspace_bytes(dims: Dims) -> int:
    return int(_lib.ckv_score_workspace_bytes(ctypes.byref(dims)))


def score_chunks(dims: Dims, q, k_prefix, chunk_scores, ws, stream=None) -> None:
    _check(_lib.ckv_score_chunks(ctypes.byref(dims), _ptr(q), _ptr(k_prefix), _ptr(chunk_scores),
                                 _ptr(ws), ws.numel() * ws.element_size() if ws is not None else 0,
                                 _stream(stream)), "ckv_score_chunks")


def select_workspace_bytes(m: int) -> int:
    return int(_lib.ckv_select_workspace_bytes(m))


def select_topk_chunks(chunk_scores, m: int, k: int, sel_idx, ws=None, stream=None) -> None:
    nbytes = ws.numel() * ws.element_size() if ws is not None else 0
    _check(_lib.ckv_select_topk_chunks(_ptr(chunk_scores), m, k, _ptr(sel_idx), _ptr(ws), nbytes,
                                       _stream(stream)), "ckv_select_topk_chunks")


def gather_chunks(dims: Dims, k_src, v_src, sel_idx, k: int, k_sel, v_sel, stream=None) -> None:
    _check(_lib.ckv_gather_chunks(ctypes.byref(dims), _ptr(k_src), _ptr(v_src), _ptr(sel_idx), k,
                                  _ptr(k_sel), _ptr(v_sel), _stream(stream)), "ckv_gather_chunks")


def attn_workspace_bytes(dims: Dims, k: int) -> int:
    return int(_lib.ckv_attn_workspace_bytes(ctypes.byref(dims), k))


def debug_attn_wide_addressing(force_wide: bool) -> None:
    """Test hook: every later attention launch reads K/V through 64-bit row
    addresses (the form sources past 4 GiB take) instead of 32-bit offsets."""
    _check(_lib.ckv_debug_attn_wide_addressing(1 if force_wide else 0),
           "ckv_debug_attn_wide_addressing")


def sparse_prefill_attn(dims: Dims, q, k_sel, v_sel, sel_idx, k: int, k_suffix, v_suffix, out,
                        ws=None, stream=None) -> None:
    nbytes = ws.numel() * ws.element_size() if ws is not None else 0
    _check(_lib.ckv_sparse_prefill_attn(ctypes.byref(dims), _ptr(q), _ptr(k_sel), _ptr(v_sel),
                                        _ptr(sel_idx), k, _ptr(k_suffix), _ptr(v_suffix), _ptr(out),
                                        _ptr(ws), nbytes, _stream(stream)),
           "ckv_sparse_prefill_attn")


NOALLOC_SCRATCH_BYTES = 64 << 20


def reprefill_layer_noalloc(dims: Dims, keep_ratio: float, q, k_prefix, v_prefix, k_suffix, v_suffix,
                            out, chunk_scores=None, sel_idx=None, stream=None) -> None:
    """``ckv_reprefill_layer_noalloc``: one HBM-resident layer step that allocates
    nothing (scratch in the library's fixed device array)."""
    _check(_lib.ckv_reprefill_layer_noalloc(ctypes.byref(dims), keep_ratio, _ptr(q), _ptr(k_prefix),
                                            _ptr(v_prefix), _ptr(k_suffix), _ptr(v_suffix),
                                            _ptr(out), _ptr(chunk_scores), _ptr(sel_idx),
                                            _stream(stream)),
           "ckv_reprefill_layer_noalloc")


class Context:
    """``ckv_ctx``: owns workspace, streams, events and (host-resident prefix) HBM slots."""

    def __init__(self, dims: Dims, n_layers: int, keep_ratio: float, flags: int = 0):
        self.dims = dims
        self._h = ctypes.c_void_p()
        _check(_lib.ckv_ctx_create(ctypes.byref(dims), n_layers, keep_ratio, flags,
                                   ctypes.byref(self._h)), "ckv_ctx_create")
        self.n_layers = n_layers
        self.k = num_keep(dims.n_chunks, keep_ratio)

    def reprefill_layer(self, layer: int, q, k_suffix, v_suffix, k_probe, out, k_prefix=None,
                        v_prefix=None, kv_host=None, kv_host_next=None, chunk_scores=None,
                        sel_idx=None, stream=None, pred_idx=None) -> dict:
        """``pred_idx``: this layer's predicted chunks (ascending; a host numpy
        array or sequence, possibly empty), or None for the context's own."""
        pred = None
        if pred_idx is not None:
            import numpy as np
            pred = np.ascontiguousarray(pred_idx, np.int32)
            if pred.size == 0:
                pred = np.zeros(1, np.int32)[:0]
        io = LayerIO(_ptr(q), _ptr(k_suffix), _ptr(v_suffix), _ptr(k_probe), _ptr(k_prefix),
                     _ptr(v_prefix), _ptr(kv_host), _ptr(kv_host_next), _ptr(out),
                     _ptr(chunk_scores), _ptr(sel_idx), _stream(stream),
                     None if pred is None else (pred.ctypes.data or _EMPTY_PRED_ADDR),
                     0 if pred is None else pred.size)
        st = LayerStats()
        _check(_lib.ckv_reprefill_layer(self._h, layer, ctypes.byref(io), ctypes.byref(st)),
               "ckv_reprefill_layer")
        return st.as_dict()

    def stage_times(self) -> tuple:
        """(per-stage total ms dict, number of layers) since creation or reset."""
        ms = (ctypes.c_double * len(STAGES))()
        n = ctypes.c_int64()
        _check(_lib.ckv_ctx_stage_times(self._h, ms, ctypes.byref(n)), "ckv_ctx_stage_times")
        return dict(zip(STAGES, list(ms))), int(n.value)

    def reset(self) -> None:
        _check(_lib.ckv_ctx_reset(self._h), "ckv_ctx_reset")

    def set_period(self, period: int) -> None:
        """Layers p*i .. p*i+p-1 share the set selected at layer p*i."""
        _check(_lib.ckv_ctx_set_period(self._h, period), "ckv_ctx_set_period")

    def attach_cache(self, cache) -> None:
        """Keeps the GPU tier of ``cache`` (a :class:`Cache`, or None to detach)
        in HBM slots for this host-resident context."""
        self._cache = cache  # the context must not outlive the cache it uses
        _check(_lib.ckv_ctx_attach_cache(self._h, cache._h if cache is not None else None),
               "ckv_ctx_attach_cache")

    def set_host_layers(self, stores) -> None:
        """Registers the pinned host store of every layer (a list of n_layers
        pinned tensors), or unregisters them (None)."""
        self._host_layers = stores  # kept alive while registered
        if stores is None:
            _check(_lib.ckv_ctx_set_host_layers(self._h, None, 0), "ckv_ctx_set_host_layers")
            return
        arr = (_P * len(stores))(*[_ptr(t) for t in stores])
        _check(_lib.ckv_ctx_set_host_layers(self._h, arr, len(stores)), "ckv_ctx_set_host_layers")

    def inject_copy_error(self, layer: int) -> None:
        """Test hook: the next run of ``layer`` fails at its demand copies (-1 disarms)."""
        _check(_lib.ckv_ctx_inject_copy_error(self._h, layer), "ckv_ctx_inject_copy_error")

    def set_subperiod(self, subperiod: int) -> None:
        """Storage reads up to subperiod - 1 layers ahead inside a Period."""
        _check(_lib.ckv_ctx_set_subperiod(self._h, subperiod), "ckv_ctx_set_subperiod")

    def attach_store(self, store) -> None:
        """Takes the chunks of this host-resident context from ``store`` (a
        :class:`Store`, or None to detach)."""
        self._store = store  # the context must not outlive the store it reads
        _check(_lib.ckv_ctx_attach_store(self._h, store._h if store is not None else None),
               "ckv_ctx_attach_store")

    def close(self) -> None:
        if self._h:
            _check(_lib.ckv_ctx_destroy(self._h), "ckv_ctx_destroy")
            self._h = ctypes.c_void_p()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def _host_ptr(a) -> int | None:
    """Address of a contiguous host numpy array."""
    return a.ctypes.data if a is not None and a.size else None


def io_account(n: int, c: int, sel_idx, block_tokens: int = 64) -> dict:
    """``ckv_io_account``: tokens read for the ascending chunk indices sel_idx (host)
    by a ContiguousChunk store and by a store of block_tokens-token blocks."""
    import numpy as np
    sel = np.ascontiguousarray(sel_idx, np.int32)
    out = IoCounts()
    _check(_lib.ckv_io_account(n, c, _host_ptr(sel), sel.size, block_tokens, ctypes.byref(out)),
           "ckv_io_account")
    return {f: int(getattr(out, f)) for f, _ in out._fields_}


class Cache:
    """``ckv_cache``: the attention-guided two-tier chunk cache (host memory)."""

    def __init__(self, n_keys: int, gpu_slots: int, cpu_slots: int, policy: int = CACHE_ATTENTION):
        self.n_keys = n_keys
        self._h = ctypes.c_void_p()
        _check(_lib.ckv_cache_create(n_keys, gpu_slots, cpu_slots, policy, ctypes.byref(self._h)),
               "ckv_cache_create")

    def access(self, keys, scores):
        """One request's used chunks; returns (tier each was found in, totals dict)."""
        import numpy as np
        keys = np.ascontiguousarray(keys, np.int64)
        scores = np.ascontiguousarray(scores, np.float64)
        if keys.size != scores.size:
            raise ValueError("keys and scores differ in length")
        where = np.zeros(keys.size, np.int8)
        cnt = CacheCounts()
        _check(_lib.ckv_cache_access(self._h, _host_ptr(keys), _host_ptr(scores), keys.size,
                                     _host_ptr(where), ctypes.byref(cnt)), "ckv_cache_access")
        return where, {f: int(getattr(cnt, f)) for f, _ in cnt._fields_}

    def lookup(self, keys):
        import numpy as np
        keys = np.ascontiguousarray(keys, np.int64)
        tier = np.zeros(keys.size, np.int8)
        _check(_lib.ckv_cache_lookup(self._h, _host_ptr(keys), keys.size, _host_ptr(tier)),
               "ckv_cache_lookup")
        return tier

    def state(self):
        """(I, F, tier) arrays over every key."""
        import numpy as np
        I = np.zeros(self.n_keys, np.float64)
        F = np.zeros(self.n_keys, np.int64)
        tier = np.zeros(self.n_keys, np.int8)
        _check(_lib.ckv_cache_state(self._h, _host_ptr(I), _host_ptr(F), _host_ptr(tier)),
               "ckv_cache_state")
        return I, F, tier

    def resident(self, tier: int):
        import numpy as np
        n = ctypes.c_int64()
        keys = np.zeros(self.n_keys, np.int64)
        _check(_lib.ckv_cache_resident(self._h, tier, _host_ptr(keys), keys.size, ctypes.byref(n)),
               "ckv_cache_resident")
        return keys[: n.value].copy()

    def close(self) -> None:
        if self._h:
            _check(_lib.ckv_cache_destroy(self._h), "ckv_cache_destroy")
            self._h = ctypes.c_void_p()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


class Store:
    """``ckv_store``: a file of fixed-size spans read by I/O threads (the storage tier)."""

    def __init__(self, path: str, n_keys: int, span_bytes: int, io_threads: int = 8, flags: int = 0):
        self.span_bytes = span_bytes
        self._h = ctypes.c_void_p()
        _check(_lib.ckv_store_open(os.fsencode(path), n_keys, span_bytes, io_threads, flags,
                                   ctypes.byref(self._h)), "ckv_store_open")

    def read(self, keys, dst) -> None:
        """Spans ``keys`` into ``dst`` (a host numpy array or tensor of len(keys) spans)."""
        import numpy as np
        keys = np.ascontiguousarray(keys, np.int64)
        nbytes = dst.nbytes if hasattr(dst, "nbytes") else dst.numel() * dst.element_size()
        if nbytes < keys.size * self.span_bytes:
            raise ValueError("destination smaller than the spans read")
        ptr = dst.ctypes.data if hasattr(dst, "ctypes") else dst.data_ptr()
        _check(_lib.ckv_store_read(self._h, _host_ptr(keys), keys.size, ptr), "ckv_store_read")

    def close(self) -> None:
        if self._h:
            _check(_lib.ckv_store_close(self._h), "ckv_store_close")
            self._h = ctypes.c_void_p()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
