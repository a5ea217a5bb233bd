"""ctypes binding of libtfe with the C ABI's names (argument marshalling only).

Pointer arguments accept an integer address, None, a torch tensor (its
``data_ptr()``) or a numpy array (its host address).  Streams accept an
integer handle, None (the default stream) or a ``torch.cuda.Stream``.
A negative status raises ``TfeError`` carrying ``tfe_last_error()``.
There is no fallback: if the library cannot be built or loaded, importing
fails.
"""
import ctypes
import os

from . import _build

TFE_OK = 0
TFE_ERR_INVALID_ARG = -1
TFE_ERR_DUPLICATE_KEY = -2
TFE_ERR_OOM = -3
TFE_ERR_HIP = -4
TFE_ERR_UNSUPPORTED = -5
TFE_F32, TFE_BF16 = 0, 1
TFE_GATE_SIGMOID, TFE_GATE_CONST = 0, 1
TFE_WEIGHT_LENGTH, TFE_WEIGHT_UNIFORM = 0, 1
TFE_FILL_INLINE, TFE_FILL_SIDE_STREAM = 0, 1


class tfe_table_desc(ctypes.Structure):
    _fields_ = [
        ("n_phrases", ctypes.c_int64),
        ("n_min", ctypes.c_int32),
        ("n_max", ctypes.c_int32),
        ("vocab", ctypes.c_int32),
        ("phrase_tokens", ctypes.c_void_p),
        ("phrase_len", ctypes.c_void_p),
        ("values", ctypes.c_void_p),
        ("dim", ctypes.c_int32),
        ("dtype", ctypes.c_int32),
        ("values_on_device", ctypes.c_int32),
        ("max_load_factor", ctypes.c_double),
        ("hbm_cache_rows", ctypes.c_int64),
        ("adopt_host_values", ctypes.c_int32),
        ("prefill_rows", ctypes.c_int64),
        ("miss_fill", ctypes.c_int32),
        ("pinned_rows", ctypes.c_int64),
        ("pageable_values", ctypes.c_void_p),
    ]


class tfe_stats(ctypes.Structure):
    _fields_ = [(n, ctypes.c_uint64) for n in (
        "calls", "positions", "hits", "cache_hits", "cache_misses", "prefetch_keys",
        "prefetch_found", "prefetch_filled", "prefetch_used", "host_bytes", "prefetch_dropped")]

    def as_dict(self):
        return {n: int(getattr(self, n)) for n, _ in self._fields_}


class TfeError(RuntimeError):
    def __init__(self, status, msg):
        super().__init__("libtfe status %d: %s" % (status, msg))
        self.status = status


def hip_runtimes():
    """Distinct HIP runtime libraries mapped into this process."""
    with open("/proc/self/maps") as f:
        return sorted({ln.split()[-1] for ln in f if "libamdhip64" in ln and "/" in ln})


def share_torch_hip_runtime():
    """Makes the next HIP-linked library use torch's HIP runtime, if torch
    is installed.  torch ships its own copy of the runtime under the same
    soname as the system one; loaded first, it satisfies the library's
    dependency.  Loaded second, it would be a second runtime in the process,
    and one of the two then sees no device."""
    try:
        import torch  # noqa: F401
    except ImportError:
        pass


def _load():
    if not os.path.exists(_build.SO):
        _build.build()
    share_torch_hip_runtime()
    L = ctypes.CDLL(_build.SO)
    if len(hip_runtimes()) > 1:
        raise ImportError("more than one HIP runtime in this process: %s" % hip_runtimes())
    vp, i32, i64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64
    sig = {
        "tfe_table_load": ([ctypes.POINTER(tfe_table_desc), vp, ctypes.POINTER(vp)], ctypes.c_int),
        "tfe_table_free": ([vp], ctypes.c_int),
        "tfe_lookup_inject": ([vp, vp, i32, i32, i32, vp, vp, vp, vp, vp, i32, ctypes.c_float, vp],
                              ctypes.c_int),
        "tfe_lookup_inject_multi": ([vp, vp, i32, i32, i32, vp, vp, vp, vp, i32, i32,
                                     ctypes.c_float, vp], ctypes.c_int),
        "tfe_prefetch": ([vp, vp, i32, vp, i32, i32, vp], ctypes.c_int),
        "tfe_prefetch_scored": ([vp, vp, i32, vp, vp, i32, i32, i32, vp], ctypes.c_int),
        "tfe_head_create": ([vp, i32, i32, i32, i32, ctypes.POINTER(vp)], ctypes.c_int),
        "tfe_head_topk": ([vp, vp, i32, i32, vp, vp, vp], ctypes.c_int),
        "tfe_head_free": ([vp], ctypes.c_int),
        "tfe_head_last_fault": ([vp, ctypes.POINTER(i64)], ctypes.c_int),
        "tfe_head_topk_noalloc": ([vp, i32, i32, vp, i32, i32, vp, vp, vp], ctypes.c_int),
        "tfe_ngram_release": ([], ctypes.c_int),
        "tfe_ngram_top": ([vp, i64, i32, i32, i64, i64, vp, vp, ctypes.POINTER(i64), vp],
                          ctypes.c_int),
        "tfe_get_stats": ([vp, ctypes.POINTER(tfe_stats)], ctypes.c_int),
        "tfe_reset_stats": ([vp], ctypes.c_int),
        "tfe_residency": ([vp, vp, i64, vp, vp], ctypes.c_int),
        "tfe_last_error": ([], ctypes.c_char_p),
        "tfe_memory_held": ([ctypes.POINTER(i64), ctypes.POINTER(i64)], ctypes.c_int),
        "tfe_index_capacity": ([i64, ctypes.c_double], i64),
        "tfe_index_build_host": ([vp, vp, i64, i32, i32, i32, vp, i64], ctypes.c_int),
        "tfe_index_probe_host": ([vp, i64, vp, i32, ctypes.POINTER(i32), ctypes.POINTER(i32),
                                  ctypes.POINTER(i64)], ctypes.c_int),
    }
    for name, (args, res) in sig.items():
        f = getattr(L, name)
        f.argtypes = args
        f.restype = res
    return L


lib = _load()
# Every symbol the C header declares (checked by the CPU test suite).
EXPORTED = ("tfe_table_load", "tfe_table_free", "tfe_lookup_inject", "tfe_lookup_inject_multi",
            "tfe_prefetch",
            "tfe_prefetch_scored", "tfe_head_create", "tfe_head_topk", "tfe_head_free",
            "tfe_head_last_fault", "tfe_head_topk_noalloc",
            "tfe_ngram_top", "tfe_ngram_release",
            "tfe_get_stats", "tfe_reset_stats", "tfe_residency", "tfe_last_error",
            "tfe_memory_held", "tfe_index_capacity",
            "tfe_index_build_host", "tfe_index_probe_host")


def addr(x):
    if x is None:
        return None
    if isinstance(x, int):
        return x
    if hasattr(x, "data_ptr"):
        return x.data_ptr()
    if hasattr(x, "ctypes"):
        return x.ctypes.data
    raise TypeError("cannot take the address of %r" % type(x))


def stream_handle(s):
    if s is None:
        return None
    if isinstance(s, int):
        return s
    return s.cuda_stream


def _check(st):
    if st < 0:
        raise TfeError(st, lib.tfe_last_error().decode())
    return st


def tfe_last_error():
    return lib.tfe_last_error().decode()


def tfe_memory_held():
    """(device bytes, pinned host bytes) the library holds right now."""
    d, p = ctypes.c_int64(), ctypes.c_int64()
    _check(lib.tfe_memory_held(ctypes.byref(d), ctypes.byref(p)))
    return d.value, p.value


def tfe_table_load(desc, stream=None):
    h = ctypes.c_void_p()
    _check(lib.tfe_table_load(ctypes.byref(desc), stream_handle(stream), ctypes.byref(h)))
    return h.value


def tfe_table_free(table):
    return _check(lib.tfe_table_free(table))


def tfe_lookup_inject(table, tokens, B, ctx, S, hidden_in, hidden_out, hit_mask, slot_ids,
                      match_len, gate, scale, stream=None):
    return _check(lib.tfe_lookup_inject(table, addr(tokens), B, ctx, S, addr(hidden_in),
                                        addr(hidden_out), addr(hit_mask), addr(slot_ids),
                                        addr(match_len), gate, scale, stream_handle(stream)))


def tfe_lookup_inject_multi(table, tokens, B, ctx, S, hidden_in, hidden_out, match_mask,
                            slot_ids, weighting, gate, scale, stream=None):
    return _check(lib.tfe_lookup_inject_multi(table, addr(tokens), B, ctx, S, addr(hidden_in),
                                              addr(hidden_out), addr(match_mask),
                                              addr(slot_ids), weighting, gate, scale,
                                              stream_handle(stream)))


def tfe_prefetch(table, tail, tail_len, candidates, B, K, side_stream=None):
    return _check(lib.tfe_prefetch(table, addr(tail), tail_len, addr(candidates), B, K,
                                   stream_handle(side_stream)))


def tfe_prefetch_scored(table, tail, tail_len, candidates, cand_prob, B, K, budget,
                        side_stream=None):
    return _check(lib.tfe_prefetch_scored(table, addr(tail), tail_len, addr(candidates),
                                          addr(cand_prob), B, K, budget,
                                          stream_handle(side_stream)))


def tfe_head_create(w_pref, vocab, dim, max_batch, max_k):
    h = ctypes.c_void_p()
    _check(lib.tfe_head_create(addr(w_pref), vocab, dim, max_batch, max_k, ctypes.byref(h)))
    return h.value


def tfe_head_topk(head, hidden, B, K, top_ids, top_prob, stream=None):
    return _check(lib.tfe_head_topk(head, addr(hidden), B, K, addr(top_ids), addr(top_prob),
                                    stream_handle(stream)))


def tfe_head_topk_noalloc(w_pref, vocab, dim, hidden, B, K, top_ids, top_prob, stream=None):
    return _check(lib.tfe_head_topk_noalloc(addr(w_pref), vocab, dim, addr(hidden), B, K,
                                            addr(top_ids), addr(top_prob), stream_handle(stream)))


def tfe_head_free(head):
    return _check(lib.tfe_head_free(head))


def tfe_head_last_fault(head):
    """Number (from 1) of the head's latest one-launch call that gave up, or 0."""
    n = ctypes.c_int64()
    _check(lib.tfe_head_last_fault(head, ctypes.byref(n)))
    return n.value


def tfe_ngram_top(tokens, n_tokens, vocab, n, skip, top, out_tuples, out_counts, stream=None):
    """Returns the number of ranks written."""
    w = ctypes.c_int64(0)
    _check(lib.tfe_ngram_top(addr(tokens), n_tokens, vocab, n, skip, top, addr(out_tuples),
                             addr(out_counts), ctypes.byref(w), stream_handle(stream)))
    return w.value


def tfe_ngram_release():
    return _check(lib.tfe_ngram_release())


def tfe_get_stats(table):
    s = tfe_stats()
    _check(lib.tfe_get_stats(table, ctypes.byref(s)))
    return s.as_dict()


def tfe_reset_stats(table):
    return _check(lib.tfe_reset_stats(table))


def tfe_residency(table, rows, n, out, stream=None):
    return _check(lib.tfe_residency(table, addr(rows), n, addr(out), stream_handle(stream)))


def tfe_index_capacity(n_phrases, max_load_factor=0.5):
    return int(lib.tfe_index_capacity(n_phrases, max_load_factor))


def tfe_index_build_host(phrase_tokens, phrase_len, n_phrases, n_min, n_max, vocab, slots,
                         capacity):
    return _check(lib.tfe_index_build_host(addr(phrase_tokens), addr(phrase_len), n_phrases,
                                           n_min, n_max, vocab, addr(slots), capacity))


def tfe_index_probe_host(slots, capacity, tokens, n):
    row, nb, home = ctypes.c_int32(), ctypes.c_int32(), ctypes.c_int64()
    _check(lib.tfe_index_probe_host(addr(slots), capacity, addr(tokens), n, ctypes.byref(row),
                                    ctypes.byref(nb), ctypes.byref(home)))
    return row.value, nb.value, home.value


def make_desc(phrase_tokens, phrase_len, n_min, n_max, vocab, values, dim, dtype,
              values_on_device, max_load_factor=0.5, hbm_cache_rows=0, adopt_host_values=0,
              prefill_rows=0, miss_fill=0, pinned_rows=0, pageable_values=None):
    """Fills a tfe_table_desc; the caller keeps the arrays alive until
    tfe_table_load returns (and `values` for the table's life if adopted)."""
    d = tfe_table_desc()
    d.n_phrases = int(phrase_len.shape[0])
    d.n_min, d.n_max, d.vocab = n_min, n_max, vocab
    d.phrase_tokens = addr(phrase_tokens)
    d.phrase_len = addr(phrase_len)
    d.values = addr(values)
    d.dim, d.dtype, d.values_on_device = dim, dtype, int(values_on_device)
    d.max_load_factor = max_load_factor
    d.hbm_cache_rows = hbm_cache_rows
    d.adopt_host_values = adopt_host_values
    d.prefill_rows = prefill_rows
    d.miss_fill = miss_fill
    d.pinned_rows = pinned_rows
    d.pageable_values = addr(pageable_values)
    return d
