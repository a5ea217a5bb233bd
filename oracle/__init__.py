"""CPU oracle of the phrase-memory lookup + gated residual injection.

TEST INFRASTRUCTURE ONLY: the tests, the smoke check and the benchmark's
CPU-baseline leg may import this package; the product path never does.  The
arithmetic lives in ``oracle.cpp`` (std::map on token tuples, scalar double
loops); this file only marshals numpy arrays.  ``head.cpp`` is the
early-exit prefetch head, ``ngram.cpp`` the frequency-ranked phrase-table
construction; ``lru.py`` is the reference model of the HBM cache
tier's replacement policy.
"""
import ctypes
import os

import numpy as np

from . import _build

OK, INVALID, DUPLICATE = 0, -1, -2
GATE_SIGMOID, GATE_CONST = 0, 1
WEIGHT_LENGTH, WEIGHT_UNIFORM = 0, 1
EPS = 1e-6

_lib = None


def lib():
    global _lib
    if _lib is None:
        # ORACLE_SO names another build of the same sources (the sanitizer
        # tests load an instrumented one).
        so = os.environ.get("ORACLE_SO") or _build.SO
        if not os.path.exists(so):
            _build.build()
        L = ctypes.CDLL(so)
        vp, i64 = ctypes.c_void_p, ctypes.c_int64
        L.oracle_table_new.argtypes = [vp, vp, i64, ctypes.c_int, ctypes.c_int, ctypes.c_int,
                                       ctypes.POINTER(ctypes.c_int)]
        L.oracle_table_new.restype = vp
        L.oracle_table_free.argtypes = [vp]
        L.oracle_table_free.restype = None
        L.oracle_lookup.argtypes = [vp, vp, i64, i64, i64, vp, vp, vp]
        L.oracle_lookup_all.argtypes = [vp, vp, i64, i64, i64, vp, vp]
        L.oracle_inject_multi.argtypes = [vp, vp, i64, vp, i64, ctypes.c_int, ctypes.c_int, i64,
                                          ctypes.c_int, ctypes.c_int, ctypes.c_int,
                                          ctypes.c_double, vp]
        L.oracle_inject.argtypes = [vp, vp, i64, vp, i64, i64, ctypes.c_int, ctypes.c_int,
                                    ctypes.c_double, vp]
        L.oracle_gate.argtypes = [vp, vp, i64, ctypes.c_int, ctypes.c_int, ctypes.c_double]
        L.oracle_gate.restype = ctypes.c_double
        L.oracle_head_topk.argtypes = [vp, vp, i64, i64, i64, i64, ctypes.c_int, vp, vp, vp]
        L.oracle_ngram_top.argtypes = [vp, i64, ctypes.c_int, ctypes.c_int, i64, i64, vp, vp]
        L.oracle_ngram_top.restype = i64
        L.oracle_round_bf16.argtypes = [ctypes.c_double]
        L.oracle_round_bf16.restype = ctypes.c_uint16
        _lib = L
    return _lib


def _p(a):
    return ctypes.c_void_p(a.ctypes.data)


class OracleError(Exception):
    def __init__(self, status):
        super().__init__("oracle status %d" % status)
        self.status = status


class Table:
    """phrase tuple -> row map.  tokens: int32 [P x n_max] (oldest first,
    padded), lens: uint8 [P]."""

    def __init__(self, tokens, lens, n_min, n_max, vocab):
        self.n_min, self.n_max = n_min, n_max
        self.tokens = np.ascontiguousarray(tokens, np.int32).reshape(-1, n_max)
        self.lens = np.ascontiguousarray(lens, np.uint8)
        st = ctypes.c_int(0)
        self._h = lib().oracle_table_new(_p(self.tokens), _p(self.lens), self.lens.size, n_min,
                                         n_max, vocab, ctypes.byref(st))
        if not self._h:
            raise OracleError(st.value)

    def __del__(self):
        h = getattr(self, "_h", None)
        if h and _lib is not None:
            _lib.oracle_table_free(h)
        self._h = None

    def lookup(self, tokens, ctx, S):
        """tokens: int32 [B x (ctx+S)] -> (hit uint8, row int32, len uint8), each [B*S]."""
        tokens = np.ascontiguousarray(tokens, np.int32)
        B = tokens.shape[0]
        assert tokens.shape[1] == ctx + S
        hit = np.empty(B * S, np.uint8)
        row = np.empty(B * S, np.int32)
        ln = np.empty(B * S, np.uint8)
        st = lib().oracle_lookup(self._h, _p(tokens), B, ctx, S, _p(hit), _p(row), _p(ln))
        if st != OK:
            raise OracleError(st)
        return hit, row, ln


    def lookup_all(self, tokens, ctx, S):
        """All matched lengths: -> (mask uint8 [B*S], rows int32 [B*S x L]);
        column j is the phrase of length n_min + j (-1 if none), bit j of the
        mask is set where it matched."""
        tokens = np.ascontiguousarray(tokens, np.int32)
        B = tokens.shape[0]
        assert tokens.shape[1] == ctx + S
        L = self.n_max - self.n_min + 1
        mask = np.empty(B * S, np.uint8)
        rows = np.empty((B * S, L), np.int32)
        st = lib().oracle_lookup_all(self._h, _p(tokens), B, ctx, S, _p(mask), _p(rows))
        if st != OK:
            raise OracleError(st)
        return mask, rows


def inject(hidden, values, index, dtype, gate=GATE_SIGMOID, lam=1.0):
    """hidden [T x D] (float32, or uint16 bf16 patterns), values [R x D] of the
    same type, index int64 [T] (row of `values` or -1) -> out like hidden."""
    hidden = np.ascontiguousarray(hidden)
    values = np.ascontiguousarray(values)
    index = np.ascontiguousarray(index, np.int64)
    T, D = hidden.shape
    out = np.empty_like(hidden)
    R = values.shape[0] if values.ndim == 2 else 0
    st = lib().oracle_inject(_p(hidden), _p(values) if R else None, R, _p(index), T, D, dtype,
                             gate, float(lam), _p(out))
    if st != OK:
        raise OracleError(st)
    return out


def inject_multi(hidden, values, index, n_min, dtype, weighting=WEIGHT_LENGTH,
                 gate=GATE_SIGMOID, lam=1.0):
    """hidden [T x D], values [R x D] of the same type, index int64 [T x L]
    (row of `values` retained for length n_min + j, or -1) -> out like hidden:
    h + g * sum_j alpha_j v_j (Eq. 4, Eq. 11, Eq. 5)."""
    hidden = np.ascontiguousarray(hidden)
    values = np.ascontiguousarray(values)
    index = np.ascontiguousarray(index, np.int64)
    T, D = hidden.shape
    assert index.ndim == 2 and index.shape[0] == T
    out = np.empty_like(hidden)
    R = values.shape[0] if values.ndim == 2 else 0
    st = lib().oracle_inject_multi(_p(hidden), _p(values) if R else None, R, _p(index), T,
                                   index.shape[1], n_min, D, dtype, weighting, gate, float(lam),
                                   _p(out))
    if st != OK:
        raise OracleError(st)
    return out


def gate_value(h, m, dtype, gate=GATE_SIGMOID, lam=1.0):
    h = np.ascontiguousarray(h)
    m = np.ascontiguousarray(m)
    return float(lib().oracle_gate(_p(h), _p(m), h.size, dtype, gate, float(lam)))


def head_topk(w, h, K, dtype, with_logits=False):
    """Early-exit head (Eq. 13, Eq. 14): w [V x D], h [B x D] (float32, or
    uint16 bf16 patterns) -> ids int32 [B x K], probs float64 [B x K] (and
    the float64 logits [B x V] when asked)."""
    w = np.ascontiguousarray(w)
    h = np.ascontiguousarray(h)
    V, D = w.shape
    B = h.shape[0]
    assert h.shape[1] == D
    ids = np.empty((B, K), np.int32)
    probs = np.empty((B, K), np.float64)
    logits = np.empty((B, V), np.float64) if with_logits else None
    st = lib().oracle_head_topk(_p(w), _p(h), V, D, B, K, dtype, _p(ids), _p(probs),
                                _p(logits) if with_logits else None)
    if st != OK:
        raise OracleError(st)
    return (ids, probs, logits) if with_logits else (ids, probs)


def ngram_top(tokens, vocab, n, skip, top):
    """Offline table construction by frequency: the distinct n-grams of the
    stream ranked by count (ties: tuple ascending); ranks [skip, skip + top)
    -> (tuples int32 [m x n], counts int64 [m])."""
    tokens = np.ascontiguousarray(tokens, np.int32)
    tup = np.empty((max(top, 0), n), np.int32)
    cnt = np.empty(max(top, 0), np.int64)
    m = lib().oracle_ngram_top(_p(tokens), tokens.size, vocab, n, skip, top, _p(tup), _p(cnt))
    if m < 0:
        raise OracleError(int(m))
    return tup[:m], cnt[:m]


def round_bf16(x):
    return int(lib().oracle_round_bf16(float(x)))


def lookup_inject(table, batch_tokens, ctx, S, hidden, values, dtype, gate=GATE_SIGMOID,
                  lam=1.0):
    """Whole path for small inputs where the full value matrix is at hand."""
    hit, row, ln = table.lookup(batch_tokens, ctx, S)
    out = inject(hidden, values, row.astype(np.int64), dtype, gate, lam)
    return hit, row, ln, out
