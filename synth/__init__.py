"""Seeded synthetic workloads for the phrase-memory lookup+inject path.

This module is the only code that the oracle side and the GPU side of the
tests share.  It draws inputs (token streams, phrase tables, hidden states,
value rows) and holds none of the method's arithmetic.

Recipes (token ids stand in for a tokenizer's output; the phrase tables stand
in for the corpus-mined tables of the paper's construction pipeline, whose
corpora, tokenizer and encoder are not available):

* tokens: truncated Zipf(s) over V = 151936 ids (the vocabulary of the paper's
  backbone), p(rank) ~ rank^-s, id = rank - 1, sampled with Vose's alias
  method from a counter-based SplitMix64 stream (``csrc/synth_rng.h``);
* phrase tables: the most frequent distinct n-grams of a seeded Zipf stream,
  phrase ids ordered by count (most frequent first);
* hidden states and value rows: Irwin-Hall(12) normal draws scaled by sigma,
  a pure function of (seed, stream tag, row, column) so that multi-GiB tables
  are drawn on the device and any single row can be re-drawn on the host with
  identical bits.
"""
import ctypes
import dataclasses
import os

import numpy as np

from . import _build

V = 151936
D = 1024

# Stream tags: each random quantity of a workload has its own tag.
TAG_STREAM = 1      # table-building token stream
TAG_QUERY = 2       # query token ids (set k uses TAG_QUERY + 16 k)
TAG_HIDDEN = 3      # hidden states (set k uses TAG_HIDDEN + 16 k)
TAG_VALUES = 4      # value table
TAG_CAND = 5        # prefetch candidates

F32, BF16 = 0, 1

_host = None
_dev = None


def _load(path):
    if not os.path.exists(path):
        _build.build()
    return ctypes.CDLL(path)


def host_lib():
    global _host
    if _host is None:
        lib = _load(_build.HOST_SO)
        i64, u64, vp = ctypes.c_int64, ctypes.c_uint64, ctypes.c_void_p
        lib.synth_zipf_alias.argtypes = [ctypes.c_int, ctypes.c_double, vp, vp]
        lib.synth_zipf_tokens.argtypes = [u64, i64, i64, vp, vp, ctypes.c_int, vp]
        lib.synth_zipf_tokens.restype = None
        lib.synth_ngram_top.argtypes = [vp, i64, ctypes.c_int, ctypes.c_int, i64, i64, vp, vp]
        lib.synth_ngram_top.restype = i64
        lib.synth_normal_rows.argtypes = [u64, vp, i64, i64, ctypes.c_float, ctypes.c_int, vp]
        lib.synth_normal_rows.restype = None
        lib.synth_normal_range.argtypes = [u64, i64, i64, i64, ctypes.c_float, ctypes.c_int, vp]
        lib.synth_normal_range.restype = None
        lib.synth_stream_key.argtypes = [u64, u64]
        lib.synth_stream_key.restype = u64
        _host = lib
    return _host


def dev_lib():
    global _dev
    if _dev is None:
        # One HIP runtime per process: torch's, when it is installed (its
        # copy has the system runtime's soname and satisfies this library's
        # dependency only if it is loaded first).
        try:
            import torch  # noqa: F401
        except ImportError:
            pass
        lib = _load(_build.DEV_SO)
        i64, u64, vp = ctypes.c_int64, ctypes.c_uint64, ctypes.c_void_p
        lib.synth_normal_fill_dev.argtypes = [vp, i64, i64, i64, u64, ctypes.c_float,
                                              ctypes.c_int, vp]
        lib.synth_normal_fill_dev.restype = ctypes.c_int
        lib.synth_copy_dev.argtypes = [vp, vp, i64, ctypes.c_int, vp]
        lib.synth_copy_dev.restype = ctypes.c_int
        lib.synth_host_device_ptr.argtypes = [vp, ctypes.POINTER(vp)]
        lib.synth_host_device_ptr.restype = ctypes.c_int
        lib.synth_spin_dev.argtypes = [ctypes.c_double, vp]
        lib.synth_spin_dev.restype = ctypes.c_int
        _dev = lib
    return _dev


def _ptr(a):
    return ctypes.c_void_p(a.ctypes.data)


def stream_key(seed, tag):
    return int(host_lib().synth_stream_key(seed, tag))


def scale_of(sigma):
    """The float32 multiplier applied to an Irwin-Hall integer draw."""
    return float(np.float32(sigma / 65536.0))


_alias_cache = {}


def zipf_alias(s, vocab=V):
    k = (float(s), int(vocab))
    if k not in _alias_cache:
        prob = np.empty(vocab, np.float64)
        alias = np.empty(vocab, np.int32)
        if host_lib().synth_zipf_alias(vocab, float(s), _ptr(prob), _ptr(alias)) != 0:
            raise ValueError("bad Zipf parameters")
        _alias_cache[k] = (prob, alias)
    return _alias_cache[k]


def zipf_tokens(seed, tag, n, s, vocab=V, start=0):
    """n i.i.d. truncated-Zipf(s) token ids (int32) of stream (seed, tag)."""
    prob, alias = zipf_alias(s, vocab)
    out = np.empty(int(n), np.int32)
    host_lib().synth_zipf_tokens(stream_key(seed, tag), int(start), int(n), _ptr(prob),
                                 _ptr(alias), vocab, _ptr(out))
    return out


def ngram_top(stream, n, want, skip=0, vocab=V):
    """Ranks [skip, skip+want) of the distinct n-grams of `stream` by count
    (descending; ties by tuple ascending).  Returns (tuples [m x n], counts)."""
    stream = np.ascontiguousarray(stream, np.int32)
    tup = np.empty((int(want), n), np.int32)
    cnt = np.empty(int(want), np.int64)
    got = host_lib().synth_ngram_top(_ptr(stream), stream.size, n, vocab, int(skip),
                                     int(want), _ptr(tup), _ptr(cnt))
    if got < 0:
        raise ValueError("bad n-gram request")
    return tup[:got], cnt[:got]


def normal_rows(seed, tag, rows, cols, sigma, dtype):
    """Host draw of the given rows of a (seed, tag) normal table.  dtype F32
    gives float32, BF16 gives the bfloat16 bit patterns as uint16."""
    rows = np.ascontiguousarray(rows, np.int64)
    out = np.empty((rows.size, cols), np.float32 if dtype == F32 else np.uint16)
    host_lib().synth_normal_rows(stream_key(seed, tag), _ptr(rows), rows.size, cols,
                                 scale_of(sigma), dtype, _ptr(out))
    return out


def normal_range(seed, tag, row0, nrows, cols, sigma, dtype):
    out = np.empty((int(nrows), cols), np.float32 if dtype == F32 else np.uint16)
    host_lib().synth_normal_range(stream_key(seed, tag), int(row0), int(nrows), cols,
                                  scale_of(sigma), dtype, _ptr(out))
    return out


def normal_fill_device(ptr, row0, nrows, cols, seed, tag, sigma, dtype, stream=0):
    """Device draw of rows [row0, row0+nrows) into the device buffer `ptr`
    (an integer address), on HIP stream `stream` (an integer handle)."""
    rc = dev_lib().synth_normal_fill_dev(ctypes.c_void_p(ptr), int(row0), int(nrows), cols,
                                         stream_key(seed, tag), scale_of(sigma), dtype,
                                         ctypes.c_void_p(stream))
    if rc != 0:
        raise RuntimeError("synth_normal_fill_dev failed (%d)" % rc)


def copy_device(dst, src, nbytes, blocks=4096, stream=0):
    """Reference device copy of nbytes (multiple of 16) between device buffers."""
    rc = dev_lib().synth_copy_dev(ctypes.c_void_p(dst), ctypes.c_void_p(src), int(nbytes),
                                  int(blocks), ctypes.c_void_p(stream))
    if rc != 0:
        raise RuntimeError("synth_copy_dev failed (%d)" % rc)


def spin_device(us, stream=0):
    """Enqueue a device busy-wait of `us` microseconds (a compute stand-in)."""
    if dev_lib().synth_spin_dev(float(us), ctypes.c_void_p(stream)) != 0:
        raise RuntimeError("synth_spin_dev failed")


def host_device_ptr(host_ptr):
    """Device address of a pinned host buffer."""
    out = ctypes.c_void_p()
    if dev_lib().synth_host_device_ptr(ctypes.c_void_p(host_ptr), ctypes.byref(out)) != 0:
        raise RuntimeError("not pinned host memory")
    return out.value


def bf16_to_f32(u16):
    """bfloat16 bit patterns (uint16) -> float32 values."""
    return (np.asarray(u16, np.uint16).astype(np.uint32) << 16).view(np.float32)


@dataclasses.dataclass
class PhraseTable:
    """A phrase table: row i is the phrase tokens[i, :lens[i]] (oldest first,
    padded with -1 to n_max columns); its value row is the (seed, TAG_VALUES)
    normal table row i with standard deviation `sigma`."""
    tokens: np.ndarray
    lens: np.ndarray
    n_min: int
    n_max: int
    dtype: int
    seed: int
    sigma: float = 0.02
    dim: int = D
    vocab: int = V

    @property
    def n_phrases(self):
        return int(self.lens.size)

    def value_rows(self, rows):
        return normal_rows(self.seed, TAG_VALUES, rows, self.dim, self.sigma, self.dtype)

    def all_values(self):
        return normal_range(self.seed, TAG_VALUES, 0, self.n_phrases, self.dim, self.sigma,
                            self.dtype)


@dataclasses.dataclass
class QueryBatch:
    """Token ids [B x (ctx + S)] (the first ctx columns are history only) and
    the hidden states of the S injected positions of each row, drawn from the
    (seed, hidden_tag) normal table with standard deviation 1."""
    tokens: np.ndarray
    ctx: int
    S: int
    seed: int
    hidden_tag: int
    dtype: int
    dim: int = D

    @property
    def B(self):
        return int(self.tokens.shape[0])

    @property
    def T(self):
        return self.B * self.S

    def hidden(self):
        return normal_range(self.seed, self.hidden_tag, 0, self.T, self.dim, 1.0, self.dtype)

    def hidden_rows(self, rows):
        return normal_rows(self.seed, self.hidden_tag, rows, self.dim, 1.0, self.dtype)


def stack_tables(parts, n_max):
    """Concatenate [(tuples, counts), ...] of different n into one table,
    rows ordered by count descending, then n ascending, then tuple."""
    toks, lens, cnts = [], [], []
    for tup, cnt in parts:
        n = tup.shape[1]
        t = np.full((tup.shape[0], n_max), -1, np.int32)
        t[:, :n] = tup
        toks.append(t)
        lens.append(np.full(tup.shape[0], n, np.uint8))
        cnts.append(cnt)
    toks = np.concatenate(toks)
    lens = np.concatenate(lens)
    cnts = np.concatenate(cnts)
    keys = [toks[:, j] for j in range(n_max - 1, -1, -1)] + [lens, -cnts]
    order = np.lexsort(keys)
    return toks[order], lens[order], cnts[order]


from .workloads import *  # noqa: E402,F401,F403
