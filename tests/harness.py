"""Shared driving code for the GPU tests and the benchmark: loads synthetic
phrase tables into libtfe, runs lookup + inject through the C ABI binding and
computes the oracle's answer for the same seeded inputs.  The oracle is
imported only by the functions that compute its answer, so the benchmark's
timed GPU path never loads it."""
import numpy as np
import torch

import synth
from paper_2607_07388_amd import tfe

TORCH_DT = {synth.F32: torch.float32, synth.BF16: torch.bfloat16}


def cur_stream():
    return torch.cuda.current_stream().cuda_stream


def release_pinned():
    """Returns the pinned host blocks torch keeps cached after their tensors
    died, so that a large pinned allocation that follows finds the memory."""
    import gc
    gc.collect()
    empty = getattr(torch._C, "_host_emptyCache", None)
    if empty is not None:
        empty()


def release_device():
    """Returns the device memory torch's caching allocator keeps after its
    tensors died, and the library's idle construction scratch, so that a
    large device allocation by the library that follows finds the memory."""
    import gc
    gc.collect()
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    tfe.tfe_ngram_release()


def device_values(table):
    """The table's value rows drawn on the device (bit-identical to the host draw)."""
    v = torch.empty((table.n_phrases, table.dim), dtype=TORCH_DT[table.dtype], device="cuda")
    if table.n_phrases:
        synth.normal_fill_device(v.data_ptr(), 0, table.n_phrases, table.dim, table.seed,
                                 synth.TAG_VALUES, table.sigma, table.dtype, cur_stream())
    return v


def pageable_values(table, first, stream=None, chunk=1 << 19):
    """Value rows [first, P) of `table` (bf16) in ordinary pageable host
    memory, drawn on the device chunk by chunk and copied down."""
    stream = stream or torch.cuda.current_stream()
    P, D = table.n_phrases, table.dim
    host = np.empty((P - first, D), np.int16)
    ht = torch.from_numpy(host)
    dbuf = torch.empty((min(chunk, P - first), D), dtype=torch.bfloat16, device="cuda")
    for r0 in range(first, P, chunk):
        n = min(chunk, P - r0)
        synth.normal_fill_device(dbuf.data_ptr(), r0, n, D, table.seed, synth.TAG_VALUES,
                                 table.sigma, synth.BF16, stream.cuda_stream)
        ht[r0 - first:r0 - first + n].copy_(dbuf[:n].view(torch.int16))
    torch.cuda.synchronize()
    return host


def to_device(a, dtype):
    """Host array (float32, or uint16 bf16 patterns) -> device tensor."""
    if dtype == synth.BF16:
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).cuda().view(torch.bfloat16)
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def to_host(t, dtype):
    t = t.detach().cpu()
    if dtype == synth.BF16:
        return t.view(torch.int16).numpy().view(np.uint16)
    return t.numpy()


class GpuTable:
    """A phrase table loaded through tfe_table_load."""

    def __init__(self, table, values_on_device=None, lf=0.5):
        self.table = table
        self.handle = None
        if values_on_device is None:
            values_on_device = table.n_phrases * table.dim > (1 << 22)
        vals = device_values(table) if values_on_device else table.all_values()
        torch.cuda.synchronize()
        desc = tfe.make_desc(table.tokens, table.lens, table.n_min, table.n_max, table.vocab,
                             vals if table.n_phrases else None, table.dim, table.dtype,
                             values_on_device, lf)
        self.handle = tfe.tfe_table_load(desc, cur_stream())
        big = values_on_device and table.n_phrases * table.dim * 2 > (1 << 30)
        del vals
        if big:  # the library holds its own copy now
            release_device()

    def close(self):
        if self.handle:
            tfe.tfe_table_free(self.handle)
            self.handle = None

    def __del__(self):
        # At interpreter shutdown the binding may already be torn down.
        if tfe is not None and getattr(tfe, "lib", None) is not None:
            self.close()


class Outputs:
    def __init__(self, T, dim, dtype, with_len=True):
        self.hit = torch.full((T,), 0xEE, dtype=torch.uint8, device="cuda")
        self.slot = torch.full((T,), -7, dtype=torch.int32, device="cuda")
        self.len = torch.full((T,), 0xEE, dtype=torch.uint8, device="cuda") if with_len else None
        self.out = torch.empty((T, dim), dtype=TORCH_DT[dtype], device="cuda")


def run(gt, tokens_d, B, ctx, S, hidden_d, outs, gate=tfe.TFE_GATE_SIGMOID, scale=1.0,
        inplace=False, stream=None):
    hout = hidden_d if inplace else outs.out
    tfe.tfe_lookup_inject(gt.handle, tokens_d, B, ctx, S, hidden_d, hout, outs.hit, outs.slot,
                          outs.len, gate, scale, stream if stream is not None else cur_stream())
    return hout


def oracle_answer(table, otable, tokens, ctx, S, hidden, gate=0, scale=1.0,
                  positions=None, row_map=None):
    """Oracle lookup + inject.  Value rows are drawn on the host for the
    matched rows only.  `positions` restricts the injection to a sample.
    `row_map` maps the oracle table's rows to the full table's rows when the
    oracle holds only the phrases that can match (see subset_rows)."""
    import oracle
    hit, row, ln = otable.lookup(tokens, ctx, S)
    if row_map is not None:
        row = np.where(row >= 0, row_map[np.maximum(row, 0)], -1).astype(np.int32)
    if positions is None:
        positions = np.arange(hit.size)
    sel = row[positions].astype(np.int64)
    uniq, inv = np.unique(sel[sel >= 0], return_inverse=True)
    vals = table.value_rows(uniq) if uniq.size else np.zeros((0, table.dim), np.float32)
    idx = np.full(sel.size, -1, np.int64)
    idx[sel >= 0] = inv
    out = oracle.inject(hidden[positions], vals, idx, table.dtype, gate, scale)
    return hit, row, ln, out


def assert_close(got, want, dtype):
    """fp32: max abs error 1e-5.  bf16: |a - b| <= 2e-2 max(|b|, 1e-3)."""
    if dtype == synth.F32:
        err = np.abs(got.astype(np.float64) - want.astype(np.float64))
        assert err.max() <= 1e-5, err.max()
    else:
        a = synth.bf16_to_f32(got).astype(np.float64)
        b = synth.bf16_to_f32(want).astype(np.float64)
        bound = 2e-2 * np.maximum(np.abs(b), 1e-3)
        bad = np.abs(a - b) > bound
        assert not bad.any(), (int(bad.sum()), a[bad][:5], b[bad][:5])


def oracle_table(table):
    import oracle
    return oracle.Table(table.tokens, table.lens, table.n_min, table.n_max, table.vocab)


def subset_rows(table, tokens, ctx, S):
    """Rows of `table` whose phrase equals some n-gram window of the query
    (n_min..n_max, exact tuple comparison by packed integer keys, n <= 3).
    An oracle built from these rows answers the query exactly as one built
    from the whole table, since no other phrase can match."""
    assert table.n_max <= 3
    V = np.uint64(table.vocab)
    want = []
    for n in range(table.n_min, table.n_max + 1):
        cols = [tokens[:, j:tokens.shape[1] - n + 1 + j].astype(np.int64) for j in range(n)]
        w = np.stack(cols, axis=-1).reshape(-1, n)
        w = w[np.all((w >= 0) & (w < table.vocab), axis=1)]
        k = np.zeros(w.shape[0], np.uint64)
        for j in range(n):
            k = k * V + w[:, j].astype(np.uint64)
        want.append((n, np.unique(k)))
    rows = []
    for n, k in want:
        idx = np.flatnonzero(table.lens == n)
        t = table.tokens[idx, :n].astype(np.uint64)
        pk = np.zeros(idx.size, np.uint64)
        for j in range(n):
            pk = pk * V + t[:, j]
        pos = np.minimum(np.searchsorted(k, pk), k.size - 1) if k.size else None
        rows.append(idx[k[pos] == pk] if k.size else idx[:0])
    return np.sort(np.concatenate(rows)).astype(np.int64)
