"""Allocation failures that the host can force without a GPU.

TFE_FAIL_ALLOC=k makes the k-th allocation of a library call fail.  The
first two allocations of tfe_table_load are on the host (the index, then the
table object), before any HIP call, so they can be checked here; the device
and pinned allocations after them are covered by the GPU tests.  A source
check keeps every device and pinned allocation behind the library's wrappers,
which are the only places the hook and the held-memory count live."""
import os
import re

import numpy as np
import pytest

import synth
from paper_2607_07388_amd import tfe

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2607_07388_amd", "csrc")


@pytest.fixture
def fail_at(monkeypatch):
    def set_k(k):
        monkeypatch.setenv("TFE_FAIL_ALLOC", str(k))
    yield set_k
    monkeypatch.delenv("TFE_FAIL_ALLOC", raising=False)


def _desc(table, vals, **kw):
    return tfe.make_desc(table.tokens, table.lens, table.n_min, table.n_max, table.vocab, vals,
                         table.dim, synth.F32, 0, **kw)


@pytest.mark.parametrize("cache_rows", [0, 1024])
def test_host_allocations_of_a_load_fail_cleanly(fail_at, cache_rows):
    table, _ = synth.config1()
    vals = np.zeros((table.n_phrases, table.dim), np.float32)
    before = tfe.tfe_memory_held()
    for k, what in ((1, "host index of"), (2, "table object")):
        fail_at(k)
        with pytest.raises(tfe.TfeError) as e:
            tfe.tfe_table_load(_desc(table, vals, hbm_cache_rows=cache_rows))
        assert e.value.status == tfe.TFE_ERR_OOM and what in str(e.value)
        assert tfe.tfe_memory_held() == before


def test_argument_errors_come_before_allocations(fail_at):
    """A bad descriptor is reported as such even when the first allocation
    would fail: validation allocates nothing."""
    table, _ = synth.config1()
    vals = np.zeros((table.n_phrases, table.dim), np.float32)
    fail_at(1)
    bad = _desc(table, vals, max_load_factor=0.95)
    with pytest.raises(tfe.TfeError) as e:
        tfe.tfe_table_load(bad)
    assert e.value.status == tfe.TFE_ERR_INVALID_ARG


def test_memory_held_starts_empty_and_rejects_no_output():
    assert tfe.tfe_memory_held() == (0, 0)
    assert tfe.lib.tfe_memory_held(None, None) == tfe.TFE_ERR_INVALID_ARG


def _code(path):
    """Source without comments."""
    s = open(path).read()
    s = re.sub(r"/\*.*?\*/", "", s, flags=re.S)
    return re.sub(r"//[^\n]*", "", s)


def test_every_device_and_pinned_allocation_goes_through_the_wrappers():
    raw = re.compile(r"\b(hipMalloc\w*|hipFree|hipHostMalloc|hipHostFree|hipExtMalloc\w*|"
                     r"hipMallocManaged|hipMallocAsync|hipFreeAsync)\s*\(")
    found = {}
    for f in sorted(os.listdir(CSRC)):
        if not f.endswith((".cpp", ".hip", ".h")):
            continue
        hits = raw.findall(_code(os.path.join(CSRC, f)))
        if hits:
            found[f] = hits
    # The four wrappers themselves: one hipMalloc, hipFree, hipHostMalloc and
    # hipHostFree each, all in tfe_api.cpp.
    assert found == {"tfe_api.cpp": ["hipMalloc", "hipFree", "hipHostMalloc", "hipHostFree"]}
    # Host objects that a load or head creation allocates ask the hook first.
    api = _code(os.path.join(CSRC, "tfe_api.cpp"))
    head = _code(os.path.join(CSRC, "tfe_head_api.cpp"))
    assert "alloc_fails() ? nullptr : new (std::nothrow) tfe_table" in api
    assert "alloc_fails() ? nullptr : new (std::nothrow) tfe_head" in head
    assert "if (alloc_fails()) throw std::bad_alloc();" in api
