"""Host-side logic of libtfe (no GPU): the exported symbols, the exact-match
phrase index built on the host (self-lookup, absent keys, duplicates, errors)
and the spread of its hash, pinned to the occupancy formula of Eq. 7."""
import ctypes
import math
import os
import re

import numpy as np
import pytest

import synth
from paper_2607_07388_amd import tfe

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_library_exports_every_declared_symbol():
    hdr = open(os.path.join(ROOT, "include", "tfe.h")).read()
    declared = set(re.findall(r"^\S.*?\b(tfe_[a-z_]+)\s*\(", hdr, re.M))
    assert declared == set(tfe.EXPORTED)
    for name in declared:
        assert hasattr(tfe.lib, name)
    so = ctypes.CDLL(os.path.join(ROOT, "paper_2607_07388_amd", "libtfe.so"))
    for name in declared:
        getattr(so, name)


def build(tokens, lens, n_min, n_max, vocab=synth.V, lf=0.5):
    cap = tfe.tfe_index_capacity(lens.size, lf)
    slots = np.zeros(cap * 16, np.uint8)
    tfe.tfe_index_build_host(tokens, lens, lens.size, n_min, n_max, vocab, slots, cap)
    return slots, cap


def test_capacity_rule():
    assert tfe.tfe_index_capacity(0, 0.5) == 8
    assert tfe.tfe_index_capacity(4096, 0.5) == 8192
    assert tfe.tfe_index_capacity(1 << 20, 0.5) == 1 << 21
    assert tfe.tfe_index_capacity(1 << 20, 0.0) == 1 << 21
    assert tfe.tfe_index_capacity(3000, 0.5) == 8192
    assert tfe.tfe_index_capacity(10, 0.95) == -1


def test_self_lookup_and_absent_keys_workload1():
    table, _ = synth.config1()
    slots, cap = build(table.tokens, table.lens, 2, 3)
    for i in range(table.n_phrases):
        row, nb, _ = tfe.tfe_index_probe_host(slots, cap, table.tokens[i], int(table.lens[i]))
        assert row == i and nb >= 1
    stored = {tuple(r[:l]) for r, l in zip(table.tokens.tolist(), table.lens.tolist())}
    rng = np.random.default_rng(0)
    for _ in range(500):
        n = int(rng.integers(2, 4))
        w = rng.integers(0, synth.V, n).astype(np.int32)
        row, _, _ = tfe.tfe_index_probe_host(slots, cap, w, n)
        assert row == (-1 if tuple(w.tolist()) not in stored else row)
    # A 2-gram that is the suffix of a stored 3-gram is a different key.
    i3 = int(np.flatnonzero(table.lens == 3)[0])
    suffix = table.tokens[i3, 1:3].copy()
    row, _, _ = tfe.tfe_index_probe_host(slots, cap, suffix, 2)
    assert row == -1 or tuple(suffix.tolist()) in stored


def test_four_gram_keys_use_the_extension_word():
    # Phrases that agree on their newest three tokens and differ in the oldest.
    toks = np.array([[1, 7, 8, 9], [2, 7, 8, 9], [7, 8, 9, -1], [0, 7, 8, 9]], np.int32)
    lens = np.array([4, 4, 3, 4], np.uint8)
    slots, cap = build(toks, lens, 2, 4)
    for i in range(4):
        row, _, _ = tfe.tfe_index_probe_host(slots, cap, toks[i], int(lens[i]))
        assert row == i
    row, _, _ = tfe.tfe_index_probe_host(slots, cap, np.array([3, 7, 8, 9], np.int32), 4)
    assert row == -1


def test_boundary_token_ids_round_trip():
    V = synth.V
    toks = np.array([[0, 0, -1, -1], [V - 1, V - 1, -1, -1], [0, V - 1, 0, -1],
                     [V - 1, 0, V - 1, 0], [0, 0, 0, 0]], np.int32)
    lens = np.array([2, 2, 3, 4, 4], np.uint8)
    slots, cap = build(toks, lens, 2, 4)
    for i in range(5):
        assert tfe.tfe_index_probe_host(slots, cap, toks[i], int(lens[i]))[0] == i
    assert tfe.tfe_index_probe_host(slots, cap, np.array([0, 0, 0], np.int32), 3)[0] == -1


@pytest.mark.parametrize("toks,lens,n_min,n_max,status", [
    ([[1, 2, -1], [1, 2, -1]], [2, 2], 2, 3, tfe.TFE_ERR_DUPLICATE_KEY),
    ([[1, 2, 3], [4, 5, -1], [1, 2, 3]], [3, 2, 3], 2, 3, tfe.TFE_ERR_DUPLICATE_KEY),
    ([[1, 2, -1]], [1], 2, 3, tfe.TFE_ERR_INVALID_ARG),
    ([[1, 2, 3]], [4], 2, 3, tfe.TFE_ERR_INVALID_ARG),
    ([[1, synth.V, -1]], [2], 2, 3, tfe.TFE_ERR_INVALID_ARG),
    ([[1, -3, -1]], [2], 2, 3, tfe.TFE_ERR_INVALID_ARG),
    ([[1, 2, -1]], [2], 1, 3, tfe.TFE_ERR_INVALID_ARG),
    ([[1, 2, -1]], [2], 3, 2, tfe.TFE_ERR_INVALID_ARG),
])
def test_build_errors(toks, lens, n_min, n_max, status):
    toks = np.array(toks, np.int32)
    lens = np.array(lens, np.uint8)
    with pytest.raises(tfe.TfeError) as e:
        build(toks, lens, n_min, n_max)
    assert e.value.status == status
    assert tfe.tfe_last_error()


def test_too_small_capacity_is_rejected():
    toks = np.arange(40, dtype=np.int32).reshape(20, 2)
    lens = np.full(20, 2, np.uint8)
    slots = np.zeros(16 * 16, np.uint8)
    with pytest.raises(tfe.TfeError):
        tfe.tfe_index_build_host(toks, lens, 20, 2, 2, synth.V, slots, 16)


def test_home_bucket_occupancy_follows_eq7():
    """Eq. 7: M keys thrown into B slots occupy B(1 - (1 - 1/B)^M) of them on
    average.  The index's home buckets for the Zipf-built 2^20-phrase table
    must agree within 5 standard deviations of the occupancy law."""
    table = synth.config2_table()
    P = table.n_phrases
    cap = tfe.tfe_index_capacity(P, 0.5)
    slots = np.zeros(cap * 16, np.uint8)
    tfe.tfe_index_build_host(table.tokens, table.lens, P, 2, 3, synth.V, slots, cap)
    nb = cap // 8
    sample = np.arange(0, P, 1)
    homes = np.empty(sample.size, np.int64)
    reads = np.empty(sample.size, np.int32)
    for k, i in enumerate(sample[:200000]):
        row, nr, home = tfe.tfe_index_probe_host(slots, cap, table.tokens[i], int(table.lens[i]))
        assert row == i
        homes[k], reads[k] = home, nr
    M = 200000
    occupied = np.unique(homes[:M]).size
    q1 = (1 - 1 / nb) ** M
    mean = nb * (1 - q1)
    var = nb * (nb - 1) * (1 - 2 / nb) ** M + nb * q1 - nb * nb * q1 * q1
    assert abs(occupied - mean) < 5 * math.sqrt(var), (occupied, mean, math.sqrt(var))
    # Load factor 1/2 with 8-slot buckets: nearly every hit reads one bucket.
    assert reads[:M].mean() < 1.05


def test_empty_table_index():
    slots, cap = build(np.zeros((0, 3), np.int32), np.zeros(0, np.uint8), 2, 3)
    assert cap == 8
    assert tfe.tfe_index_probe_host(slots, cap, np.array([1, 2], np.int32), 2)[0] == -1


def test_parallel_build_finds_a_planted_duplicate():
    """The multi-threaded build reports a repeated phrase wherever it lands."""
    table = synth.config2_table()
    for src, dst in ((5, table.n_phrases - 1), (777777, 3)):
        toks = table.tokens.copy()
        lens = table.lens.copy()
        toks[dst], lens[dst] = toks[src], lens[src]
        with pytest.raises(tfe.TfeError) as e:
            build(toks, lens, 2, 3)
        assert e.value.status == tfe.TFE_ERR_DUPLICATE_KEY
        assert str(min(src, dst)) in tfe.tfe_last_error()


def test_one_hip_runtime_whatever_the_import_order():
    """torch carries its own HIP runtime under the system runtime's soname.
    Loading libtfe (or the workload generator's device library) before
    torch must not map a second runtime: with two, one of them sees no
    device.  Checked in a fresh process, libraries first, torch last."""
    import subprocess
    import sys
    code = ("import sys; sys.path.insert(0, %r)\n"
            "from paper_2607_07388_amd import tfe\n"
            "import synth; synth.dev_lib()\n"
            "import torch\n"
            "print(len(tfe.hip_runtimes()))\n" % ROOT)
    r = subprocess.run([sys.executable, "-c", code], stdout=subprocess.PIPE,
                       stderr=subprocess.PIPE, text=True, timeout=300)
    assert r.returncode == 0 and r.stdout.strip() == "1", r.stdout + r.stderr
