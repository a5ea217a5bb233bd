"""Host-side logic of bench.py (no GPU): the one-GPU refusal, the
algorithmic-bytes formulas and the key counts they use."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       stdout=subprocess.PIPE, stderr=subprocess.PIPE, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr and r.stdout == ""


def test_algorithmic_bytes_per_decode_token():
    """bf16, D = 1024, out of place: hidden in + out (4096), the value row
    and row id per hit (2052 h), 8 per key, 4 per window token, 6 outputs."""
    T, hits = 16384, 10666
    b = bench.algorithmic_bytes(T, hits, 2 * T, 3)
    assert b == T * 4096 + hits * 2052 + 2 * T * 8 + T * 3 * 4 + T * 6
    # The stacked decode launch at hit rate 0.651: 5465.6 bytes per token.
    assert bench.algorithmic_bytes(1, 0.651, 2, 3) == pytest.approx(5465.9, abs=0.5)


def test_keys_formed_counts_short_prefixes():
    # Decode windows: every position forms n_max - n_min + 1 keys.
    assert bench.keys_formed(64, 2, 1, 2, 3) == 64 * 2
    # Prefill from column 0: position s forms the lengths n <= s + 1.
    assert bench.keys_formed(8, 0, 4096, 2, 4) == 8 * (0 + 1 + 2 + 3 * 4093)
    assert bench.keys_formed(1, 0, 1, 2, 4) == 0


def test_build_bytes_per_window():
    # 36-bit 2-gram keys: four 9-bit passes; 37 bits (vocab 2^18): five.
    assert bench.build_bytes_per_window(2, 151936) == 16 + 3 * 24 + 16
    assert bench.build_bytes_per_window(2, 1 << 18) == 16 + 4 * 24 + 16
    assert bench.build_bytes_per_window(4, 151936) == 20 + 5 * 32 + 2 * 28 + 24
    assert bench.build_bytes_per_window(4, 1 << 18) == 20 + 5 * 32 + 3 * 28 + 24
    assert bench.build_bytes_per_window(3, 151936) > bench.build_bytes_per_window(2, 151936)


def test_host_cpu_fields():
    h = bench.host_cpu()
    assert set(h) == {"host_cpu", "host_threads"} and h["host_threads"] >= 1


def test_hit_counts_come_from_sets_that_ran():
    """With fewer warmup calls than rotating sets, the sets the warmup never
    reached still hold the output buffers' sentinel fill; every count must
    come from a set's own call (the driver's --warmup 5 with 8 sets)."""
    n_sets, warmup, rows = 8, 5, 64
    sentinel = 0xEE
    hit = [[sentinel] * rows for _ in range(n_sets)]
    truth = [(7 * k + 3) % rows for k in range(n_sets)]   # hits each set's call writes
    calls = []

    def run(k):
        k %= n_sets
        calls.append(k)
        hit[k] = [1] * truth[k] + [0] * (rows - truth[k])

    for k in range(warmup):
        run(k)
    synced = []
    counts = bench.counts_after_run(n_sets, run, lambda: synced.append(len(calls)),
                                    lambda k: sum(hit[k]))
    assert counts == truth
    assert sorted(set(calls)) == list(range(n_sets))
    assert synced == [warmup + n_sets]          # one sync, after every set ran
    assert all(0 <= c <= rows for c in counts)


def test_check_line_rejects_impossible_rates():
    good = {"config": {"hit_rate": 0.65}, "roofline": {"frac": 0.6},
            "runs": [{"frac_of_8tbs": 0.7, "hit_rate": 0.35}]}
    assert bench.check_line(good) is good
    for bad in ({"config": {"hit_rate": 89.66}}, {"roofline": {"frac": 16.6}},
                {"runs": [{"frac_of_8tbs": -0.1}]}):
        with pytest.raises(AssertionError):
            bench.check_line(bad)
    # Missing fields (traffic unmeasured, no hit rate) are not an error.
    assert bench.check_line({"roofline": {"frac": None}})
