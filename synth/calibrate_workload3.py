"""How workload 3's stop-phrase filter was chosen.

Workload 3 asks for a 4M-phrase 2/3/4-gram table built from a 200M-token
Zipf(1.1) stream with a hit rate of about 30-40% on Zipf(1.1) prefill.
Taking the most frequent n-grams gives a much higher rate, so the table skips
the STOP most frequent n-grams of each length first (a stop-phrase filter).
This script prints the hit rate of the first query batch for a range of STOP
values, computing membership with packed integer keys (4-grams through a
64-bit mix; collisions only blur the estimate).  The exact rate of the chosen
value is checked by the test suite with the oracle.

    python -m synth.calibrate_workload3
"""
import numpy as np

from . import V, TAG_STREAM, ngram_top, zipf_tokens
from .workloads import prefill_batch

WANT = {2: 1 << 21, 3: 1 << 20, 4: 1 << 20}


def packed(t):
    t = t.astype(np.uint64)
    k = np.zeros(t.shape[0], np.uint64)
    for j in range(t.shape[1]):
        k = k * np.uint64(V) + t[:, j]
    return k


def main(stops=(6000, 20000, 40000, 60000, 80000, 100000, 130000, 160000)):
    stream = zipf_tokens(2, TAG_STREAM, 200_000_000, 1.1)
    top = {n: ngram_top(stream, n, max(stops) + WANT[n])[0] for n in (2, 3, 4)}
    q = prefill_batch(2, 8, 4096).tokens
    win = {}
    for n in (2, 3, 4):
        w = np.stack([q[:, n - 1 - j:q.shape[1] - j] for j in range(n - 1, -1, -1)], axis=-1)
        win[n] = packed(w.reshape(-1, n)).reshape(q.shape[0], -1)
    for stop in stops:
        hit = np.zeros(q.shape, bool)
        for n in (2, 3, 4):
            keys = packed(top[n][stop:stop + WANT[n]])
            m = np.isin(win[n], keys)
            hit[:, n - 1:] |= m
        print("STOP=%6d hit rate %.4f" % (stop, hit.mean()))


if __name__ == "__main__":
    main()
