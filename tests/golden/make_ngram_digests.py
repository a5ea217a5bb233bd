"""Writes ngram_top_workload2.json: the CPU oracle's frequency ranking of the
2^26-token Zipf(1.1) stream behind the 2^20-phrase decode table (phrase
mining by n-gram frequency, Sec. 4.2), for n = 2, 3, 4, top 2^19 ranks each.

Only the oracle (oracle.ngram_top) and the seeded stream generator
(synth.workload2_stream) are called.  The output holds, per n, the number of
ranks written, SHA-256 digests of the tuples (int32, [m x n], row-major,
little-endian) and of the counts (int64, little-endian), and the first ranks
in clear; and the SHA-256 of the stream itself, so that a change of the
generator shows as such and not as a construction error.

Run from the repository root:  python tests/golden/make_ngram_digests.py
(about 10 GB of memory and a few minutes: the oracle sorts one vector per
window).
"""
import hashlib
import json
import os
import re
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)

import oracle  # noqa: E402
import synth  # noqa: E402

OUT = os.path.join(os.path.dirname(os.path.abspath(__file__)), "ngram_top_workload2.json")
TOP = 1 << 19
HEAD = 8


def digest(a):
    return hashlib.sha256(np.ascontiguousarray(a).astype(a.dtype.newbyteorder("<")).tobytes()).hexdigest()


def main():
    stream = synth.workload2_stream()
    assert stream.dtype == np.int32 and stream.size == 1 << 26
    doc = {
        "what": "top 2^19 n-grams of the 2^26-token workload-2 stream by count, ties by tuple "
                "(oracle.ngram_top); tuples int32 [m x n] and counts int64, little-endian",
        "stream_tokens": int(stream.size),
        "stream_sha256": digest(stream),
        "vocab": synth.V,
        "top": TOP,
        "n": {},
    }
    for n in (2, 3, 4):
        t0 = time.time()
        tup, cnt = oracle.ngram_top(stream, synth.V, n, 0, TOP)
        doc["n"][str(n)] = {
            "ranks": int(cnt.size),
            "tuples_sha256": digest(tup),
            "counts_sha256": digest(cnt),
            "count_sum": int(cnt.sum()),
            "head": [[tup[i].tolist(), int(cnt[i])] for i in range(min(HEAD, cnt.size))],
            "last": [tup[-1].tolist(), int(cnt[-1])],
        }
        print("n=%d: %d ranks in %.0f s" % (n, cnt.size, time.time() - t0), flush=True)
    with open(OUT, "w") as f:
        f.write(layout(doc) + "\n")


def layout(doc):
    """JSON with one line per (tuple, count) entry."""
    out = json.dumps(doc, indent=1)
    out = re.sub(r"\[\s+([-\d,\s]+?)\s+\]",
                 lambda m: "[" + ", ".join(x.strip() for x in m.group(1).split(",")) + "]", out)
    out = re.sub(r"\[\s+(\[[^\[\]]*\]),\s+(\d+)\s+\]", r"[\1, \2]", out)
    assert json.loads(out) == doc
    return out


if __name__ == "__main__":
    main()
