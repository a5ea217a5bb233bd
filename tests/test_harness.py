"""The test harness's oracle shortcut for very large tables: an oracle built
from only the phrases that equal some query window answers the query exactly
like one built from the whole table."""
import numpy as np

import oracle
import synth

from . import harness as H


def test_subset_oracle_equals_full_oracle():
    table = synth.config2_table()
    full = H.oracle_table(table)
    for k, B in enumerate((64, 2000)):
        batch = synth.decode_batch(1, B, set_index=30 + k)
        rows = H.subset_rows(table, batch.tokens, batch.ctx, batch.S)
        sub = oracle.Table(table.tokens[rows], table.lens[rows], 2, 3, synth.V)
        h1, r1, l1 = full.lookup(batch.tokens, batch.ctx, batch.S)
        h2, r2, l2 = sub.lookup(batch.tokens, batch.ctx, batch.S)
        np.testing.assert_array_equal(h1, h2)
        np.testing.assert_array_equal(l1, l2)
        np.testing.assert_array_equal(r1, np.where(r2 >= 0, rows[np.maximum(r2, 0)], -1))
        assert 0.4 < h1.mean() < 0.9
