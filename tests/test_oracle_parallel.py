"""The parallel drivers of the oracle used by the GPU parity tests at the
large workloads (row ranges in threads) give the bits of one oracle call over
all rows."""
import numpy as np

import oracle
from oracle.parallel import oracle_assign, oracle_p


def test_parallel_p_equals_one_call():
    rng = np.random.default_rng(11)
    anc = rng.standard_normal((3, 37, 192))
    vis = rng.standard_normal((3, 301, 192))
    p = oracle_p(anc, vis)
    for b in range(3):
        ref = oracle.dedup(anc[b:b + 1], vis[b:b + 1], 50, want_assign=False)["p"][0]
        assert np.array_equal(p[b], ref)


def test_parallel_assign_equals_one_call():
    rng = np.random.default_rng(12)
    vis = rng.standard_normal((523, 128))
    kept = np.sort(rng.choice(523, 97, replace=False)).astype(np.int32)
    rows = np.setdiff1d(np.arange(523), kept).astype(np.int32)
    a, b1, b2 = oracle_assign(vis, kept, rows)
    ra, rb1, rb2 = oracle.assign(vis, kept, rows)
    assert np.array_equal(a, ra) and np.array_equal(b1, rb1) and np.array_equal(b2, rb2)
    full = oracle.dedup(np.ones((1, 1, 128)), vis[None], 97)  # any kept list works here
    fa, _, _ = oracle_assign(vis, full["kept"][0], np.arange(523, dtype=np.int32))
    assert np.array_equal(fa, full["assign"][0])
