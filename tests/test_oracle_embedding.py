"""Pins of the embedding-table oracle (CPU): de-duplication against numpy.unique, the
sparse SGD sum against numpy.add.at, counters against collections.Counter, eviction by
brute force, and the row-capacity rule."""
import collections

import numpy as np
import pytest

from oracle.embedding import DictTable


def zipf_ids(rng, n, universe, a=1.2):
    return (rng.zipf(a, n) % universe).astype(np.uint64) * np.uint64(2654435761) + np.uint64(7)


def test_dedup_matches_numpy_unique():
    rng = np.random.default_rng(0)
    for n in (0, 1, 7, 1000):
        ids = zipf_ids(rng, n, 50)
        unique, occ, inverse = DictTable.dedup(ids)
        ref_u, ref_inv, ref_cnt = np.unique(ids, return_inverse=True, return_counts=True)
        assert sorted(unique) == [int(x) for x in ref_u]
        assert [unique[i] for i in inverse] == [int(x) for x in ids]
        counts = dict(zip((int(x) for x in ref_u), (int(c) for c in ref_cnt)))
        assert [counts[u] for u in unique] == occ
        # first-occurrence order
        seen = []
        for x in ids:
            if int(x) not in seen:
                seen.append(int(x))
        assert unique == seen


def test_sgd_matches_add_at():
    rng = np.random.default_rng(1)
    dim = 8
    ids = zipf_ids(rng, 300, 20)
    t = DictTable(100, dim)
    u, occ, inv = t.dedup(ids)
    t.lookup(u, occ, now=5, insert=True)
    grad = rng.standard_normal((len(ids), dim))
    t.sgd(ids, grad, lr=0.25)
    acc = np.zeros((len(u), dim))
    np.add.at(acc, np.asarray(inv), grad)
    got = t.gather(u)
    np.testing.assert_allclose(got, -0.25 * acc, rtol=1e-12, atol=1e-12)
    # every position of an ID sees the same row
    np.testing.assert_array_equal(t.gather(ids), got[np.asarray(inv)])


def test_counts_and_timestamps_over_batches():
    rng = np.random.default_rng(2)
    t = DictTable(1000, 4)
    total = collections.Counter()
    last = {}
    for step in range(5):
        ids = zipf_ids(rng, 200, 80)
        u, occ, _ = t.dedup(ids)
        t.lookup(u, occ, now=10 * step, insert=True)
        total.update(int(x) for x in ids)
        for x in u:
            last[x] = 10 * step
    assert {k: r.count for k, r in t.rows.items()} == dict(total)
    assert {k: r.last_ts for k, r in t.rows.items()} == last


def test_lookup_without_insert_and_absent_rows():
    t = DictTable(10, 4)
    t.lookup([5, 6], [1, 1], now=1, insert=True)
    has = t.lookup([6, 7], [2, 3], now=2, insert=False)
    assert has == [True, False]
    assert 7 not in t.rows and t.rows[6].count == 3 and t.rows[6].last_ts == 2
    np.testing.assert_array_equal(t.gather([7, 5]), np.zeros((2, 4)))


def test_evict_brute_force():
    rng = np.random.default_rng(3)
    t = DictTable(500, 2)
    stamp = {}
    for step in range(6):
        ids = zipf_ids(rng, 60, 200)
        u, occ, _ = t.dedup(ids)
        t.lookup(u, occ, now=step, insert=True)
        for x in u:
            stamp[x] = step
    for thr in (0, 3, 7):
        keep = {k for k, s in stamp.items() if s >= thr}
        gone = len(t.rows) - len(keep & set(t.rows))
        assert t.evict(thr) == gone
        assert set(t.rows) == keep & set(stamp)
    # a re-inserted ID starts from a zero row and zero count
    t.lookup([12345], [4], now=9, insert=True)
    assert t.rows[12345].count == 4 and not t.rows[12345].value.any()


def test_row_capacity():
    t = DictTable(3, 2)
    t.lookup([1, 2], [1, 1], now=0, insert=True)
    with pytest.raises(OverflowError):
        t.lookup([3, 4], [1, 1], now=0, insert=True)
    t.evict(1)
    t.lookup([3, 4, 5], [1, 1, 1], now=1, insert=True)
    assert len(t.rows) == 3


def test_evict_by_count_brute_force():
    rng = np.random.default_rng(4)
    t = DictTable(1000, 2)
    total = collections.Counter()
    for step in range(4):
        ids = zipf_ids(rng, 300, 150)
        u, occ, _ = t.dedup(ids)
        t.lookup(u, occ, now=step, insert=True)
        total.update(int(x) for x in ids)
    keep = {k for k, c in total.items() if c >= 5}
    assert t.evict(0, min_count=5) == len(total) - len(keep)
    assert set(t.rows) == keep
