"""Pins of the oracle's mask, pair count and bias bucket (CPU only)."""
import os

import numpy as np
import pytest

import oracle
from synth import SEG_CAND, SEG_HIST, SEG_RT, SEG_USER, make_layout

HERE = os.path.dirname(os.path.abspath(__file__))


def load_worked_example():
    names, seg, ts, rows = [], [], [], {}
    with open(os.path.join(HERE, "golden", "worked_example_mask.txt")) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            parts = line.split()
            if parts[0] == "token":
                names.append(parts[1])
                seg.append(int(parts[2]))
                ts.append(int(parts[3]))
            elif parts[0] == "row":
                rows[parts[1]] = [int(x) for x in parts[2:]]
    mat = np.array([rows[n] for n in names], dtype=bool)
    return names, np.array(seg, np.int8), np.array(ts, np.int32), mat


def test_worked_example_matches_paper_walkthrough():
    names, seg, ts, expected = load_worked_example()
    got = oracle.mask_matrix(seg, ts)
    assert got.shape == (9, 9)
    np.testing.assert_array_equal(got, expected)
    idx = {n: i for i, n in enumerate(names)}
    # individual statements of the walk-through
    assert got[idx["rt1"], idx["rt2"]] and not got[idx["rt2"], idx["rt1"]]
    assert not got[idx["target2"], idx["rt1"]] and not got[idx["target3"], idx["rt1"]]
    assert not got[idx["target3"], idx["rt2"]]
    assert got[idx["target1"], idx["rt2"]] and got[idx["target2"], idx["rt2"]]
    for t in ("target1", "target2", "target3"):          # a candidate sees no other candidate
        for o in ("target1", "target2", "target3"):
            assert got[idx[t], idx[o]] == (t == o)


# One line per (query segment, key segment, key-vs-query time) case, stated from the rules.
RULE_CASES = [
    # static keys are visible to everybody (rule 1)
    *[(sq, sk, rel, True) for sq in range(4) for sk in (SEG_USER, SEG_HIST) for rel in (-1, 0, 1)],
    # a real-time key is seen by later real-time / candidate queries only (rule 2)
    *[(sq, SEG_RT, -1, True) for sq in (SEG_RT, SEG_CAND)],
    *[(sq, SEG_RT, rel, False) for sq in (SEG_RT, SEG_CAND) for rel in (0, 1)],
    *[(sq, SEG_RT, rel, False) for sq in (SEG_USER, SEG_HIST) for rel in (-1, 0, 1)],
    # a candidate key is never seen by another token (rule 3)
    *[(sq, SEG_CAND, rel, False) for sq in range(4) for rel in (-1, 0, 1)],
]


@pytest.mark.parametrize("seg_q,seg_k,rel,want", RULE_CASES)
def test_mask_rules(seg_q, seg_k, rel, want):
    ts_q = 1000
    ts_k = ts_q + rel                       # rel = -1: key earlier than query
    assert oracle.visible(seg_q, ts_q, seg_k, ts_k, False) == want
    assert oracle.visible(seg_q, ts_q, seg_k, ts_k, True)   # everyone sees itself


def test_mask_extreme_timestamps():
    i32min, i32max = -2**31, 2**31 - 1
    assert oracle.visible(SEG_CAND, i32max, SEG_RT, i32min, False)
    assert not oracle.visible(SEG_CAND, i32min, SEG_RT, i32max, False)
    assert not oracle.visible(SEG_RT, i32min, SEG_RT, i32min, False)


def closed_form_pairs(seg, ts):
    """Visible pairs of one [U|S|R|I] user, counted segment by segment."""
    n_s = int(np.sum(seg <= SEG_HIST))
    rt_ts = ts[seg == SEG_RT].astype(np.int64)
    cand_ts = ts[seg == SEG_CAND].astype(np.int64)
    n_r, n_i = len(rt_ts), len(cand_ts)
    rr = int(np.sum(rt_ts[None, :] < rt_ts[:, None]))
    ir = int(np.sum(rt_ts[None, :] < cand_ts[:, None]))
    return n_s * n_s + n_r * n_s + rr + n_r + n_i * n_s + ir + n_i


@pytest.mark.parametrize("config", ["tiny", "small"])
def test_pair_count_closed_form(config):
    L = make_layout(config)
    sub = L.subset(range(min(L.num_users, 6)))
    expected = sum(closed_form_pairs(sub.seg[sub.user_slice(b)], sub.ts[sub.user_slice(b)])
                   for b in range(sub.num_users))
    assert oracle.count_visible(sub.offsets, sub.seg, sub.ts) == expected


def test_pair_count_with_ties_and_empty_segments():
    seg = np.array([SEG_RT, SEG_RT, SEG_CAND, SEG_CAND, SEG_RT], np.int8)   # no static tokens
    ts = np.array([5, 5, 5, 6, 1], np.int32)                                 # ties everywhere
    off = np.array([0, 5])
    assert oracle.count_visible(off, seg, ts) == closed_form_pairs(seg, ts)
    off2 = np.array([0, 0, 5, 5])                                            # empty users
    assert oracle.count_visible(off2, seg, ts) == closed_form_pairs(seg, ts)


BUCKET_TABLE = {0: 0, 1: 1, 2: 2, 3: 3, 4: 4, 5: 4, 6: 5, 7: 5, 8: 6, 11: 6, 12: 7, 15: 7, 16: 8,
                86399: 32, 86400: 32, 98303: 32, 98304: 33, 2**31 - 1: 61, 2**31: 62, 3 * 2**30 - 1: 62, 3 * 2**30: 63,
                2**32 - 1: 63}


def test_bucket_table():
    for delta, want in BUCKET_TABLE.items():
        assert oracle.rab_bucket(delta) == want, delta


def test_bucket_bit_length_identity():
    rng = np.random.default_rng(5)
    deltas = np.concatenate([np.arange(0, 5000), rng.integers(0, 2**32, 20000, dtype=np.uint64)])
    for d in deltas.tolist():
        d = int(d)
        if d < 2:
            want = d
        else:
            e = d.bit_length() - 1
            want = 2 * e + (1 if 2 * d >= 3 * (1 << e) else 0)
        assert oracle.rab_bucket(d) == want
    got = [oracle.rab_bucket(d) for d in range(0, 70000)]
    assert all(a <= b for a, b in zip(got, got[1:]))          # monotone in the gap
    assert max(oracle.rab_bucket(int(d)) for d in deltas.tolist()) <= 63


def test_bench_pair_count_matches_oracle():
    import bench
    for config in ("tiny", "small"):
        L = make_layout(config)
        sub = L.subset(range(min(L.num_users, 8)))
        assert int(bench.visible_pairs(sub).sum()) == oracle.count_visible(sub.offsets, sub.seg, sub.ts)
