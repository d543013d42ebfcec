"""The work counts the benchmark divides by (bench.visible_pairs, bench.candidate_pairs) against
a brute-force count of the oracle's mask on small users (no GPU)."""
import numpy as np

import bench
import oracle
from synth import make_layout


def test_pair_counts_match_the_mask():
    for name, users in (("small", [0, 1, 2, 7]), ("mtgr_small", [3, 4]), ("serving", [5])):
        L = make_layout(name).subset(users)
        want_all, want_cand = [], []
        for b in range(L.num_users):
            sl = L.user_slice(b)
            M = oracle.mask_matrix(L.seg[sl], L.ts[sl])
            want_all.append(int(M.sum()))
            want_cand.append(int(M[L.seg[sl] == 3].sum()))
        assert bench.visible_pairs(L).tolist() == want_all, name
        assert bench.candidate_pairs(L).tolist() == want_cand, name
