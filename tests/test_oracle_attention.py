"""Pins of the oracle's attention (Eq. 5) forward and backward (CPU only)."""
import numpy as np
import pytest
import torch

import oracle
from synth import SEG_CAND, SEG_HIST, SEG_RT, SEG_USER, make_layout, make_values
from tests.dense_ref import dense_attention


def random_case(seed, B=3, H=2, dh=8, max_len=14, rab_buckets=0, ties=False):
    """Random [U|S|R|I] users (any segment may be empty) with random values."""
    rng = np.random.default_rng(seed)
    segs, tss, lens = [], [], []
    for _ in range(B):
        cnt = rng.integers(0, max_len // 4 + 1, size=4)
        seg = np.repeat(np.arange(4, dtype=np.int8), cnt)
        span = 6 if ties else 1000
        ts = np.where(seg <= SEG_HIST, -rng.integers(1, 500, size=len(seg)),
                      rng.integers(0, span, size=len(seg))).astype(np.int32)
        ts[seg == SEG_USER] = 0
        rt = seg == SEG_RT
        ts[rt] = np.sort(ts[rt])
        segs.append(seg)
        tss.append(ts)
        lens.append(len(seg))
    off = np.zeros(B + 1, np.int64)
    off[1:] = np.cumsum(lens)
    T = int(off[-1])
    q, k, v, do = (rng.standard_normal((T, H, dh)) for _ in range(4))
    rab = 0.3 * rng.standard_normal((H, rab_buckets)) if rab_buckets else None
    return off, np.concatenate(segs), np.concatenate(tss), q, k, v, do, rab


def t64(x, grad=False):
    return None if x is None else torch.tensor(x, dtype=torch.float64, requires_grad=grad)


@pytest.mark.parametrize("seed", range(6))
@pytest.mark.parametrize("rab_buckets", [0, 64, 9])
def test_fwd_matches_dense(seed, rab_buckets):
    off, seg, ts, q, k, v, _, rab = random_case(seed, rab_buckets=rab_buckets, ties=seed % 2 == 0)
    alpha = 0.7 if seed % 3 == 0 else 1.0
    got = oracle.attn_fwd(off, seg, ts, q, k, v, rab, alpha)
    want = dense_attention(off, seg, ts, t64(q), t64(k), t64(v), t64(rab), alpha).numpy()
    np.testing.assert_allclose(got, want, rtol=1e-12, atol=1e-13)


@pytest.mark.parametrize("seed", range(4))
@pytest.mark.parametrize("rab_buckets", [0, 64])
def test_bwd_matches_autograd(seed, rab_buckets):
    off, seg, ts, q, k, v, do, rab = random_case(100 + seed, rab_buckets=rab_buckets, ties=True)
    alpha = 1.3
    dq, dk, dv, drab = oracle.attn_bwd(off, seg, ts, q, k, v, do, rab, alpha)
    tq, tk, tv, trab = t64(q, True), t64(k, True), t64(v, True), t64(rab, rab is not None)
    out = dense_attention(off, seg, ts, tq, tk, tv, trab, alpha)
    out.backward(torch.tensor(do))
    np.testing.assert_allclose(dq, tq.grad.numpy(), rtol=1e-11, atol=1e-12)
    np.testing.assert_allclose(dk, tk.grad.numpy(), rtol=1e-11, atol=1e-12)
    np.testing.assert_allclose(dv, tv.grad.numpy(), rtol=1e-11, atol=1e-12)
    if rab is not None:
        np.testing.assert_allclose(drab, trab.grad.numpy(), rtol=1e-11, atol=1e-12)


def test_bwd_finite_differences():
    off, seg, ts, q, k, v, do, rab = random_case(7, rab_buckets=64)
    dq, dk, dv, drab = oracle.attn_bwd(off, seg, ts, q, k, v, do, rab)
    rng = np.random.default_rng(0)
    h = 1e-6
    args = {"q": q, "k": k, "v": v, "rab": rab}
    grads = {"q": dq, "k": dk, "v": dv, "rab": drab}
    for name in args:
        for _ in range(3):
            delta = rng.standard_normal(args[name].shape)
            plus = dict(args)
            minus = dict(args)
            plus[name] = args[name] + h * delta
            minus[name] = args[name] - h * delta
            fp = oracle.attn_fwd(off, seg, ts, plus["q"], plus["k"], plus["v"], plus["rab"])
            fm = oracle.attn_fwd(off, seg, ts, minus["q"], minus["k"], minus["v"], minus["rab"])
            numeric = np.sum(do * (fp - fm)) / (2 * h)
            analytic = np.sum(grads[name] * delta)
            assert abs(numeric - analytic) <= 1e-6 * max(1.0, abs(analytic)), name


def test_all_static_reduces_to_library_silu_attention():
    rng = np.random.default_rng(3)
    n, H, dh = 11, 3, 8
    seg = np.full(n, SEG_HIST, np.int8)
    seg[:2] = SEG_USER
    ts = np.sort(-rng.integers(1, 10**6, n)).astype(np.int32)
    q, k, v = (rng.standard_normal((n, H, dh)) for _ in range(3))
    got = oracle.attn_fwd([0, n], seg, ts, q, k, v, None, 0.5)
    for h in range(H):
        S = 0.5 * torch.tensor(q[:, h]) @ torch.tensor(k[:, h]).T
        want = torch.nn.functional.silu(S) / n @ torch.tensor(v[:, h])
        np.testing.assert_allclose(got[:, h], want.numpy(), rtol=1e-12, atol=1e-14)


def test_causal_reduction():
    """All tokens real-time with ts_i = i: lower-triangular mask with diagonal (causal HSTU)."""
    rng = np.random.default_rng(4)
    n, H, dh = 13, 2, 8
    seg = np.full(n, SEG_RT, np.int8)
    ts = np.arange(n, dtype=np.int32)
    q, k, v = (rng.standard_normal((n, H, dh)) for _ in range(3))
    got = oracle.attn_fwd([0, n], seg, ts, q, k, v)
    causal = torch.tril(torch.ones(n, n, dtype=torch.float64))
    for h in range(H):
        S = torch.tensor(q[:, h]) @ torch.tensor(k[:, h]).T
        want = (torch.nn.functional.silu(S) * causal) / n @ torch.tensor(v[:, h])
        np.testing.assert_allclose(got[:, h], want.numpy(), rtol=1e-12, atol=1e-14)


def test_zero_queries_give_zero():
    off, seg, ts, q, k, v, _, _ = random_case(9)
    out = oracle.attn_fwd(off, seg, ts, np.zeros_like(q), k, v)
    assert np.all(out == 0.0)


def test_jagged_equals_padded_and_masked():
    """Jagged result = padded batch with invisible pad tokens and per-user length divisor."""
    off, seg, ts, q, k, v, _, _ = random_case(11, B=4)
    got = oracle.attn_fwd(off, seg, ts, q, k, v)
    B = len(off) - 1
    L = int(np.max(np.diff(off)))
    T_pad = B * L
    H, dh = q.shape[1:]
    for b in range(B):
        n = off[b + 1] - off[b]
        sl = slice(off[b], off[b + 1])
        qp, kp, vp = (np.zeros((L, H, dh)) for _ in range(3))
        qp[:n], kp[:n], vp[:n] = q[sl], k[sl], v[sl]
        valid = np.arange(L) < n
        for h in range(H):
            S = torch.tensor(qp[:, h]) @ torch.tensor(kp[:, h]).T
            M = torch.tensor(oracle.mask_matrix(np.pad(seg[sl], (0, L - n)), np.pad(ts[sl], (0, L - n))))
            M = M & torch.tensor(valid[:, None] & valid[None, :])
            O = (torch.where(M, torch.nn.functional.silu(S), 0.0) / n) @ torch.tensor(vp[:, h])
            np.testing.assert_allclose(got[sl, h], O[:n].numpy(), rtol=1e-12, atol=1e-14)
    assert T_pad >= len(seg)


def test_candidate_independence():
    off, seg, ts, q, k, v, do, _ = random_case(12, B=2, max_len=24)
    cands = np.nonzero(seg == SEG_CAND)[0]
    assert len(cands) >= 2
    c = cands[0]
    q2, k2, v2, ts2 = q.copy(), k.copy(), v.copy(), ts.copy()
    q2[c] += 1.0
    k2[c] -= 2.0
    v2[c] *= 3.0
    ts2[c] += 77
    o1 = oracle.attn_fwd(off, seg, ts, q, k, v)
    o2 = oracle.attn_fwd(off, seg, ts2, q2, k2, v2)
    others = np.arange(len(seg)) != c
    np.testing.assert_array_equal(o1[others], o2[others])
    g1 = oracle.attn_bwd(off, seg, ts, q, k, v, do)
    g2 = oracle.attn_bwd(off, seg, ts2, q2, k2, v2, do)
    other_c = cands[cands != c]
    for a, b in zip(g1[:3], g2[:3]):
        np.testing.assert_array_equal(a[other_c], b[other_c])


def test_user_permutation():
    off, seg, ts, q, k, v, do, rab = random_case(13, B=4, rab_buckets=64)
    perm = [2, 0, 3, 1]
    idx = np.concatenate([np.arange(off[b], off[b + 1]) for b in perm])
    lens = np.diff(off)[perm]
    off2 = np.concatenate([[0], np.cumsum(lens)])
    o1 = oracle.attn_fwd(off, seg, ts, q, k, v, rab)
    o2 = oracle.attn_fwd(off2, seg[idx], ts[idx], q[idx], k[idx], v[idx], rab)
    np.testing.assert_array_equal(o1[idx], o2)
    g1 = oracle.attn_bwd(off, seg, ts, q, k, v, do, rab)
    g2 = oracle.attn_bwd(off2, seg[idx], ts[idx], q[idx], k[idx], v[idx], do[idx], rab)
    for a, b in zip(g1[:3], g2[:3]):
        np.testing.assert_array_equal(a[idx], b)
    np.testing.assert_allclose(g1[3], g2[3], rtol=1e-12, atol=1e-14)


def test_token_permutation_within_user():
    off, seg, ts, q, k, v, _, rab = random_case(14, B=1, max_len=30, rab_buckets=64)
    rng = np.random.default_rng(0)
    p = rng.permutation(len(seg))
    o1 = oracle.attn_fwd(off, seg, ts, q, k, v, rab)
    o2 = oracle.attn_fwd(off, seg[p], ts[p], q[p], k[p], v[p], rab)
    np.testing.assert_allclose(o1[p], o2, rtol=1e-12, atol=1e-14)


def test_divisor_is_user_length_including_candidates():
    """Adding candidates leaves what other tokens see unchanged and rescales them by n/n'."""
    off, seg, ts, q, k, v, _, _ = random_case(15, B=1, max_len=20)
    n = len(seg)
    extra = 5
    rng = np.random.default_rng(1)
    seg2 = np.concatenate([seg, np.full(extra, SEG_CAND, np.int8)])
    ts2 = np.concatenate([ts, rng.integers(0, 1000, extra).astype(np.int32)])
    q2, k2, v2 = (np.concatenate([x, rng.standard_normal((extra,) + x.shape[1:])]) for x in (q, k, v))
    o1 = oracle.attn_fwd([0, n], seg, ts, q, k, v)
    o2 = oracle.attn_fwd([0, n + extra], seg2, ts2, q2, k2, v2)
    np.testing.assert_allclose(o2[:n] * (n + extra) / n, o1, rtol=1e-12, atol=1e-14)


def test_empty_users_and_empty_batch():
    off, seg, ts, q, k, v, do, _ = random_case(16, B=2)
    off_e = np.array([0, 0, off[1], off[1], off[2], off[2]])
    np.testing.assert_array_equal(oracle.attn_fwd(off, seg, ts, q, k, v),
                                  oracle.attn_fwd(off_e, seg, ts, q, k, v))
    z = np.zeros((0, 2, 8))
    assert oracle.attn_fwd([0], np.zeros(0, np.int8), np.zeros(0, np.int32), z, z, z).shape == (0, 2, 8)


def test_synthetic_tiny_batch_against_dense():
    L = make_layout("tiny")
    v = make_values(L)
    got = oracle.attn_fwd(L.offsets, L.seg, L.ts, v["q"], v["k"], v["v"])
    want = dense_attention(L.offsets, L.seg, L.ts, t64(v["q"]), t64(v["k"]), t64(v["v"])).numpy()
    np.testing.assert_allclose(got, want, rtol=1e-12, atol=1e-14)
