"""Exact checks of the in-register dynamic mask and of the work schedule (GPU).

Pair extraction: with one-hot value vectors, every element of an output is a single
term of Eq. 5 or of its backward, so the device output *is* the matrix of p_ij (or of
dS_ij) for a range of keys/queries:
    v_j = e_(j - 128 h)   on head h        ->  out[i, h, c]  = p_(i, 128h + c)
    dout_i = e_(i - 128 h)                 ->  dv[j, h, c]   = p_(128h + c, j)
    q_i = e_(i - 128 h)                    ->  dk[j, h, c]   = alpha dS_(128h + c, j)
    k_j = e_(j - 128 h)                    ->  dq[i, h, c]   = alpha dS_(i, 128h + c)
A pair the mask hides gives an exact zero, a visible one a non-zero value (the scores
are random), so the zero patterns of device and oracle must agree bit for bit; the
values must agree to bf16 precision.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2505_18654_amd import ops
from synth import SEG_CAND, SEG_HIST, SEG_RT, SEG_USER, make_layout
from tests.gpu_util import say

pytestmark = pytest.mark.gpu

U, S, R, C = SEG_USER, SEG_HIST, SEG_RT, SEG_CAND


@pytest.fixture(scope="module", autouse=True)
def need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def users_for_extraction():
    rng = np.random.default_rng(11)
    out = {}
    # canonical order [U|S|R|I] spanning 3 query tiles of 128 and 5 key tiles of 64
    seg = [U] * 5 + [S] * 180 + [R] * 60 + [C] * 55
    ts = [0] * 5 + sorted(rng.integers(-10**6, 0, 180).tolist()) + \
        sorted(rng.choice(1000, 60, replace=False).tolist()) + rng.integers(0, 1000, 55).tolist()
    out["canonical"] = (seg, ts)
    # shuffled segments with many timestamp ties
    perm = rng.permutation(300)
    seg2 = np.array(seg)[perm].tolist()
    ts2 = np.where(np.array(seg2) >= R, rng.integers(0, 8, 300), np.array(ts)[perm]).tolist()
    out["shuffled_ties"] = (seg2, ts2)
    # candidates first, then real-time: masked tiles in the upper left
    seg3 = [C] * 130 + [R] * 100 + [S] * 70
    ts3 = rng.integers(0, 500, 130).tolist() + sorted(rng.integers(0, 500, 100).tolist()) + [-1] * 70
    out["cand_first"] = (seg3, ts3)
    return out


def bf16(x):
    return torch.tensor(x, dtype=torch.float32).to(torch.bfloat16)


def run_case(seg, ts, which, seed=0, bias=False, alpha=1.0):
    n = len(seg)
    H, dh = (n + 127) // 128, 128
    rng = np.random.default_rng(seed)
    rab = (0.5 * rng.standard_normal((H, 64))) if bias else None
    onehot = np.zeros((n, H, dh), np.float32)
    for j in range(n):
        onehot[j, j // 128, j % 128] = 1.0
    rnd = lambda: (rng.standard_normal((n, H, dh)) / np.sqrt(dh)).astype(np.float32)
    q, k, v, do = rnd(), rnd(), rnd(), rnd()
    if which == "fwd":
        v = onehot
    elif which == "dv":
        do = onehot
    elif which == "dk":
        q = onehot
    elif which == "dq":
        k = onehot
    # values exactly as the device sees them
    q, k, v, do = (bf16(x).float().numpy() for x in (q, k, v, do))
    off = np.array([0, n])
    seg_a, ts_a = np.array(seg, np.int8), np.array(ts, np.int32)
    jag = ops.Jagged.from_host(off, seg_a, ts_a)
    tq, tk, tv, tdo = (torch.from_numpy(x).to("cuda", torch.bfloat16) for x in (q, k, v, do))
    trab = None if rab is None else torch.tensor(rab, dtype=torch.float32, device="cuda")
    if which == "fwd":
        got = ops.attn_fwd(tq, tk, tv, jag, trab, alpha)
        want = oracle.attn_fwd(off, seg_a, ts_a, q, k, v, rab, alpha)
    else:
        dq, dk, dv, _ = ops.attn_bwd(tq, tk, tv, tdo, jag, trab, alpha, need_drab=False)
        rq, rk, rv, _ = oracle.attn_bwd(off, seg_a, ts_a, q, k, v, do, rab, alpha)
        got, want = {"dv": (dv, rv), "dk": (dk, rk), "dq": (dq, rq)}[which]
    torch.cuda.synchronize()
    return got.float().cpu().numpy(), want


@pytest.mark.parametrize("which", ["fwd", "dv", "dk", "dq"])
@pytest.mark.parametrize("name", list(users_for_extraction()))
def test_pair_extraction(name, which):
    check_extraction(name, which)


# With a relative bias the forward masks through the score (alpha s + rab about -1e30, so
# silu gives exactly zero); with |alpha| < 1e-7 it selects zero element by element instead.
@pytest.mark.parametrize("which, alpha", [("fwd", 1.0), ("fwd", 1e-8), ("fwd", -0.7), ("dv", 1.0), ("dk", 1.0),
                                          ("dq", 1.0)])
@pytest.mark.parametrize("name", list(users_for_extraction()))
def test_pair_extraction_with_bias(name, which, alpha):
    check_extraction(name, which, bias=True, alpha=alpha)


def check_extraction(name, which, bias=False, alpha=1.0):
    seg, ts = users_for_extraction()[name]
    say(f"[mask] {name} {which} n={len(seg)} bias={bias} alpha={alpha}")
    got, want = run_case(seg, ts, which, bias=bias, alpha=alpha)
    n = len(seg)
    H = (n + 127) // 128
    # extracted matrices: rows = the other index, cols = 128h + c (< n)
    g = np.concatenate([got[:, h, :] for h in range(H)], axis=1)[:, :n]
    w = np.concatenate([want[:, h, :] for h in range(H)], axis=1)[:, :n]
    zero_g, zero_w = g == 0.0, w == 0.0
    assert np.array_equal(zero_g, zero_w), f"mask pattern differs at {np.argwhere(zero_g != zero_w)[:5]}"
    vis = ~zero_w
    # bf16 rounding of p (or dS) is <= 2^-8 relative; scores q.k that nearly cancel carry
    # an fp32 accumulation error that is absolute, hence the small floor.
    floor = 1e-4 * np.abs(w).max()
    excess = np.abs(g[vis] - w[vis]) - 2.0 ** -7 * np.abs(w[vis])
    say(f"[mask] {name} {which} visible={int(vis.sum())} max excess/floor={excess.max() / floor:.2e}")
    assert excess.max() <= floor


def test_schedule_covers_every_tile_once():
    """Work list of the bf16 kernels: every (user, head, 128-row tile) exactly once."""
    L = make_layout("mtgr_large")
    H, dh = L.spec.heads, L.spec.head_dim
    T, B = L.total_tokens, L.num_users
    jag = ops.Jagged.from_host(L.offsets, L.seg, L.ts)
    q = torch.zeros((T, H, dh), dtype=torch.bfloat16, device="cuda")
    p = ops.attn_problem(jag, q, q, q, q)
    ws = ops.workspace_for(p, "cuda")
    say("[schedule] mtgr_large")
    ops.attn_fwd(q, q, q, jag, workspace=ws)
    torch.cuda.synchronize()
    tile = 128
    ntile = (L.max_seqlen + 63) // 64
    items_bound = H * (T // tile + B)
    slots = 8 * ((L.max_seqlen + tile - 1) // tile + (items_bound + 7) // 8)
    off_items = (B * ntile * 16 + 255) // 256 * 256
    raw = ws.cpu().numpy()
    items = raw[off_items:off_items + slots * 8].view(np.int32).reshape(slots, 2)
    live = items[items[:, 0] >= 0]
    got = sorted((int(b), int(y) & 255, int(y) >> 8) for b, y in live)
    n = np.diff(L.offsets)
    want = sorted((b, h, t) for b in range(B) for h in range(H) for t in range((n[b] + tile - 1) // tile))
    assert got == want
    # all tiles of one (user, head) share an XCD (slot mod 8)
    xcd = {}
    for s in np.nonzero(items[:, 0] >= 0)[0]:
        key = (int(items[s, 0]), int(items[s, 1]) & 255)
        xcd.setdefault(key, set()).add(int(s) % 8)
    assert all(len(v) == 1 for v in xcd.values())
    # tile summaries
    summ = raw[:B * ntile * 16].view(np.int32).reshape(B, ntile, 4)
    for b in range(B):
        sl = L.user_slice(b)
        sg, tsv = L.seg[sl], L.ts[sl].astype(np.int64)
        for t in range((n[b] + 63) // 64):
            s_, t_ = sg[64 * t:64 * t + 64], tsv[64 * t:64 * t + 64]
            flags = (1 if np.any(s_ <= S) else 0) | (2 if len(s_) == 64 and np.all(s_ <= S) else 0) | \
                (4 if np.any(s_ == R) else 0) | (8 if np.any(s_ >= R) else 0) | (16 if np.any(s_ == R + 1) else 0)
            mn = int(t_[s_ == R].min()) if np.any(s_ == R) else 2**31 - 1
            mx = int(t_[s_ >= R].max()) if np.any(s_ >= R) else -2**31
            assert tuple(summ[b, t, :3]) == (flags, mn, mx), (b, t)
