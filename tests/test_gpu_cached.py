"""Serving with the user side cached across requests (mtgr_hstu_attn_fwd_cached, through the
C ABI): each user's user-side keys and values (U | S | R) sit in a caller-held cache with its own
plan, and a request brings only its candidates.  The candidate rows must match
  - the oracle on the concatenated sequence [user side | candidates] (the bf16 bar of
    test_gpu_parity.py; n_b counts both sides), and
  - the candidate rows of the full forward on the concatenated batch, up to the order of the
    float sums (the candidate's own term is added after the cached tiles),
for the serving workload's users and for custom users covering RT keys later than, equal to
and earlier than the candidates, users without cached tokens or without candidates, a relative
bias, head dims 64 and 128, and two requests served from one cache.  A candidate of a user
without cached tokens sees only itself: its output is one product p_ii v_i, whose bf16 operand
p_ii keeps its rounding (up to 2^-8 relative) undiluted, so there each element's bound of the P
rounding (tests/dense_ref.operand_rounding_bounds) is subtracted as well (a numpy emulation of
the same rounding points gives the device's figures exactly)."""
import numpy as np
import pytest
import torch

import oracle
from paper_2505_18654_amd import hstu, ops
from synth import SEG_CAND, SEG_HIST, SEG_RT, SEG_USER, make_layout, make_values
from tests.dense_ref import operand_rounding_bounds
from tests.gpu_util import TOL, custom_layout, jagged, make_inputs, per_user_err, record, say, to_np
from synth.batches import Layout

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def split(L: Layout):
    """Row indices (into the full layout) of every user's user-side tokens and candidates, and
    the jagged layouts of the two sides."""
    side, cand, off_s, off_c = [], [], [0], [0]
    for b in range(L.num_users):
        sl = np.arange(L.offsets[b], L.offsets[b + 1])
        c = sl[L.seg[sl] == SEG_CAND]
        s = sl[L.seg[sl] != SEG_CAND]
        side.append(s)
        cand.append(c)
        off_s.append(off_s[-1] + len(s))
        off_c.append(off_c[-1] + len(c))
    side = np.concatenate(side).astype(np.int64) if side else np.zeros(0, np.int64)
    cand = np.concatenate(cand).astype(np.int64) if cand else np.zeros(0, np.int64)
    jag_s = ops.Jagged.from_host(off_s, L.seg[side], L.ts[side])
    jag_c = ops.Jagged.from_host(off_c, L.seg[cand], L.ts[cand])
    return side, cand, jag_s, jag_c


def run_case(L, label, requests=1):
    inp = make_inputs(L, all_exact=True)
    q, k, v, rab = inp["q"], inp["k"], inp["v"], inp["rab"]
    side, cand, jag_s, jag_c = split(L)
    say(f"[cached] {label}: {L.num_users} users, {len(side)} cached tokens, {len(cand)} candidates")
    ts_side = torch.from_numpy(side).cuda()
    ts_cand = torch.from_numpy(cand).cuda()
    cache = ops.user_cache(k[ts_side].contiguous(), v[ts_side].contiguous(), jag_s)
    full = ops.attn_fwd(q, k, v, jagged(inp), rab)
    outs = []
    for r in range(requests):
        qc, kc, vc = (x[ts_cand].contiguous() for x in (q, k, v))
        if r:   # a second request: other candidate values against the same cache
            qc, kc, vc = (torch.roll(x, 1, dims=0).contiguous() for x in (qc, kc, vc))
        outs.append((qc, kc, vc, ops.attn_fwd_cached(qc, kc, vc, jag_c, cache, rab)))
    torch.cuda.synchronize()
    vals = make_values(L, tensors=("q", "k", "v"))
    ref_full = oracle.attn_fwd(L.offsets, L.seg, L.ts, vals["q"], vals["k"], vals["v"], inp["rab_np"])
    users = list(range(L.num_users))
    sub = ops_layout(jag_c, L)
    for r, (qc, kc, vc, got) in enumerate(outs):
        if r == 0:
            want = ref_full[cand]
            # against the full forward's candidate rows: the same products, another sum order
            e_full = per_user_err(sub, users, to_np(got), to_np(full)[cand], "bf16", TOL["bf16"])
            say(f"[cached] {label} vs full forward: checked {e_full['checked']:.2e} literal {e_full['literal']:.2e}")
            assert e_full["checked"] <= TOL["bf16"]
        else:
            # oracle on [user side | this request's candidates]
            qf, kf, vf = (vals[n].copy() for n in ("q", "k", "v"))
            for n, x in (("q", qf), ("k", kf), ("v", vf)):
                x[cand] = to_np({"q": qc, "k": kc, "v": vc}[n])
            want = oracle.attn_fwd(L.offsets, L.seg, L.ts, qf, kf, vf, inp["rab_np"])[cand]
        bound = operand_rounding_bounds(L.offsets, L.seg, L.ts, qf if r else vals["q"], kf if r else vals["k"],
                                        vf if r else vals["v"], vals["q"], inp["rab_np"])["o"][cand]
        e = per_user_err(sub, users, to_np(got), want, "bf16", TOL["bf16"], bound)
        record(f"cached-{label}-request{r}", {"o": e})
        say(f"[cached] {label} request {r} vs oracle: checked {e['checked']:.2e} literal {e['literal']:.2e}")
        assert e["checked"] <= TOL["bf16"], (label, r, e)


def ops_layout(jag_c, L):
    """Layout object over the candidate rows (per-user offsets of the request)."""
    off = jag_c.offsets.cpu().numpy().astype(np.int64)
    return Layout(L.spec, off, jag_c.seg.cpu().numpy(), jag_c.ts.cpu().numpy(), L.counts, {})


def custom(dh, rab):
    U, S, R, C = SEG_USER, SEG_HIST, SEG_RT, SEG_CAND
    rng = np.random.default_rng(31)
    segs, tss = [], []
    for n_s, n_r, n_c, cts in ((300, 40, 150, "window"), (200, 30, 90, "request"), (130, 10, 0, "window"),
                               (0, 0, 70, "window"), (5, 3, 2, "window"), (60, 70, 140, "ties"),
                               (1000, 100, 260, "request")):
        hist = sorted(rng.integers(-10**6, 0, n_s).tolist())
        rt = sorted(rng.choice(86400, n_r, replace=False).tolist())
        if cts == "window":
            cand = rng.integers(0, 86400, n_c).tolist()
        elif cts == "request":
            cand = [86400] * n_c
        else:   # candidates stamped exactly at RT times (ties are hidden, rule 2)
            cand = [rt[i % max(n_r, 1)] if n_r else 0 for i in range(n_c)]
        segs.append([U] * 4 + [S] * n_s + [R] * n_r + [C] * n_c)
        tss.append([0] * 4 + hist + rt + cand)
    segs.append([C] * 40)                                  # no user-side token at all
    tss.append(rng.integers(0, 86400, 40).tolist())
    return custom_layout(segs, tss, heads=2, head_dim=dh, dtype="bf16", rab_buckets=rab)


@pytest.mark.parametrize("dh,rab", [(128, 0), (64, 64), (128, 64)])
def test_custom_users(dh, rab):
    run_case(custom(dh, rab), f"custom-{dh}-rab{rab}", requests=2)


def long_user(dh, rab):
    """A user whose cached side spans two windows of the tile walker (4,864 tokens, 76 tiles of
    64; real-time tokens in time order), with 300 candidates, and a short user beside it."""
    U, S, R, C = SEG_USER, SEG_HIST, SEG_RT, SEG_CAND
    rng = np.random.default_rng(37)
    segs, tss = [], []
    for n_u, n_s, n_r, n_c in ((4, 60, 4800, 300), (2, 30, 5, 20)):
        segs.append([U] * n_u + [S] * n_s + [R] * n_r + [C] * n_c)
        tss.append([0] * n_u + sorted(rng.integers(-10**7, 0, n_s).tolist()) +
                   sorted(rng.choice(10**6, n_r, replace=False).tolist()) + rng.integers(0, 10**6, n_c).tolist())
    return custom_layout(segs, tss, heads=2, head_dim=dh, dtype="bf16", rab_buckets=rab)


@pytest.mark.parametrize("dh,rab", [(128, 0), (64, 64)])
def test_long_cached_side(dh, rab):
    run_case(long_user(dh, rab), f"long-{dh}-rab{rab}", requests=2)


def test_serving_users():
    L = make_layout("serving")
    lens = np.diff(L.offsets)
    users = sorted({0, 1, int(np.argmax(lens)), int(np.argmin(lens)), L.num_users - 1})
    run_case(L.subset(users), "serving-subset", requests=2)


def test_cached_rejects_mismatch():
    L = custom(64, 0)
    inp = make_inputs(L, all_exact=True)
    side, cand, jag_s, jag_c = split(L)
    k = inp["k"]
    cache = ops.user_cache(k[torch.from_numpy(side).cuda()].contiguous(), inp["v"][torch.from_numpy(side).cuda()].contiguous(), jag_s)
    qc = inp["q"][torch.from_numpy(cand).cuda()].contiguous()
    bad = ops.UserCache(ops.Jagged(jag_s.offsets[:-1], jag_s.seg, jag_s.ts, jag_s.max_seqlen), cache.k, cache.v,
                        cache.plan)
    with pytest.raises(hstu.MtgrError) as e:     # one user fewer in the cache
        ops.attn_fwd_cached(qc, qc, qc, jag_c, bad)
    assert e.value.status == hstu.MTGR_ERROR_INVALID_ARGUMENT
